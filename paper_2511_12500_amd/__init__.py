"""symtile: one GPU's share of the fused GEMM + All-Scatter (arXiv 2511.12500)
on MI355X, as a C-ABI library (``libsymtile.so``) plus this thin binding.

The binding only marshals arguments: every step of the hot path runs in the
HIP kernels of ``libsymtile.so``.  Importing the package fails loudly when
the library has not been built (``python -m paper_2511_12500_amd.build``);
there is no CPU fallback.  PyTorch supplies device memory and streams.
"""
from ._binding import (  # noqa: F401
    ATOMIC_OPS, BF16, BULK_SYNC, F16, F32, FUSED_SEQ, LIB_PATH, SCOPES, SEMS, WG_SPEC,
    GasConfig, SymtileError, lib, symtile_atomic_exercise, symtile_barrier,
    symtile_device_info, symtile_gemm_all_scatter, symtile_heap_alloc, symtile_heap_bases,
    symtile_heap_create, symtile_heap_create_on, symtile_heap_destroy, symtile_heap_fill,
    symtile_heap_info, symtile_heap_ptr, symtile_last_error, symtile_tile_copy,
    symtile_translate, symtile_translate_device, symtile_version,
)
from .heap import GatheredOutput, Heap, current_stream  # noqa: F401
