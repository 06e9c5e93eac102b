"""symtile: one GPU's share of the fused GEMM + All-Scatter (arXiv 2511.12500)
on MI355X, as a C-ABI library (``libsymtile.so``) plus this thin binding.

The binding only marshals arguments: every step of the hot path runs in the
HIP kernels of ``libsymtile.so``.  The library is loaded on first use of any
binding name; that raises ImportError when it has not been built
(``python -m paper_2511_12500_amd.build``).  There is no CPU fallback.
PyTorch supplies device memory and streams.  ``paper_2511_12500_amd.build``
itself imports without the library, so a fresh checkout can build it.
"""
_BINDING = (
    "ATOMIC_OPS", "BF16", "BULK_SYNC", "F16", "F32", "FUSED_SEQ", "GET", "LIB_PATH", "LOAD",
    "PUT", "SCOPES", "SEMS", "STORE", "MP_FORMS", "SB_FORMS", "symtile_litmus_sb",
    "SPLIT_REDUCE_AUTO", "SPLIT_REDUCE_LAST", "SPLIT_REDUCE_BANDED", "SPLIT_REDUCE_KERNEL",
    "TRACE_WORDS", "UNFUSED_PC", "WAVE_SPEC", "WG_SPEC", "GasConfig", "SymtileError", "lib", "symtile_atomic_exercise",
    "symtile_barrier", "symtile_clock_rate_khz", "symtile_device_info",
    "symtile_gas_workspace_bytes", "symtile_gemm_all_scatter",
    "symtile_gemm_all_scatter_noalloc", "NOALLOC_SCRATCH_BYTES", "symtile_heap_alloc", "symtile_heap_bases", "symtile_litmus_mp", "symtile_heap_create", "symtile_heap_create_on",
    "symtile_heap_destroy", "symtile_heap_fill", "symtile_heap_info", "symtile_heap_ptr",
    "symtile_last_error", "symtile_tile_copy", "symtile_tile_copy_timed", "symtile_translate", "symtile_translate_device",
    "symtile_value_exercise", "symtile_version",
)
_HEAP = ("GatheredOutput", "Heap", "current_stream")

__all__ = list(_BINDING + _HEAP)


def __getattr__(name):
    if name in _BINDING:
        from . import _binding
        return getattr(_binding, name)
    if name in _HEAP:
        from . import heap
        return getattr(heap, name)
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")


def __dir__():
    return sorted(list(globals()) + __all__)
