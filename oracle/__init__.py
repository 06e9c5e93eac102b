"""ORACLE — test infrastructure, not part of the product.

Plain, slow CPU model of one rank's share of the fused GEMM + All-Scatter of
"Iris: First-Class Multi-GPU Programming Experience in Triton"
(arXiv 2511.12500), used only by ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py``.  The arithmetic lives in
``oracle.c`` (built with gcc, no fast-math); this module only marshals numpy
arrays into it and composes the steps in the paper's order:

1. decode the 16-bit input bits to binary32 (exact widening);
2. GEMM with an fp32 accumulator in increasing k (Section 4, GEMM main-loop
   listing);
3. placement of the rank's block at column offset ``rank * N_local`` of the
   gathered output in every slot, own slot included (Section 4.2.1);
4. one arrival count per tile per slot (counter reading of the lock
   protocol of Section 4.2.2);
5. the heap tile copy rank r -> rank (r + shift) mod w (Section 3.3.2).

It imports nothing from the HIP package and the HIP package imports nothing
from here.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F16 = 1
BF16 = 2

_lib = None


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile ``oracle.c`` with gcc into a shared library and return its path."""
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-shared", "-fPIC", "-o", out, src]
    subprocess.run(cmd, check=True)
    return out


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    _lib = load_library(_LIB)
    return _lib


def load_library(path: str):
    """Load an oracle shared library and declare its C signatures."""
    lib = ctypes.CDLL(path)
    p = ctypes.c_void_p
    i64 = ctypes.c_int64
    i32 = ctypes.c_int
    lib.oracle_decode16.argtypes = [p, p, i64, i32]
    lib.oracle_decode16.restype = i32
    lib.oracle_gemm_f32.argtypes = [p, p, p, i64, i64, i64, i64, i64, i64]
    lib.oracle_gemm_f32.restype = None
    lib.oracle_gemm_entries.argtypes = [p, p, i64, i64, i64, p, p, i64, p]
    lib.oracle_gemm_entries.restype = None
    lib.oracle_place.argtypes = [p, i64, i64, i32, i32, p, p]
    lib.oracle_place.restype = None
    lib.oracle_flags.argtypes = [p, i32, i32, i64, i64, ctypes.c_uint32]
    lib.oracle_flags.restype = None
    lib.oracle_tile_copy.argtypes = [p, p, p, i32, i64, i64, i32, i64, i64, i32, i32, i32]
    lib.oracle_tile_copy.restype = None
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _dtype_code(dtype: str) -> int:
    if dtype in ("f16", "float16", "fp16"):
        return F16
    if dtype in ("bf16", "bfloat16"):
        return BF16
    raise ValueError(f"unknown 16-bit dtype {dtype!r}")


def decode16(bits: np.ndarray, dtype: str, lib=None) -> np.ndarray:
    """Exact binary32 value of every 16-bit pattern in ``bits`` (uint16)."""
    lib = lib or _load()
    src = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(src.shape, dtype=np.float32)
    rc = lib.oracle_decode16(_ptr(src), _ptr(out), src.size, _dtype_code(dtype))
    if rc != 0:
        raise ValueError("oracle_decode16 rejected the dtype")
    return out


def gemm(A: np.ndarray, B: np.ndarray, lib=None) -> np.ndarray:
    """fp32 C = A @ B, one fp32 accumulator per element, increasing k."""
    lib = lib or _load()
    A = np.ascontiguousarray(A, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.float32)
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    C = np.empty((M, N), dtype=np.float32)
    if M and N:
        lib.oracle_gemm_f32(_ptr(A), _ptr(B), _ptr(C), M, N, K, K, N, N)
    return C


def gemm_entries(A: np.ndarray, B: np.ndarray, rows, cols, lib=None) -> np.ndarray:
    """fp32 C[rows[t], cols[t]] by the same definition as :func:`gemm`."""
    lib = lib or _load()
    A = np.ascontiguousarray(A, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.float32)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    M, K = A.shape
    _, N = B.shape
    if rows.shape != cols.shape:
        raise ValueError("rows and cols differ in shape")
    if rows.size and (rows.min() < 0 or rows.max() >= M or cols.min() < 0 or cols.max() >= N):
        raise IndexError("sample index out of range")
    out = np.empty(rows.shape, dtype=np.float32)
    if rows.size:
        lib.oracle_gemm_entries(_ptr(A), _ptr(B), K, K, N, _ptr(rows), _ptr(cols),
                                rows.size, _ptr(out))
    return out


def tiles(extent: int, tile: int) -> int:
    """Number of tiles of size ``tile`` covering ``extent`` (ragged edge counted)."""
    return (extent + tile - 1) // tile


class GatheredState:
    """Expected post-state of the gathered output and the arrival counters.

    ``G`` is [w, M, w*N_local] fp32 (NaN where nothing was stored),
    ``written`` the matching byte mask, ``arrived`` [w, w, tiles_m, tiles_n]
    uint32 counters.
    """

    def __init__(self, world: int, M: int, N_local: int, tile_m: int, tile_n: int):
        self.world, self.M, self.N_local = world, M, N_local
        self.tile_m, self.tile_n = tile_m, tile_n
        self.G = np.full((world, M, world * N_local), np.nan, dtype=np.float32)
        self.written = np.zeros((world, M, world * N_local), dtype=np.uint8)
        self.arrived = np.zeros((world, world, tiles(M, tile_m), tiles(N_local, tile_n)),
                                dtype=np.uint32)


def gemm_all_scatter(state: GatheredState, A_bits: np.ndarray, B_bits: np.ndarray,
                     dtype: str, rank: int, lib=None) -> np.ndarray:
    """Apply one call of rank ``rank`` to ``state`` and return its fp32 block.

    A_bits is [M, K] uint16, B_bits the rank's shard [K, N_local] uint16, both
    the 16-bit patterns of ``dtype``.  Steps in the paper's order: decode,
    GEMM with fp32 accumulation, placement into every slot, one arrival per
    tile per slot.
    """
    lib = lib or _load()
    world, M, N_local = state.world, state.M, state.N_local
    if not 0 <= rank < world:
        raise ValueError("rank out of range")
    if A_bits.shape[0] != M or B_bits.shape[1] != N_local:
        raise ValueError("shapes do not match the state")
    A = decode16(A_bits, dtype, lib)
    B = decode16(B_bits, dtype, lib)
    C = gemm(A, B, lib)
    G = np.ascontiguousarray(state.G)
    W = np.ascontiguousarray(state.written)
    if M and N_local:
        lib.oracle_place(_ptr(C), M, N_local, world, rank, _ptr(G), _ptr(W))
    state.G, state.written = G, W
    arr = np.ascontiguousarray(state.arrived)
    lib.oracle_flags(_ptr(arr), world, rank, arr.shape[2], arr.shape[3], 1)
    state.arrived = arr
    return C


def tile_copy(send: np.ndarray, recv: np.ndarray, tile_r: int, tile_c: int,
              shift: int = 1, only_rank: int = -1, lib=None, get: bool = False):
    """Expected (recv, copyflag) after every rank r (or only ``only_rank``)
    copies tile by tile, Section 3.3.2: put (default) sends send[r] to
    recv[(r + shift) mod w]; get pulls send[(r - shift) mod w] into recv[r].
    The counter of a tile is in the destination slot.  send/recv are
    [w, rows, cols]."""
    lib = lib or _load()
    send = np.ascontiguousarray(send)
    out = np.array(recv, copy=True, order="C")
    if send.shape != out.shape or send.dtype != out.dtype:
        raise ValueError("send and recv differ in shape or dtype")
    world, rows, cols = send.shape
    flags = np.zeros((world, tiles(rows, tile_r) * tiles(cols, tile_c)), dtype=np.uint32)
    lib.oracle_tile_copy(_ptr(send), _ptr(out), _ptr(flags), world, rows, cols,
                         send.dtype.itemsize, tile_r, tile_c, shift, only_rank, int(get))
    return out, flags
