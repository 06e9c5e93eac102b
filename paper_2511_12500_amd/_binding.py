"""ctypes declarations of ``include/symtile.h``; one Python function per C
entry point, with the same name.  Pointers and streams are plain ints."""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsymtile.so")

F16, BF16, F32 = 1, 2, 3
BULK_SYNC, FUSED_SEQ, WG_SPEC, UNFUSED_PC, WAVE_SPEC = 0, 1, 2, 3, 4
SPLIT_REDUCE_AUTO, SPLIT_REDUCE_LAST, SPLIT_REDUCE_BANDED, SPLIT_REDUCE_KERNEL = 0, 1, 2, 3
PUT, GET = 0, 1
LOAD, STORE = 0, 1
ATOMIC_OPS = {"add": 0, "xchg": 1, "cas": 2, "and": 3, "or": 4, "xor": 5, "min": 6, "max": 7}
SEMS = {"relaxed": 0, "acquire": 1, "release": 2, "acq_rel": 3}
SCOPES = {"block": 0, "gpu": 1, "sys": 2}
MP_FORMS = {"relaxed": 0, "fences": 1, "rmw": 2, "cas": 3, "wt": 4, "ack": 5,
            "wt_coherent": 6, "wt_plain": 7}
SB_FORMS = {"relaxed": 0, "acq_rel": 1, "seq_cst": 2}

_STATUS = {0: "OK", -1: "EINVAL", -2: "ENOMEM", -3: "EHIP", -4: "ETIMEOUT", -5: "EUNSUPPORTED"}


class SymtileError(RuntimeError):
    """A non-zero symtile_status, with the library's message."""

    def __init__(self, status: int, func: str, message: str):
        self.status = status
        self.name = _STATUS.get(status, str(status))
        super().__init__(f"{func}: {self.name}: {message}")


class GasConfig(ctypes.Structure):
    """Mirror of ``symtile_gas_config``."""

    _fields_ = [
        ("variant", ctypes.c_int),
        ("tile_m", ctypes.c_int),
        ("tile_n", ctypes.c_int),
        ("gemm_wgs", ctypes.c_int),
        ("copy_wgs", ctypes.c_int),
        ("epoch", ctypes.c_uint32),
        ("spin_limit", ctypes.c_uint32),
        ("nontemporal", ctypes.c_int),
        ("group_m", ctypes.c_int),
        ("waves_per_wg", ctypes.c_int),
        ("copy_stream", ctypes.c_void_p),
        ("trace", ctypes.c_void_p),
        ("split_k", ctypes.c_int),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("split_reduce", ctypes.c_int),
    ]


TRACE_WORDS = 8   # SYMTILE_TRACE_WORDS
(TRACE_START, TRACE_MAINLOOP, TRACE_STORED, TRACE_RELEASED, TRACE_WHERE, TRACE_COPY_WAIT,
 TRACE_COPY_GO, TRACE_COPY_DONE) = range(8)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2511_12500_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, sz, i32, u32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_uint32
    pvp = ctypes.POINTER(ctypes.c_void_p)
    decl = {
        "symtile_heap_create": [i32, i32, sz, pvp],
        "symtile_heap_create_on": [i32, i32, sz, vp, sz, pvp],
        "symtile_heap_destroy": [vp],
        "symtile_heap_alloc": [vp, sz, sz, ctypes.POINTER(sz)],
        "symtile_heap_ptr": [vp, i32, sz, pvp],
        "symtile_heap_info": [vp, ctypes.POINTER(i32), ctypes.POINTER(sz), ctypes.POINTER(sz),
                              ctypes.POINTER(i32)],
        "symtile_heap_bases": [vp, pvp, ctypes.POINTER(ctypes.c_uint64)],
        "symtile_translate": [vp, vp, i32, i32, pvp],
        "symtile_translate_device": [vp, vp, i32, i32, i32, vp, vp],
        "symtile_barrier": [vp, vp],
        "symtile_heap_fill": [vp, i32, sz, sz, i32, vp],
        "symtile_atomic_exercise": [vp, i32, i32, i32, sz, i32, i32, i32, u32, u32, vp, vp],
        "symtile_tile_copy": [vp, sz, sz, i32, i32, i32, i32, i32, i32, i32, i32, sz, i32, i32,
                              vp],
        "symtile_tile_copy_timed": [vp, sz, sz, i32, i32, i32, i32, i32, i32, i32, i32, sz, i32,
                                    i32, vp, ctypes.POINTER(ctypes.c_float)],
        "symtile_gemm_all_scatter": [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32,
                                     i32, ctypes.POINTER(GasConfig), vp],
        "symtile_gemm_all_scatter_noalloc": [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                             i32, i32, i32, ctypes.POINTER(GasConfig), vp],
        "symtile_device_info": [i32, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "symtile_gas_workspace_bytes": [i32, i32, i32, i32, i32, ctypes.POINTER(sz)],
        "symtile_clock_rate_khz": [i32, ctypes.POINTER(i32)],
        "symtile_litmus_mp": [vp, sz, sz, i32, i32, i32, i32, i32, u32, vp, vp],
        "symtile_litmus_sb": [vp, sz, i32, i32, i32, i32, u32, vp, vp],
        "symtile_value_exercise": [vp, i32, sz, sz, sz, i32, i32, i32, vp],
    }
    for name, args in decl.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = i32
    L.symtile_last_error.argtypes = []
    L.symtile_last_error.restype = ctypes.c_char_p
    L.symtile_version.argtypes = []
    L.symtile_version.restype = ctypes.c_char_p
    return L


lib = _load()


def symtile_last_error() -> str:
    return lib.symtile_last_error().decode()


def symtile_version() -> str:
    return lib.symtile_version().decode()


def _check(status: int, func: str) -> None:
    if status != 0:
        raise SymtileError(status, func, symtile_last_error())


def _vp(x) -> ctypes.c_void_p:
    return ctypes.c_void_p(int(x) if x else None)


def symtile_heap_create(device: int, world_size: int, slot_bytes: int) -> int:
    out = ctypes.c_void_p()
    _check(lib.symtile_heap_create(device, world_size, slot_bytes, ctypes.byref(out)),
           "symtile_heap_create")
    return out.value


def symtile_heap_create_on(device: int, world_size: int, slot_bytes: int, base: int,
                           total_bytes: int) -> int:
    out = ctypes.c_void_p()
    _check(lib.symtile_heap_create_on(device, world_size, slot_bytes, _vp(base), total_bytes,
                                      ctypes.byref(out)), "symtile_heap_create_on")
    return out.value


def symtile_heap_destroy(h: int) -> None:
    _check(lib.symtile_heap_destroy(_vp(h)), "symtile_heap_destroy")


def symtile_heap_alloc(h: int, nbytes: int, align: int = 256) -> int:
    off = ctypes.c_size_t()
    _check(lib.symtile_heap_alloc(_vp(h), nbytes, align, ctypes.byref(off)), "symtile_heap_alloc")
    return off.value


def symtile_heap_ptr(h: int, rank: int, offset: int) -> int:
    out = ctypes.c_void_p()
    _check(lib.symtile_heap_ptr(_vp(h), rank, offset, ctypes.byref(out)), "symtile_heap_ptr")
    return out.value or 0


def symtile_heap_info(h: int):
    w, dev = ctypes.c_int(), ctypes.c_int()
    stride, used = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib.symtile_heap_info(_vp(h), ctypes.byref(w), ctypes.byref(stride), ctypes.byref(used),
                                 ctypes.byref(dev)), "symtile_heap_info")
    return w.value, stride.value, used.value, dev.value


def symtile_heap_bases(h: int):
    """(device address of the bases array, [host copy of the bases])."""
    w = symtile_heap_info(h)[0]
    dev = ctypes.c_void_p()
    host = (ctypes.c_uint64 * w)()
    _check(lib.symtile_heap_bases(_vp(h), ctypes.byref(dev), host), "symtile_heap_bases")
    return dev.value, list(host)


def symtile_translate(h: int, p: int, from_rank: int, to_rank: int) -> int:
    out = ctypes.c_void_p()
    _check(lib.symtile_translate(_vp(h), _vp(p), from_rank, to_rank, ctypes.byref(out)),
           "symtile_translate")
    return out.value or 0


def symtile_translate_device(h: int, in_ptr: int, n: int, from_rank: int, to_rank: int,
                             out_ptr: int, stream: int = 0) -> None:
    _check(lib.symtile_translate_device(_vp(h), _vp(in_ptr), n, from_rank, to_rank,
                                        _vp(out_ptr), _vp(stream)), "symtile_translate_device")


def symtile_barrier(h: int, stream: int = 0) -> None:
    _check(lib.symtile_barrier(_vp(h), _vp(stream)), "symtile_barrier")


def symtile_heap_fill(h: int, rank: int, offset: int, nbytes: int, value: int,
                      stream: int = 0) -> None:
    _check(lib.symtile_heap_fill(_vp(h), rank, offset, nbytes, value, _vp(stream)),
           "symtile_heap_fill")


def symtile_atomic_exercise(h: int, op: int, sem: int, scope: int, offset: int, from_rank: int,
                            to_rank: int, n_threads: int, operand: int, compare: int = 0,
                            old_out: int = 0, stream: int = 0) -> None:
    _check(lib.symtile_atomic_exercise(_vp(h), op, sem, scope, offset, from_rank, to_rank,
                                       n_threads, operand & 0xFFFFFFFF, compare & 0xFFFFFFFF,
                                       _vp(old_out), _vp(stream)), "symtile_atomic_exercise")


def symtile_value_exercise(h: int, op: int, src_off: int, dst_off: int, nbytes: int,
                           cur_rank: int, remote_rank: int, nontemporal: int = 0,
                           stream: int = 0) -> None:
    """op: LOAD (0) or STORE (1)."""
    _check(lib.symtile_value_exercise(_vp(h), op, src_off, dst_off, nbytes, cur_rank,
                                      remote_rank, nontemporal, _vp(stream)),
           "symtile_value_exercise")


def symtile_tile_copy(h: int, src_off: int, dst_off: int, rows: int, cols: int, ld: int,
                      dtype: int, tile_r: int, tile_c: int, shift: int, only_rank: int,
                      flag_off: int, tiles_per_wg: int = 0, stream: int = 0,
                      mode: int = 0) -> None:
    """mode: PUT (0) or GET (1); the C argument order is ..., tiles_per_wg,
    mode, stream."""
    _check(lib.symtile_tile_copy(_vp(h), src_off, dst_off, rows, cols, ld, dtype, tile_r, tile_c,
                                 shift, only_rank, flag_off, tiles_per_wg, mode, _vp(stream)),
           "symtile_tile_copy")


def symtile_tile_copy_timed(h: int, src_off: int, dst_off: int, rows: int, cols: int, ld: int,
                            dtype: int, tile_r: int, tile_c: int, shift: int, only_rank: int,
                            flag_off: int, tiles_per_wg: int = 0, stream: int = 0,
                            mode: int = 0) -> float:
    """symtile_tile_copy with the kernel bracketed by events; waits for it and
    returns its duration in ms."""
    ms = ctypes.c_float()
    _check(lib.symtile_tile_copy_timed(_vp(h), src_off, dst_off, rows, cols, ld, dtype, tile_r,
                                       tile_c, shift, only_rank, flag_off, tiles_per_wg, mode,
                                       _vp(stream), ctypes.byref(ms)), "symtile_tile_copy_timed")
    return ms.value


def symtile_gemm_all_scatter(h: int, A: int, B_shard: int, C_gathered_local: int,
                             arrived_local: int, ready: int, M: int, N_local: int, K: int,
                             lda: int, ldb: int, dtype: int, rank: int, world_size: int,
                             cfg: GasConfig | None, stream: int = 0) -> None:
    _check(lib.symtile_gemm_all_scatter(_vp(h), _vp(A), _vp(B_shard), _vp(C_gathered_local),
                                        _vp(arrived_local), _vp(ready), M, N_local, K, lda, ldb,
                                        dtype, rank, world_size,
                                        ctypes.byref(cfg) if cfg is not None else None,
                                        _vp(stream)), "symtile_gemm_all_scatter")


NOALLOC_SCRATCH_BYTES = (64 << 20) + (64 << 10)   # SYMTILE_NOALLOC_SCRATCH_BYTES


def symtile_gemm_all_scatter_noalloc(h: int, A: int, B_shard: int, C_gathered_local: int,
                                     arrived_local: int, ready: int, M: int, N_local: int, K: int,
                                     lda: int, ldb: int, dtype: int, rank: int, world_size: int,
                                     cfg: GasConfig | None, stream: int = 0) -> None:
    """symtile_gemm_all_scatter with the split-K workspace in the library's
    static scratch (cfg.workspace must be None)."""
    _check(lib.symtile_gemm_all_scatter_noalloc(_vp(h), _vp(A), _vp(B_shard),
                                                _vp(C_gathered_local), _vp(arrived_local),
                                                _vp(ready), M, N_local, K, lda, ldb, dtype, rank,
                                                world_size,
                                                ctypes.byref(cfg) if cfg is not None else None,
                                                _vp(stream)), "symtile_gemm_all_scatter_noalloc")


def symtile_gas_workspace_bytes(M: int, N_local: int, tile_m: int, tile_n: int,
                                split_k: int) -> int:
    """Bytes of the split-K workspace of a call (0 when split_k <= 1)."""
    out = ctypes.c_size_t()
    _check(lib.symtile_gas_workspace_bytes(M, N_local, tile_m, tile_n, split_k, ctypes.byref(out)),
           "symtile_gas_workspace_bytes")
    return out.value


def symtile_litmus_mp(h: int, data_off: int, flag_off: int, pairs: int, rounds: int,
                      words: int, form: int, scope: int, spin_limit: int, result: int,
                      stream: int = 0) -> None:
    """form: MP_FORMS[...]; scope: SCOPES[...]."""
    _check(lib.symtile_litmus_mp(_vp(h), data_off, flag_off, pairs, rounds, words, form, scope,
                                 spin_limit, _vp(result), _vp(stream)), "symtile_litmus_mp")


def symtile_litmus_sb(h: int, flag_off: int, pairs: int, rounds: int, form: int, scope: int,
                      spin_limit: int, out: int, stream: int = 0) -> None:
    """form: SB_FORMS[...]; scope: SCOPES[...]."""
    _check(lib.symtile_litmus_sb(_vp(h), flag_off, pairs, rounds, form, scope, spin_limit,
                                 _vp(out), _vp(stream)), "symtile_litmus_sb")


def symtile_clock_rate_khz(device: int) -> int:
    """Rate of the realtime counter behind trace timestamps, in kHz."""
    khz = ctypes.c_int()
    _check(lib.symtile_clock_rate_khz(device, ctypes.byref(khz)), "symtile_clock_rate_khz")
    return khz.value


def symtile_device_info(device: int, tile_m: int = 256, tile_n: int = 256):
    """(CU count, largest co-resident WG_SPEC grid for the tile shape)."""
    cus, lim = ctypes.c_int(), ctypes.c_int()
    _check(lib.symtile_device_info(device, tile_m, tile_n, ctypes.byref(cus), ctypes.byref(lim)),
           "symtile_device_info")
    return cus.value, lim.value
