"""Helpers shared by the GPU parity tests (imported only by ``-m gpu`` tests).

Expected values come from ``oracle`` only; the HIP path is reached through
the package's C-ABI binding."""
from __future__ import annotations

from typing import NamedTuple

import numpy as np
import pytest
import torch

import oracle
import workload

TOL = {"bf16": 2e-2, "f16": 5e-3}        # max|err| <= tol * max|C| (fp32 accumulate)
SENTINEL = 0xFFFF                         # every byte 0xFF: a NaN in both 16-bit formats


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")


def sym():
    """The HIP package (raises if libsymtile.so is missing)."""
    import paper_2511_12500_amd as pkg
    return pkg


def tdtype(dtype: str) -> torch.dtype:
    return workload.torch_dtype(dtype)


def u16(t: torch.Tensor) -> np.ndarray:
    """16-bit patterns of a (device or host) 16-bit tensor as numpy uint16."""
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


class Problem:
    """Inputs, heap and gathered buffers for one GEMM + All-Scatter case."""

    def __init__(self, world, M, N, K, dtype, tile_m, tile_n, seed=0, dist="uniform",
                 A=None, shards=None):
        pkg = sym()
        self.world, self.M, self.N, self.K, self.dtype = world, M, N, K, dtype
        self.A = A if A is not None else workload.gemm_A(M, K, dtype, dist, seed)
        self.shards = shards if shards is not None else [
            workload.gemm_B_shard(K, N, r, dtype, dist, seed) for r in range(world)]
        tiles = -(-M // tile_m) * -(-N // tile_n)
        slot = M * world * N * 2 + world * tiles * 4 + (1 << 16)
        self.heap = pkg.Heap(world, slot)
        self.out = pkg.GatheredOutput(self.heap, M, N, tdtype(dtype), tile_m, tile_n)
        self.dA = self.A.cuda()
        self.dB = [b.cuda() for b in self.shards]
        self.calls = np.zeros(world, dtype=np.int64)

    def sentinel(self):
        self.out.C_all().view(torch.int16).fill_(-1)   # all bytes 0xFF

    def run(self, rank, variant, **kw):
        self.out.run(self.dA, self.dB[rank], rank, variant, **kw)
        self.calls[rank] += 1

    def barrier(self):
        self.heap.barrier()
        torch.cuda.synchronize()


def oracle_block(A: torch.Tensor, B: torch.Tensor, dtype: str) -> np.ndarray:
    """fp32 C = A @ B by the oracle (decode, fp32 accumulate)."""
    return oracle.gemm(oracle.decode16(workload.bits(A), dtype),
                       oracle.decode16(workload.bits(B), dtype))


class BoundedBlock(NamedTuple):
    """An oracle block with what the per-element accumulation bound needs:
    c = A @ B and abs_ab = |A| @ |B| (both by the oracle, fp32), and K."""
    c: np.ndarray
    abs_ab: np.ndarray
    K: int


def oracle_block_bounded(A: torch.Tensor, B: torch.Tensor, dtype: str) -> BoundedBlock:
    a = oracle.decode16(workload.bits(A), dtype)
    b = oracle.decode16(workload.bits(B), dtype)
    return BoundedBlock(oracle.gemm(a, b), oracle.gemm(np.abs(a), np.abs(b)), int(a.shape[1]))


# precision (significand bits, implicit bit included) and least normal exponent
_FMT = {"bf16": (8, -126), "f16": (11, -14)}


def accumulation_bound_violations(got: np.ndarray, ref: np.ndarray, abs_ab: np.ndarray, K: int,
                                  dtype: str) -> np.ndarray:
    """Mask of elements where |got - ref| exceeds the error analysis of the
    computation: got is an fp32 accumulation of K products rounded once to
    the output format, ref the oracle's fp32 accumulation of the same
    products.  Each fp32 sum of K terms lies within gamma_K * sum|a||b| of
    the exact value (gamma_K = K u / (1 - K u), u = 2^-24, whatever the
    order), and the output rounding adds at most half an output ulp of the
    value (taken at the larger of |got| and |ref|, which bounds it from
    above), so |got - ref| <= half_ulp + 2 gamma_K (|A||B|)_ij."""
    p, emin = _FMT[dtype]
    u = 2.0 ** -24
    gamma = K * u / (1.0 - K * u)
    mag = np.maximum(np.abs(got), np.abs(ref)).astype(np.float64)
    with np.errstate(divide="ignore"):
        e = np.where(mag > 0, np.floor(np.log2(np.where(mag > 0, mag, 1.0))), emin)
    half_ulp = np.exp2(np.maximum(e, emin) - p)
    bound = half_ulp + 2.0 * gamma * abs_ab.astype(np.float64)
    return np.abs(got.astype(np.float64) - ref.astype(np.float64)) > bound


def check_block(got16: np.ndarray, want, dtype: str, what: str = ""):
    """Values of one rank block: finite, within tol * max|C| (the stated
    tolerance); for a BoundedBlock also every element within the per-element
    accumulation bound."""
    got = torch.from_numpy(got16.view(np.int16).copy()).view(tdtype(dtype)).float().numpy()
    want32 = want.c if isinstance(want, BoundedBlock) else want
    assert np.all(np.isfinite(got)), f"{what}: non-finite (unwritten or overflow) elements"
    scale = float(np.max(np.abs(want32))) if want32.size else 0.0
    err = float(np.max(np.abs(got.astype(np.float64) - want32))) if want32.size else 0.0
    assert err <= TOL[dtype] * max(scale, 1e-30), \
        f"{what}: max|err| {err:.3e} > {TOL[dtype]} * max|C| {scale:.3e}"
    if isinstance(want, BoundedBlock) and want32.size:
        bad = accumulation_bound_violations(got, want.c, want.abs_ab, want.K, dtype)
        assert not bad.any(), \
            f"{what}: {int(bad.sum())} elements outside the accumulation bound, first at " \
            f"{tuple(int(i) for i in np.argwhere(bad)[0])}"
    return err, scale


def check_gathered(p: Problem, want_blocks: dict, flag_count: int | None = None):
    """Full post-state check of the heap after the calls recorded in p.calls.

    * bit-exact placement: blocks of ranks that ran hold values, every other
      element still holds the sentinel;
    * every slot holds bitwise the same gathered array;
    * values of each written block within tolerance of the oracle;
    * arrival counters: arrived[s][r][m][n] == calls of rank r, for every slot.
    Bit comparisons run on the device (torch ==); values are copied to the host.
    """
    w, N = p.world, p.N
    G = p.out.C_all().view(torch.int16)        # [w, M, w*N] on the device
    for s in range(1, w):
        assert bool(torch.equal(G[s], G[0])), f"slot {s} differs from slot 0"
    for r in range(w):
        blk = G[0][:, r * N:(r + 1) * N]
        if p.calls[r] == 0:
            assert bool((blk == -1).all()), f"block of rank {r} written without a call"
        else:
            check_block(u16(blk), want_blocks[r], p.dtype, f"rank {r} block")
    arr = p.out.arrived_all().cpu().numpy().astype(np.int64)   # [slot, src, tm, tn]
    for r in range(w):
        want = p.calls[r] if flag_count is None else flag_count
        if p.calls[r] == 0:
            want = 0
        assert np.all(arr[:, r] == want), f"arrival counters of rank {r}: {np.unique(arr[:, r])}"
