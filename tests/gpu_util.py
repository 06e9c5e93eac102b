"""Helpers shared by the GPU parity tests (imported only by ``-m gpu`` tests).

Expected values come from ``oracle`` only; the HIP path is reached through
the package's C-ABI binding."""
from __future__ import annotations

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


def check_block(got16: np.ndarray, want32: np.ndarray, dtype: str, what: str = ""):
    """Values of one rank block: finite, within tol * max|C|."""
    got = torch.from_numpy(got16.view(np.int16).copy()).view(tdtype(dtype)).float().numpy()
    assert np.all(np.isfinite(got)), f"{what}: non-finite (unwritten or overflow) elements"
    scale = float(np.max(np.abs(want32))) if want32.size else 0.0
    err = float(np.max(np.abs(got.astype(np.float64) - want32))) if want32.size else 0.0
    assert err <= TOL[dtype] * max(scale, 1e-30), \
        f"{what}: max|err| {err:.3e} > {TOL[dtype]} * max|C| {scale:.3e}"
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
