"""GPU test of the allocation-free entry point symtile_gemm_all_scatter_noalloc
(through the C ABI): its heap, counters and values equal those of
symtile_gemm_all_scatter with a caller workspace, bit for bit, on two calls
in a row (the second smaller, so it runs on what the first left in the
scratch), and both match the oracle."""
import numpy as np
import pytest
import torch

from tests.gpu_util import Problem, check_gathered, oracle_block, require_gpu, sym, u16

pytestmark = pytest.mark.gpu

BULK, FUSED, WGSPEC, UNFUSED = 0, 1, 2, 3


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _noalloc(pkg, p, rank, variant, split_k, **kw):
    cfg = pkg.GasConfig(variant=variant, tile_m=p.out.tile_m, tile_n=p.out.tile_n,
                        split_k=split_k, **kw)
    dt = pkg.BF16 if p.dtype == "bf16" else pkg.F16
    pkg.symtile_gemm_all_scatter_noalloc(
        p.heap.handle, p.dA.data_ptr(), p.dB[rank].data_ptr(), p.heap.ptr(rank, p.out.c_off),
        p.heap.ptr(rank, p.out.flag_off), p.out.ready.data_ptr(), p.M, p.N, p.K, p.K, p.N, dt,
        rank, p.world, cfg, pkg.current_stream())
    p.calls[rank] += 1


CASES = [  # world, M, N, K, dtype, tile, split, rank, variant, split_reduce
    (8, 1024, 1024, 4096, "bf16", (128, 128), 4, 0, FUSED, 0),     # reduction kernel
    (3, 300, 136, 520, "f16", (64, 64), 3, 2, BULK, 1),            # last slice
]


def test_noalloc_equals_the_workspace_call_on_two_calls_in_a_row():
    pkg = sym()
    for world, M, N, K, dtype, (tm, tn), split, rank, variant, red in CASES:
        ref = Problem(world, M, N, K, dtype, tm, tn, seed=M + K)
        got = Problem(world, M, N, K, dtype, tm, tn, seed=M + K)
        for p in (ref, got):
            p.sentinel()
        ref.run(rank, variant, split_k=split, split_reduce=red)
        _noalloc(pkg, got, rank, variant, split, split_reduce=red)
        ref.barrier()
        got.barrier()
        want = {rank: oracle_block(got.A, got.shards[rank], dtype)}
        check_gathered(got, want)
        check_gathered(ref, want)
        assert np.array_equal(u16(got.out.C_all()), u16(ref.out.C_all())), (M, N, K)
        assert torch.equal(got.out.arrived_all(), ref.out.arrived_all())


def test_noalloc_without_split_and_argument_errors():
    pkg = sym()
    p = Problem(2, 128, 64, 256, "bf16", 64, 64, seed=3)
    p.sentinel()
    _noalloc(pkg, p, 1, FUSED, 0)                       # no split: no scratch involved
    p.barrier()
    check_gathered(p, {1: oracle_block(p.A, p.shards[1], "bf16")})
    ws = p.out.workspace(2)
    for kw, name in ((dict(variant=FUSED, split_k=2, workspace=ws.data_ptr(),
                           workspace_bytes=ws.numel()), "EINVAL"),     # takes no workspace
                     (dict(variant=UNFUSED, split_k=0), "EUNSUPPORTED")):
        with pytest.raises(pkg.SymtileError) as e:
            cfg = pkg.GasConfig(tile_m=64, tile_n=64, **kw)
            pkg.symtile_gemm_all_scatter_noalloc(
                p.heap.handle, p.dA.data_ptr(), p.dB[0].data_ptr(), p.heap.ptr(0, p.out.c_off),
                p.heap.ptr(0, p.out.flag_off), p.out.ready.data_ptr(), 128, 64, 256, 256, 64,
                pkg.BF16, 0, 2, cfg, pkg.current_stream())
        assert e.value.name == name, kw
    # a workspace larger than the scratch: 128 tiles of 256x256 in 3 slices (96 MiB)
    assert pkg.symtile_gas_workspace_bytes(8192, 1024, 256, 256, 3) > pkg.NOALLOC_SCRATCH_BYTES
    big = Problem(1, 8192, 1024, 96, "f16", 256, 256, seed=1)
    with pytest.raises(pkg.SymtileError) as e:
        _noalloc(pkg, big, 0, FUSED, 3)
    assert e.value.name == "EINVAL" and "exceeds the scratch" in str(e.value)
    p.barrier()
    big.barrier()
