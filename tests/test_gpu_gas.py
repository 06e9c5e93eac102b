"""GPU parity of symtile_gemm_all_scatter against the oracle (through the C ABI).

Bit-exact: placement (sentinel mask), all-slot equality, arrival counters,
cross-variant heaps.  Values: max|err| <= tol * max|C| (2e-2 bf16, 5e-3 f16)."""
import numpy as np
import pytest
import torch

import oracle
import workload
from tests.gpu_util import (SENTINEL, Problem, check_block, check_gathered, oracle_block,
                            oracle_block_bounded, require_gpu, sym, u16)

pytestmark = pytest.mark.gpu

BULK, FUSED, WGSPEC, UNFUSED = 0, 1, 2, 3
VARIANTS = [BULK, FUSED, WGSPEC, UNFUSED]
VNAMES = {BULK: "bulk_sync", FUSED: "fused_seq", WGSPEC: "wg_spec", UNFUSED: "unfused_pc"}


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _blocks(p):
    """Oracle blocks of every rank, with the per-element accumulation bound."""
    return {r: oracle_block_bounded(p.A, p.shards[r], p.dtype) for r in range(p.world)}


# ---------------------------------------------------------------- tiny two-rank case

@pytest.mark.parametrize("variant", VARIANTS, ids=VNAMES.get)
def test_tiny_rank0_then_all_ranks(variant):
    w = workload.TINY
    p = Problem(w.world, w.M, w.N_local, w.K, w.dtype, w.tile_m, w.tile_n, dist=w.dist)
    want = _blocks(p)
    p.sentinel()
    p.run(0, variant)
    p.barrier()
    check_gathered(p, want)
    arr = p.out.arrived_all().cpu().numpy()
    assert arr.shape == (2, 2, 2, 1) and int(arr.sum()) == 4   # 2 tiles x 2 slots, rank 0
    p.run(1, variant)
    p.barrier()
    check_gathered(p, want)
    assert np.all(p.out.arrived_all().cpu().numpy() == 1)      # 4 counters per slot, all 1


# ---------------------------------------------------------------- ragged shapes

RAGGED = [
    # world, M, N_local, K, tile_m, tile_n, dtype
    (3, 300, 136, 200, 128, 128, "bf16"),
    (2, 77, 40, 24, 64, 64, "f16"),
    (4, 130, 264, 72, 256, 128, "bf16"),
    (5, 257, 264, 520, 256, 256, "f16"),
    (8, 64, 8, 8, 64, 64, "bf16"),
    # 256 x 224 tiles (16x16x32 MFMAs, B staged 256 wide): ragged rows,
    # columns and K, and a column tail narrower than one 16-column block
    (3, 300, 504, 200, 256, 224, "bf16"),
    (2, 257, 232, 72, 256, 224, "f16"),
]


@pytest.mark.parametrize("case", RAGGED, ids=lambda c: "w%d_m%d_n%d_k%d_t%dx%d_%s" % c)
@pytest.mark.parametrize("variant", VARIANTS, ids=VNAMES.get)
def test_ragged_all_ranks(case, variant):
    world, M, N, K, tm, tn, dtype = case
    p = Problem(world, M, N, K, dtype, tm, tn, seed=3)
    want = _blocks(p)
    p.sentinel()
    order = list(range(world))[::-1]
    for i, r in enumerate(order):
        p.run(r, variant)
        if i == 0:
            p.barrier()
            check_gathered(p, want)     # one rank only: the rest is still sentinel
    p.barrier()
    check_gathered(p, want)


# ---------------------------------------------------------------- closed forms

def test_identity_A_gives_B_exactly():
    n = 256
    A = torch.eye(n, dtype=torch.bfloat16)
    shards = [workload.gemm_B_shard(n, 128, r, "bf16", "uniform", 5) for r in range(2)]
    p = Problem(2, n, 128, n, "bf16", 128, 128, A=A, shards=shards)
    p.sentinel()
    for r in range(2):
        p.run(r, FUSED)
    p.barrier()
    G = u16(p.out.C_all())
    for r in range(2):
        assert np.array_equal(G[1][:, r * 128:(r + 1) * 128], workload.bits(shards[r]))


def test_all_ones_f16_is_exact():
    ones = torch.ones
    p = Problem(2, 128, 64, 256, "f16", 64, 64, A=ones(128, 256, dtype=torch.float16),
                shards=[ones(256, 64, dtype=torch.float16)] * 2)
    p.sentinel()
    p.run(0, WGSPEC)
    p.barrier()
    blk = u16(p.out.C_all())[:, :, :64]
    assert np.all(blk == 0x5C00)          # binary16 256.0


def test_one_hot_B_selects_columns_of_A():
    rng = np.random.default_rng(4)
    A = workload.gemm_A(96, 128, "bf16", "uniform", 9)
    sel = rng.integers(0, 128, size=64)
    Bf = torch.zeros(128, 64)
    Bf[torch.from_numpy(sel), torch.arange(64)] = 1.0
    Bh = Bf.to(torch.bfloat16)
    p = Problem(3, 96, 64, 128, "bf16", 64, 64, A=A, shards=[Bh] * 3)
    p.sentinel()
    p.run(2, BULK)
    p.barrier()
    got = u16(p.out.C_all())[0][:, 128:192]
    assert np.array_equal(got, workload.bits(A)[:, sel])


def test_world1_is_a_plain_gemm():
    M, N, K = 384, 256, 320
    p = Problem(1, M, N, K, "f16", 128, 128, seed=8)
    p.sentinel()
    p.run(0, FUSED)
    p.barrier()
    got = u16(p.out.C(0))
    check_block(got, oracle_block(p.A, p.shards[0], "f16"), "f16", "w=1 vs oracle")
    lib_ref = (p.dA.float() @ p.dB[0].float()).cpu().numpy()     # independent library GEMM
    check_block(got, lib_ref, "f16", "w=1 vs torch.matmul")


def test_k_zero_stores_zeros():
    p = Problem(2, 64, 64, 0, "bf16", 64, 64, A=torch.zeros(64, 0, dtype=torch.bfloat16),
                shards=[torch.zeros(0, 64, dtype=torch.bfloat16)] * 2)
    p.sentinel()
    p.run(1, WGSPEC)
    p.barrier()
    G = u16(p.out.C_all())
    assert np.all(G[:, :, 64:] == 0) and np.all(G[:, :, :64] == SENTINEL)
    assert np.all(p.out.arrived_all().cpu().numpy()[:, 1] == 1)


def test_empty_problem_is_a_noop():
    pkg = sym()
    heap = pkg.Heap(2, 1 << 20)
    out = pkg.GatheredOutput(heap, 0, 64, torch.float16, 64, 64)
    A = torch.zeros(0, 64, dtype=torch.float16, device="cuda")
    B = torch.zeros(64, 64, dtype=torch.float16, device="cuda")
    for v in VARIANTS:
        out.run(A, B, 0, v)
    out.run(A, B, 0, FUSED, split_k=2)          # no tiles: no workspace needed
    heap.barrier()


def test_k_zero_with_split_k():
    """K = 0 has no stage to split: split_k > 1 is refused, split_k = 1 stores zeros."""
    pkg = sym()
    p = Problem(2, 64, 64, 0, "bf16", 64, 64, A=torch.zeros(64, 0, dtype=torch.bfloat16),
                shards=[torch.zeros(0, 64, dtype=torch.bfloat16)] * 2)
    p.sentinel()
    with pytest.raises(pkg.SymtileError) as e:
        p.out.run(p.dA, p.dB[0], 0, FUSED, split_k=2)
    assert e.value.name == "EINVAL"
    p.run(0, FUSED, split_k=1)
    p.barrier()
    G = u16(p.out.C_all())
    assert np.all(G[:, :, :64] == 0) and np.all(G[:, :, 64:] == SENTINEL)


# ---------------------------------------------------------------- evaluation workloads

@pytest.mark.parametrize("variant", VARIANTS, ids=VNAMES.get)
def test_small_bf16_w8_rank0(variant):
    w = workload.SMALL_BF16
    p = Problem(w.world, w.M, w.N_local, w.K, w.dtype, w.tile_m, w.tile_n, dist=w.dist)
    want = {0: oracle_block_bounded(p.A, p.shards[0], w.dtype)}
    p.sentinel()
    p.run(0, variant)
    p.barrier()
    check_gathered(p, want)


def test_small_bf16_w8_every_rank_in_turn():
    w = workload.SMALL_BF16
    p = Problem(w.world, w.M, w.N_local, w.K, w.dtype, w.tile_m, w.tile_n, dist=w.dist, seed=1)
    want = _blocks(p)
    p.sentinel()
    for r in range(w.world):
        p.run(r, WGSPEC)
    p.barrier()
    check_gathered(p, want)
    # identity: every slot holds A @ [B_0 | ... | B_7] (float64 library matmul)
    full = p.A.double() @ torch.cat([b.double() for b in p.shards], dim=1)
    G = torch.from_numpy(u16(p.out.C_all())[3].view(np.int16).copy()).view(torch.bfloat16)
    err = (G.double() - full).abs().max().item()
    assert err <= 2e-2 * full.abs().max().item()


def _large_case(w, seed=0):
    return Problem(w.world, w.M, w.N_local, w.K, w.dtype, w.tile_m, w.tile_n, dist=w.dist,
                   seed=seed)


@pytest.mark.parametrize("wl", [workload.LARGE_BF16, workload.WIDE_F16], ids=lambda w: w.name)
def test_full_size_variants_match_oracle_and_each_other(wl):
    p = _large_case(wl)
    want = {0: oracle_block(p.A, p.shards[0], wl.dtype)}
    heaps = {}
    for v in (FUSED, WGSPEC, BULK, UNFUSED):
        p.sentinel()
        p.run(0, v)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[0]))
        heaps[v] = u16(p.out.C(5))[:, :wl.N_local].copy()
    for v in (WGSPEC, BULK, UNFUSED):
        assert np.array_equal(heaps[FUSED], heaps[v]), VNAMES[v]


def test_large_bf16_224_wide_tiles_match_oracle():
    """256 x 224 tiles give the 4096 x 3584 output exactly 256 tiles; every
    schedule matches the oracle and the three leave identical heaps."""
    wl = workload.LARGE_BF16
    p = Problem(wl.world, wl.M, wl.N_local, wl.K, wl.dtype, 256, 224, dist=wl.dist, seed=6)
    assert p.out.tiles_n == 16 and p.out.tiles_m == 16
    want = {3: oracle_block(p.A, p.shards[3], wl.dtype)}
    heaps = {}
    for v in (FUSED, WGSPEC, BULK, UNFUSED):
        p.sentinel()
        p.run(3, v)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[3]))
        heaps[v] = u16(p.out.C(0))[:, 3 * wl.N_local:4 * wl.N_local].copy()
    for v in (WGSPEC, BULK, UNFUSED):
        assert np.array_equal(heaps[FUSED], heaps[v]), VNAMES[v]


def test_large_bf16_wg_spec_split_sweep_bitwise():
    wl = workload.LARGE_BF16
    pkg = sym()
    cus, limit = pkg.symtile_device_info(0, wl.tile_m, wl.tile_n)
    p = _large_case(wl, seed=2)
    p.sentinel()
    p.run(0, FUSED)
    p.barrier()
    ref = u16(p.out.C(0))[:, :wl.N_local].copy()
    check_block(ref, oracle_block(p.A, p.shards[0], wl.dtype), wl.dtype, "fused reference")
    for copy_wgs in (8, 16, 32, 48, 64):
        gemm_wgs = min(limit, cus) - copy_wgs
        p.sentinel()
        p.run(0, WGSPEC, gemm_wgs=gemm_wgs, copy_wgs=copy_wgs)
        p.barrier()
        G = u16(p.out.C_all())
        for s in range(wl.world):
            assert np.array_equal(G[s][:, :wl.N_local], ref), (copy_wgs, s)
            assert np.all(G[s][:, wl.N_local:] == SENTINEL), (copy_wgs, s)
    arr = p.out.arrived_all().cpu().numpy()
    assert np.all(arr[:, 0] == int(p.calls[0])) and np.all(arr[:, 1:] == 0)


def test_nontemporal_and_group_m_do_not_change_bits():
    wl = workload.SMALL_BF16
    p = _large_case(wl, seed=4)
    outs = []
    for nt, gm in ((0, 0), (1, 0), (0, 1), (1, 8)):
        p.sentinel()
        p.run(0, FUSED, nontemporal=nt, group_m=gm)
        p.barrier()
        outs.append(u16(p.out.C_all()).copy())
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


# ---------------------------------------------------------------- epochs and failures

def test_repeated_wg_spec_epochs_see_fresh_data():
    wl = workload.SMALL_BF16
    p = _large_case(wl, seed=6)
    want = {0: oracle_block(p.A, p.shards[0], wl.dtype)}
    for epoch in range(1, 4):
        p.sentinel()
        p.run(0, WGSPEC, copy_wgs=24)
        p.barrier()
        check_gathered(p, want)                     # counters == epoch, data complete
        assert p.out.ready.cpu().numpy().min() == epoch


def test_unfused_two_streams_split_sweep_and_epochs():
    """Unfused producer-consumer (Section 4.1.2): GEMM grid and copy grid on
    two streams partition the CUs; every split, with the heap's own copy
    stream or a caller's, leaves the heap bitwise equal to the fused kernel's,
    and repeated calls advance the ready counters one epoch each."""
    wl = workload.LARGE_BF16
    pkg = sym()
    cus, _ = pkg.symtile_device_info(0, wl.tile_m, wl.tile_n)
    p = _large_case(wl, seed=9)
    p.sentinel()
    p.run(0, FUSED)
    p.barrier()
    ref = u16(p.out.C_all()).copy()
    check_block(ref[0][:, :wl.N_local], oracle_block(p.A, p.shards[0], wl.dtype), wl.dtype,
                "fused reference")
    side = torch.cuda.Stream()
    for i, copy_wgs in enumerate((8, 32, 64)):
        p.sentinel()
        p.run(0, UNFUSED, gemm_wgs=cus - copy_wgs, copy_wgs=copy_wgs,
              copy_stream=side.cuda_stream if i == 1 else None)
        p.barrier()
        assert np.array_equal(u16(p.out.C_all()), ref), copy_wgs
        assert p.out.ready.cpu().numpy().min() == i + 1
    arr = p.out.arrived_all().cpu().numpy()
    assert np.all(arr[:, 0] == int(p.calls[0])) and np.all(arr[:, 1:] == 0)


def test_unfused_argument_errors():
    pkg = sym()
    p = Problem(2, 128, 128, 64, "f16", 64, 64, seed=7)
    cus, _ = pkg.symtile_device_info(0, 64, 64)
    with pytest.raises(pkg.SymtileError) as e:                 # grids exceed the CUs
        p.out.run(p.dA, p.dB[0], 0, UNFUSED, gemm_wgs=cus, copy_wgs=1)
    assert e.value.name == "EUNSUPPORTED"
    s = torch.cuda.Stream().cuda_stream                         # a non-default stream
    with pytest.raises(pkg.SymtileError) as e:                 # copy stream = call stream
        p.out.run(p.dA, p.dB[0], 0, UNFUSED, copy_stream=s, stream=s)
    assert e.value.name == "EINVAL"
    p.heap.barrier()


def test_unfused_consumer_timeout_is_reported_not_hung():
    pkg = sym()
    p = Problem(2, 128, 128, 64, "f16", 64, 64, seed=7)
    p.out.ready_epoch = 5                   # the copy kernel waits for 6; producers bring 1
    p.run(0, UNFUSED, spin_limit=2000)
    with pytest.raises(pkg.SymtileError) as e:
        p.heap.barrier()
    assert e.value.name == "ETIMEOUT"
    p.heap.barrier()


def test_consumer_timeout_is_reported_not_hung():
    """Consumers told to wait for an epoch the producers never reach give up
    after spin_limit polls; the error surfaces at the barrier."""
    pkg = sym()
    p = Problem(2, 128, 128, 64, "f16", 64, 64, seed=7)
    p.out.ready_epoch = 5                   # next call waits for ready >= 6; producers bring 1
    p.run(0, WGSPEC, spin_limit=2000)
    with pytest.raises(pkg.SymtileError) as e:
        p.heap.barrier()
    assert e.value.name == "ETIMEOUT"
    p.heap.barrier()                        # the error word was cleared


def test_argument_errors():
    pkg = sym()
    p = Problem(2, 128, 64, 64, "bf16", 64, 64)
    h = p.heap.handle
    cfg = pkg.GasConfig(variant=FUSED, tile_m=64, tile_n=64)
    c_other = p.heap.ptr(1, p.out.c_off)            # C in the wrong slot for rank 0
    args = dict(A=p.dA.data_ptr(), B=p.dB[0].data_ptr())

    def call(C, flags, M=128, N=64, K=64, rank=0, world=2, cfg=cfg, dtype=pkg.BF16):
        pkg.symtile_gemm_all_scatter(h, args["A"], args["B"], C, flags, p.out.ready.data_ptr(),
                                     M, N, K, K, N, dtype, rank, world, cfg, 0)

    c0, f0 = p.heap.ptr(0, p.out.c_off), p.heap.ptr(0, p.out.flag_off)
    for bad in (dict(C=c_other, flags=f0), dict(C=c0, flags=f0, K=60),
                dict(C=c0, flags=f0, rank=2), dict(C=c0, flags=f0, world=3),
                dict(C=c0, flags=f0, M=100000),
                # maximum sizes: 32-bit buffer offsets; B of 2 GiB, a 64-row band of the
                # gathered C of 2 GiB (rejected before any memory is touched)
                dict(C=c0, flags=f0, K=1 << 20, N=1024),
                dict(C=c0, flags=f0, N=1 << 23)):
        with pytest.raises(pkg.SymtileError) as e:
            call(**bad)
        assert e.value.name == "EINVAL", bad
    with pytest.raises(pkg.SymtileError) as e:
        call(c0, f0, cfg=pkg.GasConfig(variant=FUSED, tile_m=32, tile_n=32))
    assert e.value.name == "EUNSUPPORTED"
    with pytest.raises(pkg.SymtileError) as e:
        call(c0, f0, cfg=pkg.GasConfig(variant=WGSPEC, tile_m=64, tile_n=64,
                                       gemm_wgs=100000, copy_wgs=8))
    assert e.value.name == "EUNSUPPORTED"
    with pytest.raises(pkg.SymtileError) as e:
        call(c0, f0, dtype=pkg.F32)
    assert e.value.name == "EUNSUPPORTED"
    with pytest.raises(pkg.SymtileError) as e:           # 256x224 is built with 8 waves only
        call(c0, f0, cfg=pkg.GasConfig(variant=FUSED, tile_m=256, tile_n=224, waves_per_wg=4))
    assert e.value.name == "EUNSUPPORTED"
    p.heap.barrier()


def test_padded_strides_on_tightly_sized_buffers():
    """lda > K and ldb > N_local through the C ABI, with A and B in buffers
    that end exactly at their last element and NaN in every padding element:
    the padding is never read into a stored value (any NaN would show), and
    the result matches the oracle."""
    pkg = sym()
    world, rank, M, N, K, lda, ldb = 3, 1, 300, 136, 200, 264, 200
    # (256 x 256 with both wave counts: 4 waves stage 64 k through registers)
    for tm, tn, waves in ((128, 128, 0), (256, 256, 4), (256, 256, 8), (64, 64, 0)):
        p = Problem(world, M, N, K, "bf16", tm, tn, seed=21)
        bf = torch.bfloat16
        a_buf = torch.full(((M - 1) * lda + K,), float("nan"), dtype=bf, device="cuda")
        b_buf = torch.full(((K - 1) * ldb + N,), float("nan"), dtype=bf, device="cuda")
        a_buf.as_strided((M, K), (lda, 1)).copy_(p.dA)
        b_buf.as_strided((K, N), (ldb, 1)).copy_(p.dB[rank])
        p.sentinel()
        for variant in (FUSED, BULK):
            pkg.symtile_gemm_all_scatter(
                p.heap.handle, a_buf.data_ptr(), b_buf.data_ptr(), p.heap.ptr(rank, p.out.c_off),
                p.heap.ptr(rank, p.out.flag_off), p.out.ready.data_ptr(), M, N, K, lda, ldb,
                pkg.BF16, rank, world,
                pkg.GasConfig(variant=variant, tile_m=tm, tile_n=tn, waves_per_wg=waves),
                pkg.current_stream())
            p.calls[rank] += 1
            p.barrier()
            check_gathered(p, {rank: oracle_block_bounded(p.A, p.shards[rank], "bf16")})


@pytest.mark.parametrize("mode,again", [(1, 1), (2, 2), (1, 3), (2, 3)],
                         ids=["last", "banded", "last_then_kernel", "banded_then_kernel"])
def test_split_k_timeout_then_stale_workspace_is_reported(mode, again):
    """A slice allowed one poll gives up on the tiles whose partner partial
    is not yet counted (ETIMEOUT at the barrier) and leaves their counters as
    they are (last-arriver reduction: the two tickets; banded: the two first
    tickets plus the second ticket of a slice that went on).  A later call on
    the same workspace, made without zeroing it, reports the stale counters
    (EINVAL at the barrier): the ticketed reductions write no stale sum; the
    reduction kernel (whose partials are all this call's) stores the tiles
    but publishes none of the stale ones.  The Python wrapper zeroes the
    workspace after either report, and its next call is exact."""
    pkg = sym()
    world, rank = 2, 0
    p = Problem(world, 1024, 512, 2048, "bf16", 64, 64, seed=17)     # 128 tiles x 2 slices
    want = {rank: oracle_block_bounded(p.A, p.shards[rank], "bf16")}
    stale_ok = (0, 2) if mode == 1 else (0, 2, 3)
    p.sentinel()
    p.run(rank, FUSED, split_k=2, spin_limit=1, split_reduce=mode)
    try:
        p.heap.barrier()
        timed_out = False
    except pkg.SymtileError as e:
        assert e.name == "ETIMEOUT", e
        timed_out = True
    torch.cuda.synchronize()
    if not timed_out:                        # every partner was early: an ordinary call
        check_gathered(p, want)
        assert np.all(_ws_counters(p) == 0)
    else:
        stale = _ws_counters(p).reshape(-1, 2)
        assert np.any(stale[:, 0] != 0)      # tickets left behind by the timed-out tiles
        assert np.all(np.isin(stale[:, 0], stale_ok)), np.unique(stale[:, 0])
        # the same workspace again, through the C ABI (no reset)
        ws = p.out.ws
        p.out.C_all().view(torch.int16).fill_(-1)
        flags0 = p.out.arrived_all().cpu().numpy().copy()
        pkg.symtile_gemm_all_scatter(
            p.heap.handle, p.dA.data_ptr(), p.dB[rank].data_ptr(), p.heap.ptr(rank, p.out.c_off),
            p.heap.ptr(rank, p.out.flag_off), p.out.ready.data_ptr(), p.M, p.N, p.K, p.K, p.N,
            pkg.BF16, rank, world,
            pkg.GasConfig(variant=FUSED, tile_m=64, tile_n=64, split_k=2,
                          workspace=ws.data_ptr(), workspace_bytes=ws.numel(),
                          split_reduce=again),
            pkg.current_stream())
        with pytest.raises(pkg.SymtileError) as e:
            p.heap.barrier()
        assert e.value.name == "EINVAL" and "workspace" in str(e.value)
        torch.cuda.synchronize()
        G = u16(p.out.C_all())[0][:, :p.N].reshape(16, 64, 8, 64)
        bad = (stale != 0).any(axis=1).reshape(16, 8)
        tm, tn = np.nonzero(bad)
        if again != 3:
            for m, n in zip(tm, tn):         # a stale tile is left unwritten
                assert np.all(G[m, :, n, :] == SENTINEL), (m, n)
        else:
            # every tile stored, exact; the stale ones unpublished in every slot
            check_block(G.reshape(p.M, p.N), want[rank], "bf16")
            d = p.out.arrived_all().cpu().numpy() - flags0      # [slot, rank, tm, tn]
            assert np.all(d[:, rank][:, bad] == 0)
            assert np.all(d[:, rank][:, ~bad] == 1)
    # the wrapper zeroes the workspace after a failed barrier: exact again
    p.sentinel()
    p.calls[:] = 0
    p.out.arrived_all().zero_()
    p.run(rank, FUSED, split_k=2, split_reduce=mode)
    p.barrier()
    check_gathered(p, want)
    assert np.all(_ws_counters(p) == 0)


@pytest.mark.parametrize("case", [(8, 1024, 1024, 4096, 256, 128, "bf16"),
                                  (8, 1024, 1024, 4096, 256, 256, "bf16"),
                                  (3, 300, 264, 200, 256, 256, "f16"),
                                  (2, 520, 264, 72, 256, 256, "bf16"),
                                  (3, 300, 264, 200, 256, 128, "f16"),
                                  (2, 512, 256, 320, 256, 128, "bf16"),
                                  (4, 300, 264, 200, 128, 128, "bf16"),
                                  (8, 1024, 1024, 4096, 128, 128, "f16")],
                         ids=lambda c: "w%d_m%d_n%d_k%d_t%dx%d_%s" % c)
def test_four_and_eight_wave_kernels_agree_bitwise(case):
    """Both wave layouts compute each accumulator in the same order, so the
    heaps they leave are identical; both match the oracle."""
    world, M, N, K, tm, tn, dtype = case
    p = Problem(world, M, N, K, dtype, tm, tn, seed=5)
    want = {1 % world: oracle_block(p.A, p.shards[1 % world], dtype)}
    heaps = []
    for waves in (4, 8):
        p.sentinel()
        p.run(1 % world, FUSED, waves_per_wg=waves)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[1 % world]))
        heaps.append(u16(p.out.C_all()).copy())
    assert np.array_equal(heaps[0], heaps[1])


@pytest.mark.parametrize("split", [2, 3])
def test_four_wave_256_split_k_matches_eight_waves_bitwise(split):
    """256 x 256 tiles with 4 waves stage 64 k at a time; K slices of an odd
    number of 32-k stages end inside such a stage, whose k past the slice
    must read zero.  The sums agree bit for bit with the 8-wave kernel's."""
    world, M, N, K = 4, 512, 520, 4000 + 96
    p = Problem(world, M, N, K, "bf16", 256, 256, seed=11)
    want = {2: oracle_block(p.A, p.shards[2], "bf16")}
    heaps = []
    for waves in (4, 8):
        p.sentinel()
        p.run(2, FUSED, waves_per_wg=waves, split_k=split)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[2]))
        heaps.append(u16(p.out.C_all()).copy())
        assert np.all(_ws_counters(p) == 0)
    assert np.array_equal(heaps[0], heaps[1])


# ---------------------------------------------------------------- trace

@pytest.mark.parametrize("variant", VARIANTS, ids=VNAMES.get)
def test_trace_records_every_tile_in_causal_order(variant):
    """Per-tile timeline: every tile has its producer events in order; a
    WG_SPEC consumer acquires only after the producer's stores were
    acknowledged; the bulk copy kernel starts after every producer released.
    Tracing does not change the results."""
    from paper_2511_12500_amd import trace as T
    world, rank = 4, 1
    p = Problem(world, 600, 520, 264, "bf16", 128, 128, seed=7)
    want = {rank: oracle_block(p.A, p.shards[rank], "bf16")}
    tr = p.out.new_trace()
    p.sentinel()
    p.run(rank, variant, trace=tr)
    p.barrier()
    check_gathered(p, want)
    raw = tr.cpu().numpy().view(np.uint64)
    assert raw.shape == (p.out.tiles_m * p.out.tiles_n, T.WORDS)
    prod = raw[:, [T.START, T.MAINLOOP, T.STORED, T.RELEASED]]
    assert np.all(prod > 0)
    assert np.all(np.diff(prod.astype(np.int64), axis=1) >= 0)
    where = raw[:, T.WHERE]
    assert np.all((where & np.uint64(0xFFFF)) < 1024)                 # workgroup id
    assert np.all(((where >> np.uint64(16)) & np.uint64(0xFFFF)) < 8)  # XCC id
    copy = raw[:, [T.COPY_WAIT, T.COPY_GO, T.COPY_DONE]].astype(np.int64)
    if variant == FUSED:
        assert np.all(copy == 0)
    else:
        assert np.all(copy > 0) and np.all(np.diff(copy, axis=1) >= 0)
        if variant in (WGSPEC, UNFUSED):
            assert np.all(copy[:, 1] >= raw[:, T.STORED].astype(np.int64))
        else:
            assert copy[:, 0].min() >= raw[:, T.RELEASED].astype(np.int64).max()
    khz = sym().symtile_clock_rate_khz(0)
    t = T.decode(raw, khz)
    s = T.summary(t)
    assert s["tiles"] == raw.shape[0] and s["span_us"] > 0


# ---------------------------------------------------------------- wave specialisation

WAVESPEC = 4


@pytest.mark.parametrize("case", [
    # world, M, N_local, K, gemm_wgs, dtype
    (8, 1024, 1024, 4096, 8, "bf16"),      # 32 tiles, 4 per workgroup
    (4, 600, 520, 264, 3, "bf16"),         # ragged rows, columns and K; 5 tiles each
    (2, 257, 136, 72, 1, "f16"),           # one workgroup, every tile through the copy wave
], ids=lambda c: "w%d_m%d_n%d_k%d_g%d_%s" % c)
def test_wave_spec_matches_fused_bitwise(case):
    """Section 4.2.3: compute waves store each tile locally and one extra wave
    copies the previous tile to the other slots during the next K loop; the
    heap equals the fused kernel's bit for bit and matches the oracle."""
    world, M, N, K, g, dtype = case
    p = Problem(world, M, N, K, dtype, 256, 128, seed=11)
    r = world - 1
    want = {r: oracle_block(p.A, p.shards[r], dtype)}
    p.sentinel()
    p.run(r, FUSED, gemm_wgs=g)
    p.barrier()
    ref = u16(p.out.C_all()).copy()
    p.sentinel()
    tr = p.out.new_trace()
    p.run(r, WAVESPEC, gemm_wgs=g, trace=tr)
    p.barrier()
    check_gathered(p, want)
    assert np.array_equal(u16(p.out.C_all()), ref)
    from paper_2511_12500_amd import trace as T
    raw = tr.cpu().numpy().view(np.uint64).astype(np.int64)
    copied = raw[:, T.COPY_DONE] > 0
    # every workgroup's last tile is stored everywhere by its compute waves
    assert int(copied.sum()) == raw.shape[0] - min(g, raw.shape[0])
    assert np.all(raw[copied, T.COPY_GO] >= raw[copied, T.STORED])
    assert np.all(raw[copied, T.COPY_DONE] >= raw[copied, T.COPY_GO])


def test_wave_spec_large_and_k_zero():
    wl = workload.LARGE_BF16
    p = Problem(wl.world, wl.M, wl.N_local, wl.K, wl.dtype, 256, 128, dist=wl.dist, seed=12)
    want = {0: oracle_block(p.A, p.shards[0], wl.dtype)}
    p.sentinel()
    p.run(0, WAVESPEC, gemm_wgs=112)            # 448 tiles, 4 per workgroup
    p.barrier()
    check_gathered(p, want)
    z = Problem(2, 300, 136, 0, "bf16", 256, 128, A=torch.zeros(300, 0, dtype=torch.bfloat16),
                shards=[torch.zeros(0, 136, dtype=torch.bfloat16)] * 2)
    z.sentinel()
    z.run(1, WAVESPEC, gemm_wgs=1)
    z.barrier()
    G = u16(z.out.C_all())
    assert np.all(G[:, :, 136:] == 0) and np.all(G[:, :, :136] == SENTINEL)
    assert np.all(z.out.arrived_all().cpu().numpy()[:, 1] == 1)


def test_wave_spec_other_tiles_unsupported():
    pkg = sym()
    p = Problem(2, 128, 128, 64, "bf16", 128, 128, seed=7)
    with pytest.raises(pkg.SymtileError) as e:
        p.run(0, WAVESPEC)
    assert e.value.name == "EUNSUPPORTED"
    p.heap.barrier()


# ---------------------------------------------------------------- split-K

SPLITK = [
    # world, M, N_local, K, tile_m, tile_n, dtype, split_k
    (2, 300, 136, 520, 128, 128, "bf16", 2),     # ragged M, N; 17 stages split 8 + 9
    (3, 257, 264, 1000, 256, 256, "f16", 3),     # 32 stages 10/11/11, last stage 8 of 32 k
    (4, 130, 264, 72, 256, 128, "bf16", 3),      # one stage per slice, the last ragged
    (5, 77, 40, 200, 64, 64, "f16", 7),          # one stage per slice, 7 slices
    (8, 64, 8, 64, 64, 64, "bf16", 2),           # one tile, 8 columns
    (3, 300, 504, 200, 256, 224, "bf16", 2),     # 16x16x32 MFMA tile shape
    (2, 512, 512, 2048, 256, 256, "bf16", 8),    # 8 slices of 8 stages
]


def _ws_counters(p):
    n = 2 * p.out.tiles_m * p.out.tiles_n
    return p.out.ws[:n * 4].view(torch.int32).cpu().numpy()


@pytest.mark.parametrize("case", SPLITK, ids=lambda c: "w%d_m%d_n%d_k%d_t%dx%d_%s_s%d" % c)
@pytest.mark.parametrize("variant", [FUSED, BULK], ids=VNAMES.get)
def test_split_k_all_ranks(case, variant):
    """Each tile as split_k slices of K: placement and counters bit-exact,
    values within tolerance, and the workspace counters back at zero."""
    world, M, N, K, tm, tn, dtype, split = case
    p = Problem(world, M, N, K, dtype, tm, tn, seed=11)
    want = _blocks(p)
    p.sentinel()
    for i, r in enumerate(reversed(range(world))):
        p.run(r, variant, split_k=split)
        if i == 0:
            p.barrier()
            check_gathered(p, want)
            assert np.all(_ws_counters(p) == 0)
    p.barrier()
    check_gathered(p, want)
    assert np.all(_ws_counters(p) == 0)


@pytest.mark.parametrize("split", [2, 3, 5])
@pytest.mark.parametrize("mode", [0, 1], ids=["auto", "last"])
def test_split_k_is_deterministic_across_grids(split, mode):
    """The slices add their partials in slice order, so neither the grid size
    (how many slices run at once, and which finishes last; down to one
    workgroup for the last-slice reduction, which assumes no co-residency)
    nor a repeated call changes a bit."""
    world, rank = 4, 2
    p = Problem(world, 520, 392, 1544, "bf16", 128, 128, seed=12)
    want = {rank: oracle_block(p.A, p.shards[rank], "bf16")}
    units = p.out.tiles_m * p.out.tiles_n * split
    ref = None
    for g in (0, units, 7, 1, 0):
        p.sentinel()
        p.run(rank, FUSED, split_k=split, gemm_wgs=g, split_reduce=mode)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[rank]))
        got = u16(p.out.C_all())
        if ref is None:
            ref = got.copy()
        assert np.array_equal(got, ref), g
        assert np.all(_ws_counters(p) == 0)


BANDED = [
    # world, M, N_local, K, tile_m, tile_n, dtype, split_k
    (2, 300, 136, 520, 128, 128, "bf16", 2),     # ragged M, N; two 64-row bands
    (3, 1000, 520, 1000, 128, 128, "f16", 4),    # 32-row bands; the last tile row ragged
    (4, 130, 264, 520, 256, 256, "bf16", 8),     # large accumulators: own rows via memory
    (3, 300, 504, 200, 256, 224, "bf16", 2),     # 16x16x32 MFMA tile, 128-row bands
    (2, 200, 72, 96, 64, 64, "f16", 2),          # 64x64 tile (4 waves), 32-row bands
    (2, 512, 512, 2048, 256, 256, "f16", 2),     # large accumulators, two slices
]


@pytest.mark.parametrize("case", BANDED, ids=lambda c: "w%d_m%d_n%d_k%d_t%dx%d_%s_s%d" % c)
def test_banded_split_reduce_matches_last_arriver_bitwise(case):
    """The banded reduction (slice s sums and stores band s of the tile) and
    the last-arriver reduction form the same slice-order sums: heaps equal
    bit for bit, both against the oracle with the accumulation bound,
    counters exact, workspace counters back at zero."""
    pkg = sym()
    world, M, N, K, tm, tn, dtype, split = case
    rank = world - 1
    p = Problem(world, M, N, K, dtype, tm, tn, seed=21)
    want = {rank: oracle_block_bounded(p.A, p.shards[rank], dtype)}
    heaps = {}
    for mode in (pkg.SPLIT_REDUCE_LAST, pkg.SPLIT_REDUCE_BANDED, pkg.SPLIT_REDUCE_BANDED):
        p.sentinel()
        p.run(rank, FUSED, split_k=split, split_reduce=mode)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[rank]))
        assert np.all(_ws_counters(p) == 0), mode
        got = u16(p.out.C_all())
        if heaps:
            assert np.array_equal(got, next(iter(heaps.values()))), mode
        heaps[mode] = got


@pytest.mark.parametrize("case", SPLITK + BANDED[1:3] + [
    (2, 2048, 2048, 96, 64, 64, "f16", 3),     # 1024 tiles: reduction units past the CU count
], ids=lambda c: "w%d_m%d_n%d_k%d_t%dx%d_%s_s%d" % c)
@pytest.mark.parametrize("variant", [FUSED, BULK], ids=VNAMES.get)
def test_reduction_kernel_matches_last_arriver_bitwise(case, variant):
    """The reduction-kernel mode (every slice writes its partial, a second
    kernel sums each tile's bands in slice order and stores them) gives the
    last-arriver reduction's bits, at the default grid and at grids of 7 and
    1 workgroups for the first kernel; against the oracle with the
    accumulation bound, counters exact, workspace counters back at zero."""
    pkg = sym()
    world, M, N, K, tm, tn, dtype, split = case
    rank = world // 2
    p = Problem(world, M, N, K, dtype, tm, tn, seed=23)
    want = {rank: oracle_block_bounded(p.A, p.shards[rank], dtype)}
    ref = None
    for mode, g in ((pkg.SPLIT_REDUCE_LAST, 0), (pkg.SPLIT_REDUCE_KERNEL, 0),
                    (pkg.SPLIT_REDUCE_KERNEL, 7), (pkg.SPLIT_REDUCE_KERNEL, 1)):
        p.sentinel()
        p.run(rank, variant, split_k=split, split_reduce=mode, gemm_wgs=g)
        p.barrier()
        check_gathered(p, want, flag_count=int(p.calls[rank]))
        assert np.all(_ws_counters(p) == 0), (mode, g)
        got = u16(p.out.C_all())
        if ref is None:
            ref = got
        assert np.array_equal(got, ref), (mode, g)


def test_banded_split_reduce_argument_errors():
    """BANDED needs one resident workgroup per slice and whole bands;
    otherwise EUNSUPPORTED (AUTO falls back to the last-arriver reduction)."""
    pkg = sym()
    p = Problem(2, 300, 136, 520, "bf16", 128, 128, seed=22)
    for kw in (dict(split_k=3), dict(split_k=2, gemm_wgs=5), dict(split_k=8)):
        with pytest.raises(pkg.SymtileError, match="EUNSUPPORTED"):
            p.out.run(p.dA, p.dB[0], 0, FUSED, split_reduce=pkg.SPLIT_REDUCE_BANDED, **kw)
    with pytest.raises(pkg.SymtileError, match="EINVAL"):
        p.out.run(p.dA, p.dB[0], 0, FUSED, split_k=2, split_reduce=4)
    want = {0: oracle_block(p.A, p.shards[0], "bf16")}
    p.sentinel()
    p.run(0, FUSED, split_k=3)                     # AUTO: 128 rows do not split in 3 bands
    p.barrier()
    check_gathered(p, want)


def test_split_k_two_slices_match_one_within_rounding():
    """split_k = 2 changes only the fp32 summation order: against the
    unsplit call, at most a rounding step of the output in any element."""
    world, rank = 2, 0
    p = Problem(world, 512, 256, 4096, "bf16", 256, 256, seed=13, dist="normal_sqrtk")
    p.sentinel()
    p.run(rank, FUSED)
    p.barrier()
    one = p.out.C(0)[:, :256].float().cpu()
    p.run(rank, FUSED, split_k=2)
    p.barrier()
    two = p.out.C(0)[:, :256].float().cpu()
    # one bf16 step of the larger value, plus the fp32 reordering error near
    # zero (about sqrt(K) * 2^-24 * |C|, far below this floor)
    step = torch.maximum(one.abs(), two.abs()) * 2.0 ** -7 + one.abs().max() * 2.0 ** -16
    assert bool((torch.abs(one - two) <= step).all())
    check_block(u16(p.out.C(0)[:, :256]), oracle_block(p.A, p.shards[0], "bf16"), "bf16")


@pytest.mark.parametrize("wl,tile,split",
                         [(workload.WIDE_F16, 256, 2), (workload.SMALL_BF16, 256, 16),
                          (workload.SMALL_BF16, 128, 4)],
                         ids=lambda x: getattr(x, "name", str(x)))
def test_split_k_full_size_matches_oracle(wl, tile, split):
    """The full-size shapes with few tiles, split so every CU has a slice:
    fp16 8192x8192.8192x1024 with 256x256 tiles in 2 slices and bf16
    1024x4096.4096x1024 with 128x128 tiles (8 waves) in 4 slices, the
    configurations the benchmark runs, and the latter with 256x256 tiles in
    16 slices."""
    p = Problem(wl.world, wl.M, wl.N_local, wl.K, wl.dtype, tile, tile, dist=wl.dist, seed=4)
    want = {0: (oracle_block_bounded if wl.M * wl.N_local <= 1 << 22 else oracle_block)(
        p.A, p.shards[0], wl.dtype)}
    p.sentinel()
    p.run(0, FUSED, split_k=split, nontemporal=2)
    p.barrier()
    check_gathered(p, want, flag_count=1)
    assert np.all(_ws_counters(p) == 0)


@pytest.mark.parametrize("mode", [1, 3], ids=["last", "kernel"])
def test_split_k_trace_is_causal(mode):
    """With split-K the start and main-loop words are slice 0's and the
    stored and released words the reducing slice's (or the last band of the
    reduction kernel); still in order."""
    from paper_2511_12500_amd import trace as T
    world, rank = 4, 1
    p = Problem(world, 600, 520, 264, "bf16", 128, 128, seed=7)
    want = {rank: oracle_block(p.A, p.shards[rank], "bf16")}
    tr = p.out.new_trace()
    p.sentinel()
    p.run(rank, FUSED, trace=tr, split_k=3, split_reduce=mode)
    p.barrier()
    check_gathered(p, want)
    raw = tr.cpu().numpy().view(np.uint64)
    prod = raw[:, [T.START, T.MAINLOOP, T.STORED, T.RELEASED]]
    assert np.all(prod > 0)
    assert np.all(np.diff(prod.astype(np.int64), axis=1) >= 0)


def test_split_k_argument_errors():
    pkg = sym()
    p = Problem(2, 128, 64, 256, "bf16", 64, 64)
    h = p.heap.handle
    c0, f0 = p.heap.ptr(0, p.out.c_off), p.heap.ptr(0, p.out.flag_off)
    ws = p.out.workspace(2)
    need = pkg.symtile_gas_workspace_bytes(128, 64, 64, 64, 2)
    assert ws.numel() == need == 256 + 2 * 2 * 64 * 64 * 4       # 2 tiles of 64x64

    def call(**kw):
        base = dict(variant=FUSED, tile_m=64, tile_n=64, split_k=2, workspace=ws.data_ptr(),
                    workspace_bytes=need)
        base.update(kw)
        K = base.pop("K", 256)
        pkg.symtile_gemm_all_scatter(h, p.dA.data_ptr(), p.dB[0].data_ptr(), c0, f0,
                                     p.out.ready.data_ptr(), 128, 64, K, 256, 64, pkg.BF16, 0, 2,
                                     pkg.GasConfig(**base), 0)

    for kw, name in ((dict(variant=WGSPEC, gemm_wgs=8, copy_wgs=8), "EUNSUPPORTED"),
                     (dict(variant=UNFUSED), "EUNSUPPORTED"),
                     (dict(variant=WAVESPEC), "EUNSUPPORTED"),
                     (dict(split_k=65), "EINVAL"),
                     (dict(split_k=-1), "EINVAL"),
                     (dict(split_k=9), "EINVAL"),                   # K = 256 has 8 stages
                     (dict(workspace=None), "EINVAL"),
                     (dict(workspace_bytes=need - 1), "EINVAL"),
                     (dict(workspace=ws.data_ptr() + 8), "EINVAL"),  # misaligned
                     (dict(workspace=c0, workspace_bytes=1 << 20), "EINVAL")):   # overlaps C
        with pytest.raises(pkg.SymtileError) as e:
            call(**kw)
        assert e.value.name == name, kw
    p.out.reset_workspace()
    p.sentinel()
    p.run(0, FUSED, split_k=8)                                        # 8 stages: allowed
    p.barrier()
    check_gathered(p, {0: oracle_block(p.A, p.shards[0], "bf16")})
    assert np.all(_ws_counters(p) == 0)


# ---------------------------------------------------------------- seeded random sweep

def _random_cases(n=64, seed=2027):
    """Seeded draws over world size, shape (ragged M, N, K), tile, wave count,
    schedule, split-K, dtype and rank; each is a valid call."""
    rng = np.random.RandomState(seed)
    tiles = [(64, 64), (128, 128), (256, 128), (256, 256), (256, 224)]
    cases = []
    for _ in range(n):
        world = int(rng.randint(1, 9))
        tm, tn = tiles[rng.randint(len(tiles))]
        M = int(rng.randint(1, 700))
        N = 8 * int(rng.randint(1, 76))
        K = 8 * int(rng.randint(1, 151))
        dtype = ("bf16", "f16")[rng.randint(2)]
        variants = [BULK, FUSED, WGSPEC, UNFUSED] + ([WAVESPEC] if (tm, tn) == (256, 128) else [])
        variant = variants[rng.randint(len(variants))]
        waves = 0
        if (tm, tn) in ((256, 128), (256, 256)) and variant != WAVESPEC and rng.rand() < 0.3:
            waves = 4 if (tm, tn) == (256, 128) else 0   # 256x256 is built with 8 waves only
        split = 0
        stages = -(-K // 32)
        if variant in (BULK, FUSED) and stages > 1 and rng.rand() < 0.5:
            split = min(stages, (2, 2, 3, 4, 6)[rng.randint(5)])
        rank = int(rng.randint(world))
        cases.append((world, M, N, K, tm, tn, dtype, variant, waves, split, rank))
    return cases


@pytest.mark.parametrize("case", _random_cases(),
                         ids=lambda c: "w%d_m%d_n%d_k%d_t%dx%d_%s_v%d_wv%d_s%d_r%d" % c)
def test_random_calls_match_oracle(case):
    world, M, N, K, tm, tn, dtype, variant, waves, split, rank = case
    p = Problem(world, M, N, K, dtype, tm, tn, seed=M + N + K)
    want = {rank: oracle_block_bounded(p.A, p.shards[rank], dtype)}
    p.sentinel()
    p.run(rank, variant, waves_per_wg=waves, split_k=split)
    p.barrier()
    check_gathered(p, want)
    if split > 1:
        assert np.all(_ws_counters(p) == 0)
