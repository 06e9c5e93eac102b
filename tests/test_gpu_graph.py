"""GPU tests: GEMM + All-Scatter calls captured in a HIP graph
(torch.cuda.graph) and replayed.

The calls launch on the caller's stream with nothing but kernel launches
(split-K: one or two kernels; the bulk-synchronous schedule: two), so a
capture records them and every replay repeats them: placement and values
as the oracle gives them after each replay, the arrival counters one higher
per replay, the split-K workspace counters back at zero, and the heap equal
bit for bit to that of eager calls.  Between replays the program runs eager
work of its own (refilling the output with the sentinel), as a caller would.
The WG-specialised and unfused schedules bake the epoch their consumers
wait for into the launch, so they are not replayable as captured and are
not covered here."""
import numpy as np
import pytest
import torch

from tests.gpu_util import Problem, check_gathered, oracle_block_bounded, require_gpu, u16

pytestmark = pytest.mark.gpu

BULK, FUSED, WAVESPEC = 0, 1, 4
VNAMES = {BULK: "bulk", FUSED: "fused", WAVESPEC: "wavespec"}


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


CASES = [
    # world, M, N_local, K, dtype, tile, variant, split_k, split_reduce
    (2, 128, 64, 256, "f16", (64, 64), FUSED, 0, 0),        # the tiny two-rank workload
    (4, 300, 136, 520, "bf16", (128, 128), BULK, 0, 0),     # two kernels per call
    (3, 300, 264, 1000, "bf16", (128, 128), FUSED, 4, 3),   # split-K, reduction kernel
    (3, 300, 264, 1000, "f16", (128, 128), FUSED, 3, 1),    # split-K, last slice
    (2, 300, 136, 520, "bf16", (128, 128), FUSED, 2, 2),    # split-K, banded
    (4, 513, 264, 200, "bf16", (256, 128), WAVESPEC, 0, 0),  # copy wave
]


def _ws_counters(p):
    n = 2 * p.out.tiles_m * p.out.tiles_n
    return p.out.ws[:n * 4].view(torch.int32).cpu().numpy()


@pytest.mark.parametrize(
    "case", CASES,
    ids=lambda c: "w%d_m%d_n%d_k%d_%s_t%dx%d_%s_s%d_r%d" % (
        c[0], c[1], c[2], c[3], c[4], c[5][0], c[5][1], VNAMES[c[6]], c[7], c[8]))
def test_graph_replays_match_the_oracle_and_eager_calls(case):
    world, M, N, K, dtype, (tm, tn), variant, split, red = case
    p = Problem(world, M, N, K, dtype, tm, tn, seed=31)
    want = {r: oracle_block_bounded(p.A, p.shards[r], dtype) for r in range(world)}
    kw = dict(split_k=split, split_reduce=red)
    # eager calls first: they also create the split-K workspace outside the capture
    p.sentinel()
    for r in range(world):
        p.run(r, variant, **kw)
    p.barrier()
    check_gathered(p, want)
    eager = u16(p.out.C_all()).copy()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for r in range(world):
            p.out.run(p.dA, p.dB[r], r, variant, **kw)
    torch.cuda.synchronize()
    # capturing launched nothing: the counters still show the eager calls
    check_gathered(p, want)
    for rep in range(3):
        p.sentinel()                        # eager work between replays
        g.replay()
        p.calls += 1
        p.barrier()
        check_gathered(p, want)
        assert np.array_equal(u16(p.out.C_all()), eager), rep
        if split > 1:
            assert np.all(_ws_counters(p) == 0), rep
    del g


def test_current_stream_is_torchs_current_stream():
    """The binding launches on torch's current stream: the raw handle it
    reads equals torch's, on the default stream, inside a stream context and
    inside a graph capture (where the calls above are recorded)."""
    from tests.gpu_util import sym
    pkg = sym()
    assert pkg.current_stream() == torch.cuda.current_stream().cuda_stream
    assert pkg.current_stream(0) == torch.cuda.current_stream(0).cuda_stream
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        assert pkg.current_stream() == s.cuda_stream
    g = torch.cuda.CUDAGraph()
    seen = []
    x = torch.zeros(4, device="cuda")
    with torch.cuda.graph(g):
        seen.append((pkg.current_stream(), torch.cuda.current_stream().cuda_stream))
        x.add_(1)
    assert seen[0][0] == seen[0][1]
    g.replay()
    torch.cuda.synchronize()
    assert x.tolist() == [1.0] * 4
