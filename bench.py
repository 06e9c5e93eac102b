#!/usr/bin/env python3
"""Benchmark of one GPU's share of the fused GEMM + All-Scatter on MI355X.

A step is one call of ``symtile_gemm_all_scatter`` for rank 0 of the
eight-rank bf16 workload (A [4096, 8192], B_shard [8192, 3584], gathered
output [4096, 28672] in an 8-slot heap): persistent MFMA GEMM, scatter of
every tile into all 8 slots, per-tile counters.  Inputs are synthetic
(seeded, N(0,1)/sqrt(K)) and resident in HBM before timing.

Printed: one JSON line with the GEMM + All-Scatter throughput (TFLOP/s),
its roofline fraction against the dense bf16 MFMA peak, the heap tile copy
(2048 x 2048 fp32 per rank, 8 ranks, ring r -> r+1) in GB/s against the
HBM peak, and the CPU oracle timed on a bounded sample as a baseline.  The
``configs`` array adds every other workload and schedule (the tiny fp16
case, bf16 1024x4096.4096x1024, the schedules and the producer/consumer
split sweep of the largest shape, the bulk-synchronous / fused /
specialised comparison on fp16 8192x8192.8192x1024, and the copy with
64x64 and 256x256 tiles), each with its own roofline fraction, and
``cpu_configs`` the oracle on every GEMM workload.

Every timed leg first runs a clock-settling phase: the GPU's clocks ramp
up over roughly the first 100 launches (30 ms) of sustained load after
idle, so each leg launches its own kernel back to back for at least 100
launches and 100 ms (reported as ``settle``) before its --warmup launches
and its timed steps.  --steps and --warmup are used exactly as given.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused GEMM+scatter TFLOP/s (% MFMA peak); heap tile-copy GB/s (% HBM peak)"
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f16": 2500.0}     # MI355X dense bf16/fp16
PEAK_HBM_GBS = 8000.0                                   # MI355X HBM3E
PROFILES = os.path.join(ROOT, "profiles")
DEVICE_HEADER = os.path.join(ROOT, "include", "symtile_device.h")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2511_12500_amd", "csrc", "gemm_all_scatter.hip"),
                  DEVICE_HEADER]
COPY_SOURCES = [os.path.join(ROOT, "paper_2511_12500_amd", "csrc", "tile_copy.hip"),
                DEVICE_HEADER]


def sources_sha(paths) -> str:
    """The profiles' hash of the kernel code (comments and layout ignored)."""
    from paper_2511_12500_amd.profiling import sources_sha as sha
    return sha(paths)


def counter_traffic(name: str, sources) -> float | None:
    """HBM bytes per launch from a committed rocprofv3 --pmc summary
    ``profiles/<name>`` (written by ``python -m paper_2511_12500_amd.profiling``):
    lines ``- bytes_per_dispatch: X`` (``- bytes_per_call: X`` for a call of
    several kernels) and ``- source_sha: H``.  None when absent or when the
    kernel source changed since the counters were taken."""
    path = os.path.join(PROFILES, name)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ":" in line:
                k, v = line[2:].split(":", 1)
                v = v.strip().split()
                fields[k.strip()] = v[0] if v else ""
    if fields.get("source_sha") != sources_sha(sources):
        return None
    try:
        return float(fields.get("bytes_per_call", fields["bytes_per_dispatch"]))
    except (KeyError, ValueError):
        return None


def gas_profile_name(args, wl) -> str:
    """The profiles/ summary that holds the counters of exactly this launch
    configuration (workload, schedule, tile, store policy, producer/consumer
    split, K slices)."""
    sk = f"_k{args.split_k}" if args.split_k > 1 else ""
    if args.split_k > 1 and getattr(args, "split_reduce", 0):
        sk += f"_r{args.split_reduce}"
    if getattr(args, "waves", 0):
        sk += f"_w{args.waves}"
    if (args.variant, args.tile, args.nontemporal, args.gemm_wgs, args.copy_wgs,
            args.group_m, sk) == ("fused_seq", "256x256", 2, 0, 0, 0, ""):
        return f"gas_kernel_{wl.name}.md"
    return (f"gas_kernel_{wl.name}_{args.variant}_{args.tile}_nt{args.nontemporal}"
            f"_g{args.gemm_wgs}_c{args.copy_wgs}_m{args.group_m}{sk}.md")


def copy_profile_name(args, wl, tile=None) -> str:
    name = f"tile_copy_kernel_{wl.name}_t{args.copy_tile if tile is None else tile}"
    return name + (f"_per{args.copy_per_wg}" if args.copy_per_wg else "") + ".md"


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    # (the clock ramp after idle is covered by each leg's settling phase, so
    # --warmup is only the extra launches before the timed ones)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="minimum length of each leg's clock-settling phase")
    ap.add_argument("--settle-launches", type=int, default=100,
                    help="minimum launches of each leg's clock-settling phase")
    ap.add_argument("--no-sweep", action="store_true",
                    help="only the headline legs (no configs array, no per-config oracle)")
    ap.add_argument("--sweep-steps", type=int, default=20, help="timed launches per configs entry")
    ap.add_argument("--sweep-min-ms", type=float, default=2.0,
                    help="configs entries time at least this long (more launches for short calls)")
    ap.add_argument("--workload", default="gas_bf16_w8_m4096_k8192_n3584")
    ap.add_argument("--variant", default="fused_seq",
                    choices=["bulk_sync", "fused_seq", "wg_spec", "unfused_pc", "wave_spec"])
    ap.add_argument("--tile", default=None,
                    help="output tile MxN (default 256x256; 256x128 for wave_spec, the only "
                         "tile that schedule is built for)")
    ap.add_argument("--waves", type=int, default=0,
                    help="waves per producer workgroup (0 = the tile's default)")
    ap.add_argument("--gemm-wgs", type=int, default=0)
    ap.add_argument("--copy-wgs", type=int, default=0)
    ap.add_argument("--group-m", type=int, default=0)
    ap.add_argument("--split-k", type=int, default=0,
                    help="K slices per output tile (bulk_sync, fused_seq; 0 or 1 = none)")
    ap.add_argument("--split-reduce", type=int, default=0,
                    help="who sums the K slices: 0 auto, 1 the last slice, 2 banded (every slice "
                         "sums and stores one band of rows), 3 a second reduction kernel")
    ap.add_argument("--nontemporal", type=int, default=2,
                    help="output store policy: 0 default, 1 non-temporal, 2 write-through")
    ap.add_argument("--copy-tile", type=int, default=128)
    ap.add_argument("--copy-iters", type=int, default=30)
    ap.add_argument("--copy-per-wg", type=int, default=0, help="tiles per workgroup (0 = auto)")
    ap.add_argument("--no-copy", action="store_true", help="skip the heap tile-copy leg")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--oracle-time", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--oracle-rows", type=int, default=0, help=argparse.SUPPRESS)
    ap.add_argument("--calibrate-traffic", action="store_true",
                    help="also run a plain 256 MiB device copy (known bytes) for counter runs")
    return ap.parse_args(argv)


VARIANTS = ("bulk_sync", "fused_seq", "wg_spec", "unfused_pc", "wave_spec")

# The configs array: (workload, schedule, tile, K slices, producer WGs,
# consumer WGs, split-K reduction: 0 auto, 1 last slice, 2 banded, 3 reduction
# kernel[, waves per producer workgroup]).  The headline leg (bf16
# 4096x8192.8192x3584, fused, 256x256, the default 4 waves) is not repeated
# here; its 8-wave build is.
SWEEP = [
    ("gas_f16_w2_m128_k256_n64", "fused_seq", "64x64", 0, 0, 0, 0),
    ("gas_f16_w2_m128_k256_n64", "wg_spec", "64x64", 0, 0, 0, 0),
    ("gas_bf16_w8_m1024_k4096_n1024", "fused_seq", "128x128", 4, 0, 0, 0),
    ("gas_bf16_w8_m1024_k4096_n1024", "fused_seq", "128x128", 4, 0, 0, 1),
    ("gas_bf16_w8_m1024_k4096_n1024", "bulk_sync", "128x128", 4, 0, 0, 0),
    ("gas_bf16_w8_m1024_k4096_n1024", "fused_seq", "256x256", 16, 0, 0, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "fused_seq", "256x256", 0, 0, 0, 0, 8),
    ("gas_bf16_w8_m4096_k8192_n3584", "bulk_sync", "256x256", 0, 0, 0, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "wave_spec", "256x128", 0, 0, 0, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "unfused_pc", "256x256", 0, 224, 32, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "wg_spec", "256x256", 0, 248, 8, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "wg_spec", "256x256", 0, 240, 16, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "wg_spec", "256x256", 0, 224, 32, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "wg_spec", "256x256", 0, 208, 48, 0),
    ("gas_bf16_w8_m4096_k8192_n3584", "wg_spec", "256x256", 0, 192, 64, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "fused_seq", "256x256", 2, 0, 0, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "fused_seq", "256x256", 2, 0, 0, 1),
    ("gas_f16_w8_m8192_k8192_n1024", "fused_seq", "256x128", 0, 0, 0, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "bulk_sync", "256x256", 2, 0, 0, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "bulk_sync", "256x128", 0, 0, 0, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "wave_spec", "256x128", 0, 0, 0, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "wg_spec", "256x128", 0, 128, 128, 0),
    ("gas_f16_w8_m8192_k8192_n1024", "unfused_pc", "256x128", 0, 192, 64, 0),
]


class GasCase:
    """Inputs in HBM, heap and gathered buffers of one workload and tile,
    reused by every leg with that workload and tile."""

    def __init__(self, torch, sym, workload, wl, tile):
        self.wl = wl
        self.tm, self.tn = (int(x) for x in tile.split("x"))
        A, B = workload.workload_inputs(wl, seed=0)
        self.A, self.B = A, B
        self.dA, self.dB = A.cuda(), B.cuda()
        tiles = -(-wl.M // self.tm) * -(-wl.N_local // self.tn)
        slot = wl.M * wl.N_gathered * 2 + wl.world * tiles * 4 + (1 << 16)
        self.heap = sym.Heap(wl.world, slot)
        self.out = sym.GatheredOutput(self.heap, wl.M, wl.N_local,
                                      workload.torch_dtype(wl.dtype), self.tm, self.tn)

    def close(self):
        self.heap.close()


def settle(launch, torch, args) -> dict:
    """Back-to-back launches until at least --settle-launches of them and
    --settle-ms have run (the clock ramp after idle); returns what ran."""
    t0 = time.perf_counter()
    n = 0
    while True:
        for _ in range(10):
            launch()
        n += 10
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3
        if n >= args.settle_launches and ms >= args.settle_ms:
            return {"launches": n, "ms": round(ms, 1)}


def time_back_to_back(launch, torch, steps: int) -> float:
    """Total ms of `steps` launches back to back between two events on the
    launch stream (the library launches on torch's current stream).  An event
    pair around every launch would add a stream barrier (and about 10 us) to
    each; launches on one stream do not overlap, so the average launch
    duration is total / steps (it includes the ~2 us between launches)."""
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(steps):
        launch()
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1)


def per_call_median_ms(launch, torch, n: int) -> float:
    """Median of n launches each timed by its own event pair."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for a, b in evs:
        a.record()
        launch()
        b.record()
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in evs)


def gas_leg(args, torch, sym, case, variant, split_k, gemm_wgs, copy_wgs, steps, warmup,
            label_args, with_median=False, split_reduce=0, min_ms=0.0, waves=None) -> dict:
    """One timed GEMM + All-Scatter configuration on `case`.  With min_ms > 0
    the number of timed launches is raised until they take about min_ms (from
    the settling phase's pace), so that the gap before the first launch of a
    short call weighs little."""
    wl = case.wl
    v = {"bulk_sync": sym.BULK_SYNC, "fused_seq": sym.FUSED_SEQ, "wg_spec": sym.WG_SPEC,
         "unfused_pc": sym.UNFUSED_PC, "wave_spec": sym.WAVE_SPEC}[variant]
    kw = dict(gemm_wgs=gemm_wgs, copy_wgs=copy_wgs, nontemporal=args.nontemporal,
              group_m=args.group_m, split_k=split_k, split_reduce=split_reduce,
              waves_per_wg=getattr(args, "waves", 0) if waves is None else waves)

    def launch():
        case.out.run(case.dA, case.dB, 0, v, **kw)

    st = settle(launch, torch, args)
    if min_ms > 0 and st["launches"]:
        steps = max(steps, math.ceil(min_ms / (st["ms"] / st["launches"])))
    # the per-call median of the measurement convention (one event pair per
    # call), before the timed region so that its launches are the last ones
    med = per_call_median_ms(launch, torch, 20) if with_median else None
    for _ in range(warmup):
        launch()
    case.heap.barrier()
    total_ms = time_back_to_back(launch, torch, steps)
    case.heap.barrier()        # raises if a device-side wait timed out
    ms = total_ms / steps
    tflops = wl.flops / (ms * 1e-3) / 1e12
    peak = PEAK_MFMA_TFLOPS[wl.dtype]
    prof = gas_profile_name(label_args, wl)
    traffic = counter_traffic(prof, KERNEL_SOURCES)
    return {"ms": ms, "tflops": tflops, "settle": st, "per_call_median_ms": med, "steps": steps,
            "roofline": {"bound": "mfma", "achieved": tflops, "peak": peak, "unit": "TFLOP/s",
                         "frac": tflops / peak, "traffic": traffic,
                         "traffic_profile": f"profiles/{prof}" if traffic is not None else None,
                         "kernel": "gas_kernel<%d,%d,%s,%d waves>" % (
                             case.tm, case.tn, wl.dtype,
                             waves_used("%dx%d" % (case.tm, case.tn), variant, split_k,
                                        kw["waves_per_wg"])),
                         "algorithmic_flops_per_launch": wl.flops,
                         "algorithmic_bytes_per_launch": gemm_bytes(wl),
                         "avg_launch_ms": ms}}


def waves_used(tile: str, variant: str, split_k: int, waves: int) -> int:
    """Waves per producer workgroup the library runs for these arguments
    (waves 0 = the library's default for the tile and schedule)."""
    if waves:
        return waves
    if tile == "64x64" or (tile == "256x256" and split_k <= 1 and
                           variant in ("fused_seq", "bulk_sync")):
        return 4
    return 8


def gemm_bytes(wl) -> int:
    """Compulsory bytes of one call: A and B_shard read once, the rank's
    block written once into each of the w slots."""
    return 2 * (wl.M * wl.K + wl.K * wl.N_local + wl.world * wl.M * wl.N_local)


class _Label:
    """The argument names gas_profile_name reads, for a configs entry."""

    def __init__(self, args, variant, tile, split_k, gemm_wgs, copy_wgs, split_reduce=0,
                 waves=0):
        self.variant, self.tile, self.split_k = variant, tile, split_k
        self.waves = waves
        self.split_reduce = split_reduce
        self.gemm_wgs, self.copy_wgs = gemm_wgs, copy_wgs
        self.nontemporal, self.group_m = args.nontemporal, args.group_m


def bench_gas(args, torch, sym, workload):
    wl = workload.GEMM_WORKLOADS[args.workload]
    if args.tile is None:
        args.tile = "256x128" if args.variant == "wave_spec" else "256x256"
    case = GasCase(torch, sym, workload, wl, args.tile)
    r = gas_leg(args, torch, sym, case, args.variant, args.split_k, args.gemm_wgs,
                args.copy_wgs, args.steps, args.warmup, args, with_median=True,
                split_reduce=args.split_reduce)
    res = {
        "value": r["tflops"],
        "ms_per_step": r["ms"],
        "per_call_median_ms": r["per_call_median_ms"],
        "settle": r["settle"],
        "roofline": r["roofline"],
        "config": {"workload": wl.name, "M": wl.M, "K": wl.K, "N_local": wl.N_local,
                   "world_size": wl.world, "rank": 0, "N_gathered": wl.N_gathered,
                   "variant": args.variant, "tile": args.tile, "gemm_wgs": args.gemm_wgs,
                   "copy_wgs": args.copy_wgs, "nontemporal": args.nontemporal,
                   "split_k": max(args.split_k, 1), "split_reduce": args.split_reduce},
        "dtype": wl.dtype,
    }
    A, B = case.A, case.B
    case.close()
    return res, wl, A, B


def library_baseline(args, torch, sym, workload) -> dict:
    """The one-GPU analogue of the paper's baseline (torch.matmul followed by
    an RCCL all-gather): torch.matmul of rank 0's share into a local tensor,
    then torch copies of it into rank 0's block of every slot (no counters).
    Timed like the headline leg, on the same workload; context, not a target."""
    wl = workload.GEMM_WORKLOADS[args.workload]
    case = GasCase(torch, sym, workload, wl, "256x256")
    c_local = torch.empty(wl.M, wl.N_local, dtype=case.dA.dtype, device="cuda")
    blocks = [case.out.C(s)[:, :wl.N_local] for s in range(wl.world)]

    def launch():
        torch.matmul(case.dA, case.dB, out=c_local)
        for b in blocks:
            b.copy_(c_local)

    st = settle(launch, torch, args)
    for _ in range(args.warmup):
        launch()
    ms = time_back_to_back(launch, torch, args.steps) / args.steps
    del blocks
    case.close()
    return {"kind": "torch.matmul + torch copies of the block into the w slots",
            "ms": ms, "value": wl.flops / (ms * 1e-3) / 1e12, "unit": "TFLOP/s",
            "steps": args.steps, "settle": st}


def bench_sweep(args, torch, sym, workload) -> list:
    """Every SWEEP entry, grouped so each workload and tile's buffers are
    built once."""
    out = []
    cases = {}
    for entry in SWEEP:
        name, variant, tile, split_k, g, c, red = entry[:7]
        waves = entry[7] if len(entry) > 7 else 0
        key = (name, tile)
        if key not in cases:
            for k in list(cases):
                cases.pop(k).close()
            cases[key] = GasCase(torch, sym, workload, workload.GEMM_WORKLOADS[name], tile)
        case = cases[key]
        label = _Label(args, variant, tile, split_k, g, c, red, waves)
        r = gas_leg(args, torch, sym, case, variant, split_k, g, c, args.sweep_steps, 5, label,
                    split_reduce=red, min_ms=args.sweep_min_ms, waves=waves)
        wl = case.wl
        out.append({"workload": name, "dtype": wl.dtype, "schedule": variant, "tile": tile,
                    "split_k": max(split_k, 1), "split_reduce": red, "gemm_wgs": g,
                    "copy_wgs": c, "waves": waves or None,
                    "ms": r["ms"], "value": r["tflops"], "unit": "TFLOP/s",
                    "steps": r["steps"], "settle": r["settle"],
                    "roofline": r["roofline"]})
    for k in list(cases):
        cases.pop(k).close()
    out += graph_legs(args, torch, sym, workload)
    return out


# Workloads whose calls are short enough that the host's launch rate bounds
# back-to-back calls: also timed as GRAPH_CALLS calls captured in one HIP
# graph and replayed (workload, schedule, tile).
GRAPH_CALLS = 20
GRAPH_LEGS = [("gas_f16_w2_m128_k256_n64", "fused_seq", "64x64")]


def graph_legs(args, torch, sym, workload) -> list:
    """Per-call time of GRAPH_CALLS calls replayed from one captured graph
    (the launch overhead of the host leaves the timed region)."""
    out = []
    for name, variant, tile in GRAPH_LEGS:
        wl = workload.GEMM_WORKLOADS[name]
        case = GasCase(torch, sym, workload, wl, tile)
        v = {"bulk_sync": sym.BULK_SYNC, "fused_seq": sym.FUSED_SEQ}[variant]
        kw = dict(nontemporal=args.nontemporal, group_m=args.group_m)
        case.out.run(case.dA, case.dB, 0, v, **kw)            # eager call before the capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(GRAPH_CALLS):
                case.out.run(case.dA, case.dB, 0, v, **kw)
        st = settle(g.replay, torch, args)
        steps = max(args.sweep_steps, math.ceil(args.sweep_min_ms / (st["ms"] / st["launches"])))
        for _ in range(5):
            g.replay()
        case.heap.barrier()
        ms = time_back_to_back(g.replay, torch, steps) / (steps * GRAPH_CALLS)
        case.heap.barrier()
        tflops = wl.flops / (ms * 1e-3) / 1e12
        peak = PEAK_MFMA_TFLOPS[wl.dtype]
        out.append({"workload": name, "dtype": wl.dtype, "schedule": variant, "tile": tile,
                    "split_k": 1, "split_reduce": 0, "gemm_wgs": 0, "copy_wgs": 0,
                    "graph_calls": GRAPH_CALLS, "ms": ms, "value": tflops, "unit": "TFLOP/s",
                    "steps": steps, "settle": st,
                    "roofline": {"bound": "mfma", "achieved": tflops, "peak": peak,
                                 "unit": "TFLOP/s", "frac": tflops / peak, "traffic": None,
                                 "kernel": "gas_kernel<%d,%d,%s>" % (case.tm, case.tn, wl.dtype),
                                 "algorithmic_flops_per_launch": wl.flops,
                                 "algorithmic_bytes_per_launch": gemm_bytes(wl),
                                 "avg_launch_ms": ms}})
        del g
        case.close()
    return out


def bench_copy(args, torch, sym, workload, tile=None):
    wl = workload.HEAP_COPY
    t = args.copy_tile if tile is None else tile
    nbytes = wl.rows * wl.cols * 4
    heap = sym.Heap(wl.world, 2 * nbytes + (1 << 20))
    src, dst = heap.alloc(nbytes), heap.alloc(nbytes)
    flags = heap.alloc(1 << 16)
    heap.slots_view(src, (wl.rows, wl.cols), torch.float32).copy_(workload.copy_send(wl).cuda())
    # Cold runs: read 1 GiB of other data first (more than the 256 MB MALL) so
    # the heap is evicted; a read leaves no dirty lines to write back later.
    flush = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
    stream = sym.current_stream()

    def launch():
        sym.symtile_tile_copy(heap.handle, src, dst, wl.rows, wl.cols, wl.cols, sym.F32, t, t,
                              wl.shift, -1, flags, tiles_per_wg=args.copy_per_wg, stream=stream)

    st = settle(launch, torch, args)
    # warm launches back to back (an event pair each), then cold ones, each
    # after the flush: first with an event pair around the launch (it holds
    # the dispatch and the kernel-end fence, ~3 us), then -- the measurement --
    # with events that bracket exactly the kernel (symtile_tile_copy_timed);
    # these are the last copy-iters dispatches of the kernel, which the
    # committed rocprofv3 summary averages
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.copy_iters)]
    for a, b in evs:
        a.record()
        launch()
        b.record()
    torch.cuda.synchronize()
    warm = [a.elapsed_time(b) for a, b in evs]
    cold_launch = []
    for i in range(args.copy_iters):
        flush.max()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        launch()
        b.record()
        torch.cuda.synchronize()
        cold_launch.append(a.elapsed_time(b))
    cold = []
    for i in range(args.copy_iters):
        flush.max()
        cold.append(sym.symtile_tile_copy_timed(heap.handle, src, dst, wl.rows, wl.cols, wl.cols,
                                                sym.F32, t, t, wl.shift, -1, flags,
                                                tiles_per_wg=args.copy_per_wg, stream=stream))
    heap.barrier()
    moved = wl.bytes_moved
    # medians of the individually timed cold launches (the mean is kept beside it)
    cold_ms = statistics.median(cold)
    cold_mean_ms = statistics.fmean(cold)
    cold_launch_ms = statistics.median(cold_launch)
    warm_ms = sum(warm) / len(warm)
    gbs = moved / (cold_ms * 1e-3) / 1e9
    prof = copy_profile_name(args, wl, t)
    traffic = counter_traffic(prof, COPY_SOURCES)
    heap.close()
    del flush
    return {
        "value": gbs, "unit": "GB/s", "tile": f"{t}x{t}", "workload": wl.name,
        "tiles_per_wg": args.copy_per_wg, "settle": st,
        "bytes_per_launch": moved, "cold_ms": cold_ms, "cold_mean_ms": cold_mean_ms,
        "cold_launch_ms": cold_launch_ms,
        "cold_launch_GBps": moved / (cold_launch_ms * 1e-3) / 1e9,
        "warm_ms": warm_ms,
        "warm_GBps": moved / (warm_ms * 1e-3) / 1e9,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gbs / PEAK_HBM_GBS, "traffic": traffic,
                     "traffic_profile": f"profiles/{prof}" if traffic is not None else None,
                     "kernel": "tile_copy_kernel", "avg_launch_ms": cold_ms},
    }


def cpu_model() -> str:
    """The host CPU as the OS reports it: the model name (the longer of
    lscpu's and /proc/cpuinfo's), the family / model / stepping numbers, the
    sockets, and the logical CPUs this process may use."""
    import subprocess
    info = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        info = {k.strip(): v.strip() for k, v in
                (l.split(":", 1) for l in out.splitlines() if ":" in l)}
    except (OSError, subprocess.SubprocessError, ValueError):
        pass
    names = [info.get("Model name", "")]
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    names.append(line.split(":", 1)[1].strip())
                    break
    except OSError:
        pass
    name = max(names, key=len) or "unknown"
    ids = [f"{k.lower()} {info[k]}" for k in ("CPU family", "Model", "Stepping")
           if info.get(k)]
    extra = ids + ([f"{info['Socket(s)']} socket(s)"] if info.get("Socket(s)") else [])
    extra.append(f"{len(os.sched_getaffinity(0))} logical CPUs available")
    return f"{name} ({', '.join(extra)})"


def oracle_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))


def oracle_gemm_rate(wl, rows: int, seconds: float, workload) -> dict:
    """The oracle (GEMM + placement into every slot + counters) on rows
    0..rows-1 of A of workload wl, rank 0, repeated for about `seconds`."""
    import oracle
    A, B = workload.workload_inputs(wl, 0)
    Ab, Bb = workload.bits(A), workload.bits(B)
    st = oracle.GatheredState(wl.world, rows, wl.N_local, wl.tile_m, wl.tile_n)
    done, total = 0, 0.0
    while (total < seconds and done < 1000) or done == 0:
        t0 = time.perf_counter()
        oracle.gemm_all_scatter(st, Ab[:rows], Bb, wl.dtype, 0)
        total += time.perf_counter() - t0
        done += 1
    flops = 2.0 * rows * wl.N_local * wl.K * done
    return {"value": flops / total / 1e12, "unit": "TFLOP/s", "cores": oracle_threads(),
            "kind": "oracle", "rows": rows, "of_rows": wl.M, "repetitions": done,
            "seconds": round(total, 2)}


def oracle_time_child(name: str, rows: int, seconds: float, threads: int) -> dict:
    """oracle_gemm_rate in a child process with `threads` OpenMP threads (the
    OpenMP runtime fixes its thread count at start-up).  The child touches no
    GPU."""
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS=str(threads))
    out = subprocess.run([sys.executable, os.path.abspath(__file__), "--oracle-time", name,
                          "--oracle-rows", str(rows), "--cpu-seconds", str(seconds)],
                         env=env, capture_output=True, text=True, check=True)
    return json.loads(out.stdout.strip().splitlines()[-1])


def cpu_configs(args, workload) -> dict:
    """The oracle (GEMM + placement + counters) on every GEMM workload with
    all host threads (the first 512 rows of A where M is larger), and with one
    thread on the tiny fp16 and the bf16 1024x4096.4096x1024 workloads, each
    for about a quarter of --cpu-seconds."""
    out = {"cpu_model": cpu_model()}
    secs = max(1.0, args.cpu_seconds / 4)
    for wl in workload.GEMM_WORKLOADS.values():
        rows = min(wl.M, 512)
        out[wl.name] = oracle_gemm_rate(wl, rows, secs, workload)
    for wl in (workload.TINY, workload.SMALL_BF16):
        out[wl.name + " (1 thread)"] = oracle_time_child(wl.name, min(wl.M, 512), secs, 1)
    return out


def copy_cpu_baseline(args, workload) -> dict:
    """The oracle's heap tile copy (one thread) on the whole copy workload."""
    import numpy as np

    import oracle
    wl = workload.HEAP_COPY
    send = workload.copy_send(wl).numpy()
    recv = np.zeros_like(send)
    done, total = 0, 0.0
    while (total < max(1.0, args.cpu_seconds / 4) and done < 100) or done == 0:
        t0 = time.perf_counter()
        oracle.tile_copy(send, recv, args.copy_tile, args.copy_tile, shift=wl.shift)
        total += time.perf_counter() - t0
        done += 1
    return {"value": wl.bytes_moved * done / total / 1e9, "unit": "GB/s", "cores": 1,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"the whole workload ({wl.world} x {wl.rows}x{wl.cols} fp32, "
                      f"{args.copy_tile}x{args.copy_tile} tiles, ring r -> r+{wl.shift}), "
                      f"{done} calls, {total:.1f} s"}


def cpu_baseline(args, wl, A, B, workload):
    """The oracle (GEMM + placement into every slot + counters) timed on the
    host cores on the first rows of the same workload, repeated until about
    --cpu-seconds of work; TFLOP/s."""
    import oracle
    Ab, Bb = workload.bits(A), workload.bits(B)
    threads = oracle_threads()
    rows = min(512, wl.M)                 # bounds the oracle's gathered state (~0.6 GB)
    st = oracle.GatheredState(wl.world, rows, wl.N_local, 256, 256)
    done, total = 0, 0.0
    while total < args.cpu_seconds and done < 64:
        t0 = time.perf_counter()
        oracle.gemm_all_scatter(st, Ab[:rows], Bb, wl.dtype, 0)
        total += time.perf_counter() - t0
        done += 1
    flops = 2.0 * rows * wl.N_local * wl.K * done
    return {"value": flops / total / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"rows 0..{rows - 1} of A (of {wl.M}) against rank 0's shard "
                      f"[{wl.K}, {wl.N_local}]: fp32 GEMM + placement into {wl.world} slots + "
                      f"counters, {done} repetitions, {total:.1f} s"}


def main(argv=None):
    args = parse_args(argv)
    if args.oracle_time:                  # child of oracle_time_child: CPU only
        import workload
        wl = workload.GEMM_WORKLOADS[args.oracle_time]
        print(json.dumps(oracle_gemm_rate(wl, args.oracle_rows or wl.M, args.cpu_seconds,
                                          workload)), flush=True)
        return 0
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (the emulated ranks live in one "
              f"GPU's HBM); --gpus {args.gpus} is not supported", file=sys.stderr)
        return 2
    import torch

    import paper_2511_12500_amd as sym
    import workload

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    # Order: the copy legs (the headline tile last), the configs array, then
    # the headline GEMM leg, so that the last dispatches of each headline
    # kernel are its timed ones (the committed rocprofv3 summaries average
    # those).  Every leg settles the clock first.
    copies = []
    if not args.no_copy:
        if not args.no_sweep:
            copies = [bench_copy(args, torch, sym, workload, tile=t)
                      for t in workload.HEAP_COPY.tiles if t != args.copy_tile]
        copy = bench_copy(args, torch, sym, workload)
    else:
        copy = None
    sweep = [] if args.no_sweep else bench_sweep(args, torch, sym, workload)
    lib = None if args.no_sweep else library_baseline(args, torch, sym, workload)
    res, wl, A, B = bench_gas(args, torch, sym, workload)
    line = {
        "metric": METRIC,
        "value": res["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": res["dtype"],
        "data": "synthetic",
        "config": res["config"],
        "roofline": res["roofline"],
        "settle": res["settle"],
        "per_call_median_ms": res["per_call_median_ms"],
    }
    if copy is not None:
        line["tile_copy"] = copy
        if not args.no_cpu_baseline:
            line["tile_copy"]["cpu_baseline"] = copy_cpu_baseline(args, workload)
    if copies or sweep:
        line["configs"] = [dict(c, schedule="heap_copy") for c in copies] + sweep
    if lib is not None:
        lib["speedup_of_this_call"] = lib["ms"] / res["ms_per_step"]
        line["library_baseline"] = lib
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args, wl, A, B, workload)
        if not args.no_sweep:
            line["cpu_configs"] = cpu_configs(args, workload)
    if args.calibrate_traffic:
        # a plain copy kernel of known size: 256 MiB read + 256 MiB written
        x = torch.ones(1 << 28, dtype=torch.uint8, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
