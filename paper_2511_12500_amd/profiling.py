"""Summaries of rocprofv3 output for the kernels of this library.

Turns a ``--kernel-trace --stats`` kernel_stats CSV and two ``--pmc`` runs
(FETCH_SIZE, then WRITE_SIZE; KiB per dispatch) into a short text summary:
average launch duration of one kernel, and its memory traffic per launch.
Calls made of several kernels (the split-K reduction kernel follows the
K-loop kernel) name the others with ``--also``: each gets its own lines, and
``call_avg_ns`` / ``bytes_per_call`` sum the kernels of one call.
An optional third ``--pmc`` run (GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES,
SQ_BUSY_CU_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16 or _F16) adds the clock the
kernel ran at, the share of SIMD cycles its matrix cores were busy, and its
throughput against the matrix-core peak at the spec clock and at that clock.
The counters are calibrated against a plain device copy of known size that
ran in the same process (``bench.py --calibrate-traffic``): each counter is
scaled by known_bytes / counter_value(copy), so the figure is in bytes even
if the counter's unit or coverage differs from its nominal KiB.

    python -m paper_2511_12500_amd.profiling \\
        --trace DIR/run_kernel_stats.csv --fetch DIR2/run_counter_collection.csv \\
        --write DIR3/run_counter_collection.csv --kernel gas_kernel \\
        --calib direct_copy --calib-bytes 268435456 --sources a.hip b.h \\
        --command "..." --out profiles/NAME.md
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import re
import statistics
import sys


def _code_only(text: str) -> str:
    """C/C++ source without comments and with whitespace runs collapsed, so
    that a comment or layout edit does not count as a kernel change."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def sources_sha(paths) -> str:
    """Hash of the code (comments and layout ignored) of the given sources."""
    h = hashlib.sha256()
    for p in paths:
        with open(p, encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def trace_stats(path: str, kernel: str) -> dict:
    """Calls and durations (ns) of the first kernel whose name matches."""
    rx = re.compile(kernel)
    with open(path) as f:
        for row in csv.DictReader(f):
            if rx.search(row["Name"]):
                return {"name": row["Name"], "calls": int(row["Calls"]),
                        "avg_ns": float(row["AverageNs"]), "min_ns": float(row["MinNs"]),
                        "max_ns": float(row["MaxNs"])}
    raise KeyError(f"no kernel matching {kernel!r} in {path}")


def trace_last(path: str, kernel: str, last: int) -> dict:
    """Durations (ns) of the last `last` dispatches of the first kernel whose
    name matches, from a --kernel-trace run_kernel_trace.csv (dispatch
    order = start time)."""
    rx = re.compile(kernel)
    rows = []
    with open(path) as f:
        for row in csv.DictReader(f):
            if rx.search(row["Kernel_Name"]):
                rows.append((int(row["Start_Timestamp"]), int(row["End_Timestamp"]),
                             row["Kernel_Name"]))
    if not rows:
        raise KeyError(f"no kernel matching {kernel!r} in {path}")
    rows.sort()
    name = rows[0][2]
    d = [e - s for s, e, n in rows if n == name][-last:]
    return {"name": name, "calls": len(d), "avg_ns": statistics.fmean(d), "min_ns": min(d),
            "max_ns": max(d)}


def counter_per_dispatch(path: str, counter: str, kernel: str) -> tuple[float, int, str]:
    """Median over matching dispatches of the counter summed over instances."""
    rx = re.compile(kernel)
    per = {}
    name = ""
    with open(path) as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] != counter or not rx.search(row["Kernel_Name"]):
                continue
            name = row["Kernel_Name"]
            per[row["Dispatch_Id"]] = per.get(row["Dispatch_Id"], 0.0) + float(row["Counter_Value"])
    if not per:
        raise KeyError(f"no {counter} for kernel {kernel!r} in {path}")
    return statistics.median(per.values()), len(per), name


def dispatch_counters(path: str, kernel: str, last: int = 0) -> tuple[str, list[dict]]:
    """Per dispatch of the first kernel whose name matches: every counter
    summed over its instances, and the dispatch's duration in ns (from the
    counter run's own timestamps).  Dispatch order = dispatch id; with
    last > 0 only the last `last` dispatches are kept."""
    rx = re.compile(kernel)
    per: dict[int, dict] = {}
    name = ""
    with open(path) as f:
        for row in csv.DictReader(f):
            if not rx.search(row["Kernel_Name"]):
                continue
            if not name:
                name = row["Kernel_Name"]
            if row["Kernel_Name"] != name:
                continue
            d = per.setdefault(int(row["Dispatch_Id"]), {
                "dur_ns": float(row["End_Timestamp"]) - float(row["Start_Timestamp"])})
            d[row["Counter_Name"]] = d.get(row["Counter_Name"], 0.0) + float(row["Counter_Value"])
    if not per:
        raise KeyError(f"no dispatch of kernel {kernel!r} in {path}")
    rows = [per[k] for k in sorted(per)]
    return name, rows[-last:] if last else rows


def mfma_lines(path: str, kernel: str, last: int, cus: int, xcds: int, flops: float | None,
               peak_clk_ghz: float, flops_per_clk_cu: float) -> list[str]:
    """Matrix-core evidence from one --pmc run (medians over dispatches):
    clock = GRBM_GUI_ACTIVE / xcds / duration (GRBM_GUI_ACTIVE counts GPU
    clocks once per XCD); MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x
    cus x clocks); counted flops = SQ_INSTS_VALU_MFMA_MOPS_* x 512."""
    _, rows = dispatch_counters(path, kernel, last)
    med = lambda xs: statistics.median(xs)
    mops = next((c for c in ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F16")
                 if c in rows[0]), None)
    clk = [r["GRBM_GUI_ACTIVE"] / xcds / r["dur_ns"] for r in rows]      # GHz
    busy = [r["SQ_VALU_MFMA_BUSY_CYCLES"] / (4 * cus * r["GRBM_GUI_ACTIVE"] / xcds) for r in rows]
    # Above the peak clock the counter window must be longer than the
    # dispatch (it happens for dispatches of a few tens of microseconds): the
    # clock is then unknown and the busy share is a lower bound.
    window_ok = med(clk) <= peak_clk_ghz * 1.02
    out = ["",
           f"- clock (GRBM_GUI_ACTIVE / {xcds} XCDs / duration): {med(clk):.3f} GHz "
           f"(median of {len(rows)} dispatches)"
           + ("" if window_ok else f"; above the {peak_clk_ghz} GHz maximum, so the counter "
              "window is longer than this short dispatch and the clock is not measured"),
           f"- MFMA busy (SQ_VALU_MFMA_BUSY_CYCLES / (4 x {cus} SIMDs x clocks)): "
           f"{100 * med(busy):.1f}% of all SIMD cycles" + ("" if window_ok else " (a lower bound)")]
    if "SQ_BUSY_CU_CYCLES" in rows[0]:
        out.append(f"- SQ_BUSY_CU_CYCLES per dispatch: {med([r['SQ_BUSY_CU_CYCLES'] for r in rows]):.0f}")
    if mops:
        counted = med([r[mops] for r in rows]) * 512
        out.append(f"- MFMA flops counted ({mops} x 512): {counted:.4g}"
                   + (f" (algorithmic {flops:.4g})" if flops else ""))
    if flops:
        dur = med([r["dur_ns"] for r in rows])
        ach = flops / dur / 1e3                                          # TFLOP/s
        spec = cus * flops_per_clk_cu * peak_clk_ghz / 1e3
        at_clk = cus * flops_per_clk_cu * med(clk) / 1e3
        line = (f"- in this run: {dur:.0f} ns per dispatch, {ach:.1f} TFLOP/s = "
                f"{100 * ach / spec:.1f}% of the spec peak ({spec:.0f} TFLOP/s at "
                f"{peak_clk_ghz} GHz)")
        if window_ok:
            line += (f", {100 * ach / at_clk:.1f}% of the peak at the measured "
                     f"clock ({at_clk:.0f} TFLOP/s)")
        out.append(line)
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--trace", required=True,
                    help="run_kernel_stats.csv, or run_kernel_trace.csv with --last")
    ap.add_argument("--last", type=int, default=0,
                    help="average only the last N dispatches (needs run_kernel_trace.csv)")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--kernel", required=True, help="regex of the kernel to summarise")
    ap.add_argument("--also", action="append", default=[],
                    help="regex of another kernel of the same call (repeatable)")
    ap.add_argument("--calib", default="direct_copy", help="regex of the calibration copy")
    ap.add_argument("--calib-bytes", type=float, default=float(1 << 28),
                    help="bytes the calibration copy reads (and writes)")
    ap.add_argument("--algorithmic-bytes", type=float, default=None)
    ap.add_argument("--sources", nargs="*", default=[])
    ap.add_argument("--command", action="append", default=[])
    ap.add_argument("--mfma", help="run_counter_collection.csv of the matrix-core --pmc run")
    ap.add_argument("--flops", type=float, default=None, help="algorithmic flops per dispatch")
    ap.add_argument("--cus", type=int, default=256)
    ap.add_argument("--xcds", type=int, default=8)
    ap.add_argument("--peak-clock-ghz", type=float, default=2.4)
    ap.add_argument("--flops-per-clk-cu", type=float, default=4096.0,
                    help="dense bf16/fp16 matrix-core flops per clock per CU")
    ap.add_argument("--title", default="")
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)

    t = trace_last(a.trace, a.kernel, a.last) if a.last else trace_stats(a.trace, a.kernel)
    lines = [f"# {a.title or t['name']}", "", "Produced by:", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", f"- kernel: `{t['name']}`",
              f"- calls: {t['calls']}" + (f" (the last {a.last} dispatches)" if a.last else ""),
              f"- avg_ns: {t['avg_ns']:.0f}",
              f"- min_ns: {t['min_ns']:.0f}",
              f"- max_ns: {t['max_ns']:.0f}"]
    others = [trace_last(a.trace, k, a.last) if a.last else trace_stats(a.trace, k)
              for k in a.also]
    for o in others:
        lines += ["", f"- also kernel: `{o['name']}`", f"- also calls: {o['calls']}",
                  f"- also avg_ns: {o['avg_ns']:.0f}"]
    if others:
        lines += [f"- call_avg_ns: {t['avg_ns'] + sum(o['avg_ns'] for o in others):.0f} "
                  f"(the {1 + len(others)} kernels of one call)"]
    if a.fetch and a.write:
        fk, n_f, _ = counter_per_dispatch(a.fetch, "FETCH_SIZE", a.kernel)
        wk, n_w, _ = counter_per_dispatch(a.write, "WRITE_SIZE", a.kernel)
        cf, _, _ = counter_per_dispatch(a.fetch, "FETCH_SIZE", a.calib)
        cw, _, _ = counter_per_dispatch(a.write, "WRITE_SIZE", a.calib)
        f_scale = a.calib_bytes / cf
        w_scale = a.calib_bytes / cw
        fetch_b, write_b = fk * f_scale, wk * w_scale
        lines += ["",
                  f"- FETCH_SIZE per dispatch (counter units): {fk:.0f} (median of {n_f})",
                  f"- WRITE_SIZE per dispatch (counter units): {wk:.0f} (median of {n_w})",
                  f"- calibration copy of {a.calib_bytes:.0f} B: FETCH_SIZE {cf:.0f}, "
                  f"WRITE_SIZE {cw:.0f} -> scale {f_scale:.2f} / {w_scale:.2f} B per unit",
                  f"- fetch_bytes_per_dispatch: {fetch_b:.0f}",
                  f"- write_bytes_per_dispatch: {write_b:.0f}",
                  f"- bytes_per_dispatch: {fetch_b + write_b:.0f}",
                  f"- counted bytes / avg duration: {(fetch_b + write_b) / t['avg_ns']:.1f} GB/s"]
        call_b = fetch_b + write_b
        for k in a.also:
            ofk, _, _ = counter_per_dispatch(a.fetch, "FETCH_SIZE", k)
            owk, _, _ = counter_per_dispatch(a.write, "WRITE_SIZE", k)
            ob = ofk * f_scale + owk * w_scale
            call_b += ob
            lines.append(f"- also fetch / write bytes per dispatch: {ofk * f_scale:.0f} / "
                         f"{owk * w_scale:.0f}")
        if a.also:
            lines.append(f"- bytes_per_call: {call_b:.0f}")
        if a.algorithmic_bytes:
            lines.append(f"- algorithmic_bytes_per_dispatch: {a.algorithmic_bytes:.0f} "
                         f"(counters / algorithmic = {call_b / a.algorithmic_bytes:.2f}"
                         + (", whole call)" if a.also else ")"))
    if a.mfma:
        lines += mfma_lines(a.mfma, a.kernel, a.last, a.cus, a.xcds, a.flops, a.peak_clock_ghz,
                            a.flops_per_clk_cu)
    if a.sources:
        lines += ["", f"- source_sha: {sources_sha(a.sources)}  (of: {' '.join(a.sources)})"]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


if __name__ == "__main__":
    sys.exit(main())
