"""Per-tile timelines of symtile_gemm_all_scatter (Section 3.4, instrumentation).

A trace buffer (GatheredOutput.new_trace) holds one record of 8 uint64 words
per output tile, written by the kernels when the config's trace pointer is
set: producer start, end of the K loop, stores acknowledged, counters
released, where the producer ran (HW_ID, XCC_ID, workgroup), and for the
schedules with a separate copy step, when the copy waited, started and
finished.  Times are ticks of the device's constant-rate realtime counter.

    tr = out.new_trace(); out.run(A, B, rank, variant, trace=tr)
    t = decode(tr.cpu().numpy(), symtile_clock_rate_khz(0))
    print(summary(t)); write_chrome(t, "timeline.json")   # chrome://tracing
"""
from __future__ import annotations

import json

import numpy as np

WORDS = 8
START, MAINLOOP, STORED, RELEASED, WHERE, COPY_WAIT, COPY_GO, COPY_DONE = range(8)
_TIMES = (START, MAINLOOP, STORED, RELEASED, COPY_WAIT, COPY_GO, COPY_DONE)


def decode(raw: np.ndarray, clock_khz: int) -> dict:
    """Times in microseconds from the earliest producer start, and the
    producer's location, per tile (arrays over tiles; NaN where a word was
    not written)."""
    raw = np.asarray(raw).reshape(-1, WORDS).astype(np.uint64)
    if clock_khz <= 0:
        raise ValueError("clock_khz must be positive")
    written = raw[:, START] != 0
    t0 = raw[written, START].min() if written.any() else 0
    us_per_tick = 1e3 / clock_khz
    out = {}
    names = {START: "start", MAINLOOP: "mainloop", STORED: "stored", RELEASED: "released",
             COPY_WAIT: "copy_wait", COPY_GO: "copy_go", COPY_DONE: "copy_done"}
    for w in _TIMES:
        v = raw[:, w]
        t = (v.astype(np.float64) - float(t0)) * us_per_tick
        t[v == 0] = np.nan
        out[names[w]] = t
    where = raw[:, WHERE]
    hw = (where >> np.uint64(32)).astype(np.uint32)
    out["wg"] = (where & np.uint64(0xFFFF)).astype(np.int64)
    out["xcc"] = ((where >> np.uint64(16)) & np.uint64(0xFFFF)).astype(np.int64)
    out["cu"] = ((hw >> 8) & 0xF).astype(np.int64)
    out["sh"] = ((hw >> 12) & 0x1).astype(np.int64)
    out["se"] = ((hw >> 13) & 0x7).astype(np.int64)
    out["written"] = written
    return out


def _stats(x: np.ndarray) -> dict:
    x = x[np.isfinite(x)]
    if x.size == 0:
        return {}
    return {"min": float(x.min()), "median": float(np.median(x)), "max": float(x.max())}


def summary(t: dict) -> dict:
    """Phase durations (us) over tiles and the span of the whole call."""
    s = {
        "tiles": int(t["written"].sum()),
        "mainloop_us": _stats(t["mainloop"] - t["start"]),
        "store_us": _stats(t["stored"] - t["mainloop"]),
        "release_us": _stats(t["released"] - t["stored"]),
        "start_us": _stats(t["start"]),
        "released_at_us": _stats(t["released"]),
    }
    if np.isfinite(t["copy_done"]).any():
        s["copy_wait_us"] = _stats(t["copy_go"] - t["copy_wait"])
        s["copy_us"] = _stats(t["copy_done"] - t["copy_go"])
        s["copy_done_at_us"] = _stats(t["copy_done"])
    ends = np.concatenate([t["released"][np.isfinite(t["released"])],
                           t["copy_done"][np.isfinite(t["copy_done"])]])
    s["span_us"] = float(ends.max()) if ends.size else 0.0
    return s


def chrome_events(t: dict) -> list:
    """Trace Event Format records: one process per XCC, one thread per
    producer workgroup; copy steps on a separate process."""
    ev = []
    n = t["start"].shape[0]
    phases = (("mainloop", "start", "mainloop"), ("store", "mainloop", "stored"),
              ("release", "stored", "released"))
    for i in range(n):
        if not t["written"][i]:
            continue
        for name, a, b in phases:
            if np.isfinite(t[a][i]) and np.isfinite(t[b][i]):
                ev.append({"name": name, "ph": "X", "ts": float(t[a][i]),
                           "dur": float(t[b][i] - t[a][i]), "pid": int(t["xcc"][i]),
                           "tid": int(t["wg"][i]), "args": {"tile": i}})
        if np.isfinite(t["copy_done"][i]):
            for name, a, b in (("copy wait", "copy_wait", "copy_go"),
                               ("copy", "copy_go", "copy_done")):
                ev.append({"name": name, "ph": "X", "ts": float(t[a][i]),
                           "dur": float(t[b][i] - t[a][i]), "pid": 100, "tid": i,
                           "args": {"tile": i}})
    return ev


def write_chrome(t: dict, path: str) -> None:
    with open(path, "w") as f:
        json.dump({"traceEvents": chrome_events(t), "displayTimeUnit": "ns"}, f)
