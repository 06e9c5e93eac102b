"""rocprofv3 summaries (paper_2511_12500_amd.profiling) on synthetic CSVs,
and bench.py's reading of them (no GPU)."""
import csv
import os
import sys

import pytest

from paper_2511_12500_amd import profiling

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


@pytest.fixture
def csvs(tmp_path):
    k, c = "void gas_kernel<256, 256, true, 8>(P)", "elementwise_kernel_manual_unroll<...>"
    _write(tmp_path / "stats.csv", ["Name", "Calls", "AverageNs", "MinNs", "MaxNs"],
           [[k, 4, 250.0, 100, 400]])
    # dispatches out of start order; durations 400, 300, 200, 100 in start order
    _write(tmp_path / "trace.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
           [[k, 3000, 3100], [k, 1000, 1400], [c, 1500, 1600], [k, 2000, 2300], [k, 2500, 2700]])
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    # two counter instances per dispatch are summed; the median over dispatches is taken
    _write(tmp_path / "fetch.csv", hdr,
           [[1, k, "FETCH_SIZE", 50], [1, k, "FETCH_SIZE", 50], [2, k, "FETCH_SIZE", 300],
            [3, k, "FETCH_SIZE", 120], [4, c, "FETCH_SIZE", 64]])
    _write(tmp_path / "write.csv", hdr, [[1, k, "WRITE_SIZE", 10], [5, c, "WRITE_SIZE", 128]])
    return tmp_path


def test_last_n_dispatches_and_calibrated_bytes(csvs, tmp_path):
    src = tmp_path / "k.hip"
    src.write_text("kernel source")
    out = tmp_path / "summary.md"
    profiling.main(["--trace", str(csvs / "trace.csv"), "--last", "2", "--kernel", "gas_kernel",
                    "--fetch", str(csvs / "fetch.csv"), "--write", str(csvs / "write.csv"),
                    "--calib", "elementwise", "--calib-bytes", "128", "--sources", str(src),
                    "--command", "cmd", "--out", str(out)])
    text = out.read_text()
    assert "- calls: 2 (the last 2 dispatches)" in text
    assert "- avg_ns: 150" in text                      # (200 + 100) / 2
    # fetch: median(100, 300, 120) = 120 units x (128 B / 64) = 240 B;
    # write: 10 units x (128 B / 128) = 10 B
    assert "- fetch_bytes_per_dispatch: 240" in text
    assert "- write_bytes_per_dispatch: 10" in text
    assert "- bytes_per_dispatch: 250" in text
    assert f"- source_sha: {profiling.sources_sha([str(src)])}" in text


def test_kernel_stats_without_counters(csvs, tmp_path):
    out = tmp_path / "s.md"
    profiling.main(["--trace", str(csvs / "stats.csv"), "--kernel", "gas_kernel",
                    "--out", str(out)])
    text = out.read_text()
    assert "- avg_ns: 250" in text and "bytes_per_dispatch" not in text


def test_bench_reads_traffic_only_for_matching_sources(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    src = tmp_path / "k.hip"
    src.write_text("v1")
    prof = tmp_path / "gas.md"
    prof.write_text(f"- bytes_per_dispatch: 1234\n- source_sha: {bench.sources_sha([str(src)])}\n")
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.counter_traffic("gas.md", [str(src)]) == 1234.0
    src.write_text("v2")                               # kernel changed since the counters
    assert bench.counter_traffic("gas.md", [str(src)]) is None
    assert bench.counter_traffic("absent.md", [str(src)]) is None
