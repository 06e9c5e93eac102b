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
    assert "- counted bytes / avg duration: 1.7 GB/s" in text     # 250 B / 150 ns
    assert f"- source_sha: {profiling.sources_sha([str(src)])}" in text


def test_call_of_two_kernels_sums_durations_and_bytes(csvs, tmp_path):
    """--also adds a second kernel of the same call: its own lines, and the
    call's duration and bytes are the sums."""
    r = "void gas_kernel<256, 256, true, 8, true>(P)"
    _write(csvs / "trace2.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
           [["void gas_kernel<256, 256, true, 8, false>(P)", 1000, 1400], [r, 1450, 1500],
            ["void gas_kernel<256, 256, true, 8, false>(P)", 2000, 2200], [r, 2250, 2330]])
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    _write(csvs / "fetch2.csv", hdr,
           [[1, "void gas_kernel<256, 256, true, 8, false>(P)", "FETCH_SIZE", 100],
            [2, r, "FETCH_SIZE", 30], [4, "elementwise_kernel_manual_unroll<...>", "FETCH_SIZE", 64]])
    _write(csvs / "write2.csv", hdr,
           [[1, "void gas_kernel<256, 256, true, 8, false>(P)", "WRITE_SIZE", 10],
            [2, r, "WRITE_SIZE", 20], [5, "elementwise_kernel_manual_unroll<...>", "WRITE_SIZE", 128]])
    out = tmp_path / "call.md"
    profiling.main(["--trace", str(csvs / "trace2.csv"), "--last", "2",
                    "--kernel", r"gas_kernel<256, 256, true, 8, false>",
                    "--also", r"gas_kernel<256, 256, true, 8, true>",
                    "--fetch", str(csvs / "fetch2.csv"), "--write", str(csvs / "write2.csv"),
                    "--calib", "elementwise", "--calib-bytes", "128", "--out", str(out)])
    text = out.read_text()
    assert "- avg_ns: 300" in text                      # (400 + 200) / 2
    assert "- also avg_ns: 65" in text                  # (50 + 80) / 2
    assert "- call_avg_ns: 365" in text
    assert "- bytes_per_dispatch: 210" in text          # 100 x 2 + 10 x 1
    assert "- also fetch / write bytes per dispatch: 60 / 20" in text
    assert "- bytes_per_call: 290" in text


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
    # a call of several kernels: the whole call's bytes
    src.write_text("v1")
    prof.write_text(f"- bytes_per_dispatch: 1234\n- bytes_per_call: 2000\n"
                    f"- source_sha: {bench.sources_sha([str(src)])}\n")
    assert bench.counter_traffic("gas.md", [str(src)]) == 2000.0


def test_source_hash_ignores_comments_and_layout(tmp_path):
    """A comment or whitespace edit keeps the profiles valid; a code edit does not."""
    sys.path.insert(0, ROOT)
    from paper_2511_12500_amd import profiling
    src = tmp_path / "k.hip"
    src.write_text("int f(int x) {\n    return x + 1;   // one more\n}\n")
    h = profiling.sources_sha([str(src)])
    src.write_text("/* header\n   comment */\nint f(int x)\n{\n  return x + 1; // changed note\n}\n")
    assert profiling.sources_sha([str(src)]) == h
    src.write_text("int f(int x) {\n    return x + 2;\n}\n")
    assert profiling.sources_sha([str(src)]) != h


def test_matrix_core_evidence(tmp_path):
    k = "void gas_kernel<256, 256, true, 8>(P)"
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
           "End_Timestamp"]
    rows = []
    # 2 CUs on 2 XCDs, 1000 ns per dispatch; dispatch 1 is dropped by --last 2.
    # GRBM_GUI_ACTIVE 4000 over 2 XCDs in 1000 ns = 2.0 GHz (2000 clocks);
    # MFMA busy 4000 of 4 x 2 x 2000 SIMD cycles = 25%; flops 1e6 in 1000 ns =
    # 1 TFLOP/s against 2 x 4096 x 2.4 GHz = 19.66 TFLOP/s spec (5.1%) and
    # 2 x 4096 x 2.0 GHz = 16.38 at the measured clock (6.1%).
    for d, (grbm, busy) in enumerate([(9999, 1), (4000, 4000), (4000, 4000)]):
        t0 = 10000 * d
        for name, val in (("GRBM_GUI_ACTIVE", grbm / 2), ("GRBM_GUI_ACTIVE", grbm / 2),
                          ("SQ_VALU_MFMA_BUSY_CYCLES", busy), ("SQ_BUSY_CU_CYCLES", 7),
                          ("SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e6 / 512)):
            rows.append([d, k, name, val, t0, t0 + 1000])
    _write(tmp_path / "mfma.csv", hdr, rows)
    _write(tmp_path / "trace.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
           [[k, 0, 900], [k, 1000, 1900], [k, 2000, 2900]])
    out = tmp_path / "m.md"
    profiling.main(["--trace", str(tmp_path / "trace.csv"), "--last", "2", "--kernel",
                    "gas_kernel", "--mfma", str(tmp_path / "mfma.csv"), "--flops", "1e6",
                    "--cus", "2", "--xcds", "2", "--out", str(out)])
    text = out.read_text()
    assert "- clock (GRBM_GUI_ACTIVE / 2 XCDs / duration): 2.000 GHz (median of 2 dispatches)" in text
    assert "25.0% of all SIMD cycles" in text
    assert "- MFMA flops counted (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512): 1e+06 (algorithmic 1e+06)" in text
    assert "1.0 TFLOP/s = 5.1% of the spec peak (20 TFLOP/s at 2.4 GHz), 6.1% of the peak at the measured clock (16 TFLOP/s)" in text
    assert "not measured" not in text and "lower bound" not in text


def test_matrix_core_evidence_flags_a_counter_window_longer_than_the_dispatch(tmp_path):
    """GRBM_GUI_ACTIVE over the dispatch duration above the peak clock means
    the counters cover more than the dispatch: no clock, busy share a bound."""
    k = "void gas_kernel<128, 128, true, 8>(P)"
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
           "End_Timestamp"]
    rows = []
    for d in range(2):                 # 6000 clocks over 2 XCDs in 1000 ns = 3.0 GHz
        for name, val in (("GRBM_GUI_ACTIVE", 3000), ("GRBM_GUI_ACTIVE", 3000),
                          ("SQ_VALU_MFMA_BUSY_CYCLES", 1200), ("SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e6 / 512)):
            rows.append([d, k, name, val, 10000 * d, 10000 * d + 1000])
    _write(tmp_path / "mfma.csv", hdr, rows)
    _write(tmp_path / "trace.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
           [[k, 0, 1000], [k, 2000, 3000]])
    out = tmp_path / "m.md"
    profiling.main(["--trace", str(tmp_path / "trace.csv"), "--last", "2", "--kernel",
                    "gas_kernel", "--mfma", str(tmp_path / "mfma.csv"), "--flops", "1e6",
                    "--cus", "2", "--xcds", "2", "--out", str(out)])
    text = out.read_text()
    assert "3.000 GHz" in text and "the clock is not measured" in text
    assert "(a lower bound)" in text
    assert "of the spec peak (20 TFLOP/s at 2.4 GHz)" in text and "measured clock (" not in text


def test_bench_refuses_more_than_one_gpu(capsys):
    sys.path.insert(0, ROOT)
    import bench
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU only" in capsys.readouterr().err


def test_bench_default_tile_follows_the_schedule():
    sys.path.insert(0, ROOT)
    import bench
    assert bench.parse_args([]).tile is None            # resolved in bench_gas
    assert bench.parse_args(["--tile", "128x128"]).tile == "128x128"


def test_bench_profile_names_are_per_configuration():
    sys.path.insert(0, ROOT)
    import bench
    import workload
    wl = workload.LARGE_BF16
    a = bench.parse_args([])
    a.tile = "256x256"
    assert bench.gas_profile_name(a, wl) == f"gas_kernel_{wl.name}.md"
    b = bench.parse_args(["--variant", "wg_spec", "--gemm-wgs", "224", "--copy-wgs", "32"])
    b.tile = "256x256"
    assert bench.gas_profile_name(b, wl) == \
        f"gas_kernel_{wl.name}_wg_spec_256x256_nt2_g224_c32_m0.md"
    assert bench.copy_profile_name(a, workload.HEAP_COPY) == \
        f"tile_copy_kernel_{workload.HEAP_COPY.name}_t128.md"
    c = bench.parse_args(["--workload", workload.WIDE_F16.name, "--split-k", "2"])
    c.tile = "256x256"
    assert bench.gas_profile_name(c, workload.WIDE_F16) == \
        f"gas_kernel_{workload.WIDE_F16.name}_fused_seq_256x256_nt2_g0_c0_m0_k2.md"
    d = bench.parse_args(["--split-k", "1"])
    d.tile = "256x256"
    assert bench.gas_profile_name(d, wl) == f"gas_kernel_{wl.name}.md"
