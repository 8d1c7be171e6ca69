"""Host logic of the rocprofv3 summaries (synthetic trace and counter files):
the run window after autotune, per-run kernel statistics, the conv class
total, and the copy-calibrated traffic per run."""

import csv
import json

import pytest

from paper_2105_03215_amd import profiling

STEM = "byoc::(anonymous namespace)::stem_conv_maxpool_kernel(byoc::StemParams)"
CONV = "void byoc::(anonymous namespace)::conv_dma_kernel<64, 64, 2, 2, 3, true, false>(byoc::ConvParams)"
POOL = "byoc::(anonymous namespace)::avgpool_nhwc_kernel(byoc::PoolParams)"


def _trace(path, runs):
    t = 0
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for run, scale in runs:
            for name, ns in ((STEM, 10000), (CONV, 20000 * scale), (CONV, 30000 * scale), (POOL, 5000)):
                w.writerow({"Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + ns})
                t += ns + 1000


def test_stats_counts_only_the_last_runs(tmp_path):
    p = tmp_path / "trace.csv"
    # two tuning-like runs with slower conv, then three measured runs
    _trace(p, [(0, 3), (1, 3), (2, 1), (3, 1), (4, 1)])
    out = tmp_path / "s.txt"
    profiling.stats(str(p), "cmd", str(out), last_runs=3, flops_per_run=60e9)
    text = out.read_text()
    assert "(3 runs of the subgraph after autotune, the last ones)" in text
    conv_line = [l for l in text.splitlines() if "conv_dma_kernel" in l][0].split()
    assert float(conv_line[-4]) == 2.0          # calls per run
    assert float(conv_line[-3]) == 25.0         # avg us
    assert float(conv_line[-2]) == 50.0         # us per run
    assert "60.0 us per run" in text            # stem 10 + conv 50
    assert "1000.0 TFLOP/s" in text             # 60 GFLOP in 60 us
    with pytest.raises(RuntimeError):
        profiling.stats(str(p), "cmd", str(out), last_runs=9)


def test_stats_cut_by_launch_count(tmp_path):
    """Workloads without a marker kernel: the last runs are the last
    runs x launches-per-run dispatches (a run here is 4 dispatches)."""
    p = tmp_path / "trace.csv"
    _trace(p, [(0, 3), (1, 1), (2, 1)])
    out = tmp_path / "s.txt"
    profiling.stats(str(p), "cmd", str(out), last_runs=2, marker=4)
    text = out.read_text()
    assert "(2 runs of the subgraph" in text
    assert "65.0 us per run" in text            # stem 10 + conv 50 + pool 5
    with pytest.raises(RuntimeError):
        profiling.stats(str(p), "cmd", str(out), last_runs=4, marker=4)


def _counters(path, rows, counter):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_traffic_scales_by_copy_calibration(tmp_path):
    run = [(STEM, 100.0), (CONV, 300.0), (POOL, 50.0)]
    _counters(tmp_path / "f.csv", [(CONV, 999.0)] + run * 3, "FETCH_SIZE")
    _counters(tmp_path / "w.csv", run * 3, "WRITE_SIZE")
    # the copy of 1 MiB reads as 512 KiB fetched and 2048 KiB written
    _counters(tmp_path / "cf.csv", [("__amd_rocclr_copyBuffer", 512.0)] * 3, "FETCH_SIZE")
    _counters(tmp_path / "cw.csv", [("__amd_rocclr_copyBuffer", 2048.0)] * 3, "WRITE_SIZE")
    out = tmp_path / "t.json"
    doc = profiling.traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(tmp_path / "cf.csv"),
                            str(tmp_path / "cw.csv"), 1, "wl", str(out), last_runs=2)
    assert doc["fetch_scale"] == 2.0 and doc["write_scale"] == 0.5
    # per run: (stem 100 + conv 300) KiB, scaled
    assert doc["conv_fetch_bytes_per_step"] == 400 * 1024 * 2
    assert doc["conv_write_bytes_per_step"] == 400 * 1024 // 2
    assert json.loads(out.read_text())["runs_counted"] == 2
