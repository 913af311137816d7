"""The benchmark's host-side summaries (no GPU): HBM traffic per FC1
weight-gradient launch from FETCH_SIZE / WRITE_SIZE runs scaled by the 1 GiB
calibration pass, and the per-GEMM MFMA table, on small hand-made counter
files in rocprofv3's CSV layout; the clock sampler's summary."""
import csv
import json

import pytest

import bench

COLS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
        "End_Timestamp"]
NEG = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(...)>"
CFG = "memfine::(anonymous namespace)::Cfg<256, 256, 2, 4, 2, 128, 3>"


def wgrad_name(acc):
    return ("void memfine::(anonymous namespace)::grouped_gemm_split_kernel<unsigned short, "
            f"{CFG}, memfine::(anonymous namespace)::ProbWgrad<unsigned short, {CFG}, true, {acc}> >")


def write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=COLS)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def row(i, name, ctr, val, t0=0, t1=1000):
    return {"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": ctr, "Counter_Value": val,
            "Start_Timestamp": t0, "End_Timestamp": t1}


def test_traffic_summary(tmp_path):
    # calibration: FETCH_SIZE reads half of the 1 GiB (scale 2), WRITE_SIZE all of it
    fetch = [row(1, NEG, "FETCH_SIZE", 524288.0),
             row(2, wgrad_name(0), "FETCH_SIZE", 1000.0), row(3, wgrad_name(0), "FETCH_SIZE", 3000.0),
             row(4, wgrad_name(1), "FETCH_SIZE", 5000.0),
             row(5, "void other_kernel", "FETCH_SIZE", 9e9)]
    write = [row(1, NEG, "WRITE_SIZE", 1048576.0),
             row(2, wgrad_name(0), "WRITE_SIZE", 100.0), row(3, wgrad_name(0), "WRITE_SIZE", 300.0),
             row(4, wgrad_name(1), "WRITE_SIZE", 700.0)]
    write_csv(tmp_path / "FETCH_SIZE_counter_collection.csv", fetch)
    write_csv(tmp_path / "WRITE_SIZE_counter_collection.csv", write)
    out = tmp_path / "traffic.json"
    d = bench.summarize_traffic(str(tmp_path), 2, path=str(out))
    # per kernel means (KiB x 1024 x scale); the per-launch figure is the
    # mean over all profiled launches (the dW modes as often as a step runs
    # them: here two launches that write dW and one that accumulates)
    f0, f1 = 2000.0 * 1024 * 2, 5000.0 * 1024 * 2
    w0, w1 = 200.0 * 1024, 700.0 * 1024
    assert d["fetch_bytes_per_launch"] == pytest.approx((2 * f0 + f1) / 3)
    assert d["write_bytes_per_launch"] == pytest.approx((2 * w0 + w1) / 3)
    assert d["bytes_per_launch"] == pytest.approx((2 * (f0 + w0) + f1 + w1) / 3)
    per = sorted(d["per_kernel"].values(), key=lambda e: e["launches"])
    assert per[0]["fetch_bytes"] == pytest.approx(f1) and per[1]["fetch_bytes"] == pytest.approx(f0)
    assert d["launches_profiled"] == 3
    assert d["source_sha256_16"] == bench.source_digest("grouped_gemm.hip")
    assert json.loads(out.read_text())["bytes_per_launch"] == pytest.approx(d["bytes_per_launch"])


def test_traffic_summary_needs_one_calibration(tmp_path):
    write_csv(tmp_path / "FETCH_SIZE_counter_collection.csv", [row(2, wgrad_name(0), "FETCH_SIZE", 1.0)])
    write_csv(tmp_path / "WRITE_SIZE_counter_collection.csv", [row(2, wgrad_name(0), "WRITE_SIZE", 1.0)])
    with pytest.raises(SystemExit):
        bench.summarize_traffic(str(tmp_path), 2, path=str(tmp_path / "x.json"))


def test_mfma_summary(tmp_path):
    fc1 = ("void memfine::(anonymous namespace)::grouped_gemm_split_kernel<unsigned short, "
           f"{CFG}, memfine::(anonymous namespace)::ProbFC1<unsigned short, {CFG}, false> >")
    # one dispatch of 100 us: 8 XCDs x 1000 GUI cycles, busy 512000 SIMD-cycles
    rows = [row(7, fc1, "GRBM_GUI_ACTIVE", 8000.0, 0, 100000),
            row(7, fc1, "SQ_VALU_MFMA_BUSY_CYCLES", 512000.0, 0, 100000),
            row(7, fc1, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e9, 0, 100000),
            row(8, NEG, "GRBM_GUI_ACTIVE", 5.0)]
    path = tmp_path / "mfma.csv"
    write_csv(path, rows)
    agg = bench.summarize_mfma(str(path))
    assert list(agg) == ["fc1"]
    a = agg["fc1"]
    assert a["util"] == pytest.approx(512000.0 / (1000.0 * 1024.0))
    assert a["tflops"] == pytest.approx(1e9 * 512 / 100e-6 / 1e12)


def test_clock_sampler_summary():
    """The clock summary: None without samples (no amdsmi, no GPU) or over a
    timed region shorter than the sampler's minimum, else the mean, range
    and count of the sampled MHz values in GHz."""
    c = bench.ClockSampler()
    assert c.summary() is None
    c.samples = [1800.0, 1700.0, 1600.0]
    c.seconds = 0.3
    assert c.summary() is None
    c.seconds = 5.0
    s = c.summary()
    assert s["mean_ghz"] == pytest.approx(1.7) and s["min_ghz"] == pytest.approx(1.6)
    assert s["max_ghz"] == pytest.approx(1.8) and s["samples"] == 3


def test_clock_sampler_without_gpu_ends():
    """On a host without a GPU the sampler thread ends at once and the timed
    block runs as usual."""
    import time
    with bench.ClockSampler() as c:
        time.sleep(0.05)
    assert not c._thread.is_alive() or c.summary() is None


def test_more_than_one_gpu_is_refused():
    """bench.py --gpus 2 exits with status 2 and says why, before any GPU
    work."""
    import os
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.abspath(bench.__file__), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
