"""Host logic of the measurement tools (no GPU): bench.py runs on one GPU only; the
HBM traffic that bench.py reports comes from the committed counter record only while
the expert GEMM sources hash to the recorded value; the counter summaries turn
rocprofv3 CSV output into per-launch bytes and per-dispatch matrix work."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_runs_on_one_gpu_only():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _record(workload):
    path = os.path.join(ROOT, "profiles", f"expert_gemm_{workload}_traffic.md")
    with open(path) as f:
        line = next(x for x in f if x.startswith("traffic-json:"))
    return json.loads(line.split(":", 1)[1])


@pytest.mark.parametrize("workload", ["irregular", "shard", "small"])
def test_traffic_record_is_used_only_for_its_sources(monkeypatch, workload):
    from paper_2604_15821_amd import counters
    rec = _record(workload)
    assert len(rec["sources_sha256"]) == 64 and rec["launches_counted"] > 0
    assert rec["fetch_bytes_per_launch"] > 0 and rec["write_bytes_per_launch"] > 0
    monkeypatch.setattr(counters, "kernel_sources_sha256", lambda: rec["sources_sha256"])
    assert counters.measured_traffic(workload) == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
    monkeypatch.setattr(counters, "kernel_sources_sha256", lambda: "0" * 64)
    assert counters.measured_traffic(workload) is None
    assert counters.measured_traffic("no_such_workload") is None


def _write_counters(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    cols = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(cols, r)))


def test_mfma_summary_arithmetic(tmp_path):
    """Two dispatches of one product, 2 ms each: 512 x MOPS FLOP, busy cycles over
    (GRBM_GUI_ACTIVE / 8) x 1024 SIMDs, clock from GRBM_GUI_ACTIVE / 8."""
    from paper_2604_15821_amd import counters
    name = "void janus::gemm_rows_kernel<false, janus::LoadPlain, janus::EpiStore>(int)"
    gui = 8 * 2.2e9 * 2e-3                       # 2.2 GHz on each of 8 XCDs for 2 ms
    busy = 0.75 * (gui / 8) * 1024               # 75 % of the SIMD cycles
    mops = 250e12 * 2e-3 / 512                   # 250 TFLOP/s of executed work
    rows = []
    for k in (1, 2):
        t0 = k * 10_000_000
        for cname, v in (("SQ_INSTS_VALU_MFMA_MOPS_F32", mops), ("SQ_VALU_MFMA_BUSY_CYCLES", busy),
                         ("GRBM_GUI_ACTIVE", gui)):
            rows.append((k, name, cname, v, t0, t0 + 2_000_000))
    _write_counters(str(tmp_path / "tr_m_toy" / "run_counter_collection.csv"), rows)
    text = counters.mfma_summary("toy", str(tmp_path))
    line = next(x for x in text.splitlines() if "gemm_rows_kernel" in x)
    cells = [c.strip() for c in line.strip("|").split("|")]
    assert cells[1] == "2"                          # dispatches
    assert float(cells[2]) == pytest.approx(2000.0)  # avg us
    assert float(cells[3]) == pytest.approx(500.0)   # executed GFLOP per dispatch
    assert float(cells[4]) == pytest.approx(250.0)   # TFLOP/s
    assert float(cells[5]) == pytest.approx(0.75)    # busy
    assert float(cells[6]) == pytest.approx(2.2)     # GHz


def test_traffic_summary_scales_by_the_copy_kernel(tmp_path):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) scaled so that the 1 GiB copy kernel
    reads and writes exactly 1 GiB."""
    from paper_2604_15821_amd import counters
    wl = "toy"
    copy = "void at::native::vectorized_elementwise_kernel<4>(int)"
    prod = "void janus::gemm_rows_kernel<true, janus::LoadPlain, janus::EpiStore>(int)"
    # the copy reads half of what the counter reports as fetched; writes are exact
    _write_counters(str(tmp_path / f"tr_f_{wl}" / "run_counter_collection.csv"),
                    [(1, copy, "FETCH_SIZE", 2 * 1048576.0, 0, 1), (2, prod, "FETCH_SIZE", 2 * 1000.0, 2, 3),
                     (3, prod, "FETCH_SIZE", 2 * 3000.0, 4, 5)])
    _write_counters(str(tmp_path / f"tr_w_{wl}" / "run_counter_collection.csv"),
                    [(1, copy, "WRITE_SIZE", 1048576.0, 0, 1), (2, prod, "WRITE_SIZE", 500.0, 2, 3),
                     (3, prod, "WRITE_SIZE", 700.0, 4, 5)])
    trace = tmp_path / f"tr_k_{wl}"
    trace.mkdir()
    with open(trace / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writerow([prod, 0, 1_000_000])
        w.writerow([prod, 2_000_000, 5_000_000])
    with open(trace / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"])
        w.writerow([prod, 2, 4_000_000, 2_000_000, 100.0])
    text = counters.summarize(wl, str(tmp_path))
    rec = json.loads(next(x for x in text.splitlines() if x.startswith("traffic-json:")).split(":", 1)[1])
    assert rec["fetch_scale"] == pytest.approx(0.5) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["launches_counted"] == 2
    assert rec["fetch_bytes_per_launch"] == pytest.approx(2000.0 * 1024)   # (1000 + 3000) KiB / 2
    assert rec["write_bytes_per_launch"] == pytest.approx(600.0 * 1024)
    row = next(x for x in text.splitlines() if x.startswith("| expert_gemm"))
    assert "| 2000.0 |" in row                                               # average of 1 ms and 3 ms
