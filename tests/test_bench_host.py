"""Host-side logic of bench.py (no GPU): the one-GPU guard, and the rocprofv3 summaries it turns
into the committed traffic and clock records (copy-calibrated FETCH_SIZE / WRITE_SIZE per head
launch; cycles, clock and MFMA busy per head dispatch), written to a temporary directory."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writerows(rows)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_record_scales_by_the_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    dirs = {n: tmp_path / n for n in ("hf", "hw", "cf", "cw")}
    for d in dirs.values():
        d.mkdir()
    # Two head dispatches, counters split over two instances each; the copy reads 1 GiB counted
    # as half (scale 2) and writes it counted in full (scale 1).
    _counters(dirs["hf"] / "p_counter_collection.csv",
              [[1, "head_bf16_pp_kernel", "FETCH_SIZE", 600.0], [1, "head_bf16_pp_kernel", "FETCH_SIZE", 400.0],
               [2, "head_bf16_pp_kernel", "FETCH_SIZE", 1000.0], [3, "sample_tiles_kernel", "FETCH_SIZE", 7.0]])
    _counters(dirs["hw"] / "p_counter_collection.csv",
              [[1, "head_bf16_pp_kernel", "WRITE_SIZE", 300.0], [2, "head_bf16_pp_kernel", "WRITE_SIZE", 500.0]])
    _counters(dirs["cf"] / "p_counter_collection.csv",
              [[9, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 524288.0]])
    _counters(dirs["cw"] / "p_counter_collection.csv",
              [[9, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 1048576.0]])
    bench._write_traffic(str(dirs["hf"]), str(dirs["hw"]), str(dirs["cf"]), str(dirs["cw"]),
                         1 << 30, "qwen3_8b")
    rec = json.loads((tmp_path / "traffic.json").read_text())
    assert rec["fetch_kib_per_launch"] == 1000.0 and rec["write_kib_per_launch"] == 400.0
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["hbm_bytes_per_launch"] == 1000.0 * 1024 * 2 + 400.0 * 1024
    assert rec["head_source_sha256_16"] == bench._head_source_hash()
    assert bench._traffic("qwen3_8b") == rec["hbm_bytes_per_launch"]
    assert bench._traffic("qwen3_4b") is None  # taken on another workload
    rec["head_source_sha256_16"] = "0" * 16
    (tmp_path / "traffic.json").write_text(json.dumps(rec))
    assert bench._traffic("qwen3_8b") is None  # taken on another head source


def test_clock_record_from_counters_and_trace(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "CLOCK_FILE", str(tmp_path / "clock.json"))
    d = tmp_path / "pmc"
    (d / "sub").mkdir(parents=True)
    # Dispatch 1 is the warm-up (left out); 2 and 3: 8 XCDs x 2.0e6 cycles over 1.25 ms
    # = 1.6 GHz, MFMA busy 0.75 of 1024 SIMDs.
    rows = []
    for i in (1, 2, 3):
        rows += [[i, "head_bf16_pp_kernel", "GRBM_GUI_ACTIVE", 8 * 2.0e6],
                 [i, "head_bf16_pp_kernel", "SQ_VALU_MFMA_BUSY_CYCLES", 0.75 * 1024 * 2.0e6]]
    _counters(d / "sub" / "p_counter_collection.csv", rows)
    with open(d / "sub" / "p_kernel_trace.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writerow([1, "head_bf16_pp_kernel", 0, 9_000_000])
        w.writerow([2, "head_bf16_pp_kernel", 10_000_000, 11_250_000])
        w.writerow([3, "head_bf16_pp_kernel", 20_000_000, 21_250_000])
        w.writerow([4, "sample_tiles_kernel", 30_000_000, 30_050_000])
    bench._write_clock(str(d), "qwen3_8b")
    rec = json.loads((tmp_path / "clock.json").read_text())
    assert rec["dispatches"] == 2
    assert rec["cycles"] == pytest.approx(2.0e6)
    assert rec["clock_ghz"] == pytest.approx(1.6)
    assert rec["mfma_busy"] == pytest.approx(0.75)
    assert rec["head_us"] == pytest.approx(1250.0)
    assert bench._clock("qwen3_8b")["clock_ghz"] == pytest.approx(1.6)
