"""The measurement side of ``bench.py`` on the CPU: the summaries that turn rocprofv3
output into the committed profiles, the algorithmic FLOP count behind the roofline
fraction, the rule-to-threshold mapping, and the refusal of more than one GPU.

The rocprofv3 inputs are small CSV files written here with the columns rocprofv3 writes,
and every expected figure is worked out by hand.
"""

import csv
import json
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RULE = "void dsattn::(anonymous namespace)::fa_fwd_kernel<2, 128, 0, false, 64>(dsattn::FwdParams)"
DENSE = "void dsattn::(anonymous namespace)::fa_fwd_kernel<0, 128, 0, false, 64>(dsattn::FwdParams)"
COPY = "void at::native::vectorized_elementwise_kernel<4, at::native::AUnaryFunctor<float>>"


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh, quoting=csv.QUOTE_ALL)
        w.writerow(header)
        w.writerows(rows)


def _counters(d, rows):
    _write(os.path.join(d, "run", "run_counter_collection.csv"),
           ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], rows)


def test_algorithmic_flops_counts_qk_always_and_pv_when_kept():
    # two heads: 1000 valid elements of which 250 skipped, and 600 with none skipped
    st = np.array([[10, 3, 1000, 250], [8, 0, 600, 0]])
    d = 128
    assert bench.algorithmic_flops(st, d) == 2 * d * 1600 + 2 * d * (1600 - 250)
    # a reused mask skips QK^T of the skipped elements as well
    assert bench.algorithmic_flops(st, d, reuse=True) == 2 * 2 * d * (1600 - 250)


def test_oracle_threshold_maps_each_rule_to_natural_log():
    N = 75600
    assert bench.oracle_threshold("dense", 0.0, N) == ("dense", 0.0)
    assert bench.oracle_threshold("blasst", 1e-2, N) == ("blasst", math.log(1e-2))
    name, lam = bench.oracle_threshold("dynsparse_recall", 0.95, N)
    assert name == "dynsparse" and lam == pytest.approx(math.log(0.05 / N))
    assert bench.oracle_threshold("dynsparse_recall", 1.0, N)[1] == -math.inf
    assert bench.oracle_threshold("dynsparse_lambda", -6.0, N) == ("dynsparse", -6.0)


def test_counter_summary_ratios(tmp_path):
    # last dispatch of each counter is used; 8 dies, 1024 SIMDs
    gui = 8 * 1.0e8                      # 1e8 cycles
    busy = 0.5 * 1024 * 1.0e8            # busy on half the cycles
    _counters(str(tmp_path / "a"), [
        [1, RULE, "GRBM_GUI_ACTIVE", 1.0],
        [2, RULE, "GRBM_GUI_ACTIVE", gui],
        [2, RULE, "SQ_WAVE_CYCLES", 4000.0],
        [2, RULE, "SQ_ACTIVE_INST_VALU", 1000.0],
        [2, DENSE, "SQ_WAVE_CYCLES", 10.0],
        [2, COPY, "SQ_WAVE_CYCLES", 99.0],
    ])
    _counters(str(tmp_path / "b"), [
        [2, RULE, "SQ_VALU_MFMA_BUSY_CYCLES", busy],
        [2, RULE, "SQ_INSTS_MFMA", 100.0],
        [2, RULE, "SQ_INSTS_VALU", 560.0],
    ])
    text = bench.counter_summary([str(tmp_path / "a"), str(tmp_path / "b")], "cmd")
    assert "# command: cmd" in text
    assert "fa_fwd_kernel<dynsparse>" in text and "fa_fwd_kernel<dense>" in text
    assert "AUnaryFunctor" not in text
    lines = text.splitlines()
    assert any("MFMA busy per SIMD per cycle" in l and l.rstrip().endswith("0.500") for l in lines)
    assert any("SQ_ACTIVE_INST_VALU" in l and "per wave cycle 0.250" in l for l in lines)
    assert any("SQ_INSTS_VALU " in l and "per MFMA 5.600" in l for l in lines)


def test_traffic_summary_scales_by_the_copy(tmp_path, monkeypatch):
    gib_kib = float(1 << 20)
    # the copy moves 1 GiB: FETCH_SIZE reads half of it, WRITE_SIZE all of it
    _counters(str(tmp_path / "f"), [
        [1, COPY, "FETCH_SIZE", 0.5 * gib_kib],
        [2, RULE, "FETCH_SIZE", 1000.0],
        [3, RULE, "FETCH_SIZE", 3000.0],
        [4, RULE, "FETCH_SIZE", 2000.0],
        [5, DENSE, "FETCH_SIZE", 7.0e9],
    ])
    _counters(str(tmp_path / "w"), [
        [1, COPY, "WRITE_SIZE", gib_kib],
        [2, RULE, "WRITE_SIZE", 100.0],
    ])
    rec = bench.traffic_summary(str(tmp_path / "f"), str(tmp_path / "w"), "wl", "cmd")
    assert rec["fetch_counter_per_copy_byte"] == pytest.approx(0.5)
    assert rec["write_counter_per_copy_byte"] == pytest.approx(1.0)
    assert rec["fetch_bytes"] == pytest.approx(2000.0 * 1024 / 0.5)     # median, rescaled
    assert rec["write_bytes"] == pytest.approx(100.0 * 1024)
    assert rec["bytes_per_launch"] == pytest.approx(rec["fetch_bytes"] + rec["write_bytes"])
    assert rec["dispatches"] == [3, 1]
    assert rec["kernel_sha256"] == bench.kernel_source_digest()


def test_measured_traffic_only_for_the_source_it_measured(tmp_path, monkeypatch):
    path = tmp_path / "hbm_traffic_wl_t.json"
    monkeypatch.setattr(bench, "traffic_path", lambda workload, tag="": str(path))
    assert bench.measured_traffic("wl", "t") is None                 # no record
    path.write_text(json.dumps({"bytes_per_launch": 5.0, "kernel_sha256": "not this source"}))
    assert bench.measured_traffic("wl", "t") is None                 # another kernel
    path.write_text(json.dumps({"bytes_per_launch": 5.0,
                                "kernel_sha256": bench.kernel_source_digest()}))
    assert bench.measured_traffic("wl", "t") == 5.0


def test_traffic_record_names():
    assert bench.traffic_path("wan720p").endswith(os.path.join("profiles",
                                                               "hbm_traffic_wan720p.json"))
    assert bench.traffic_path("wan720p", "lam6").endswith("hbm_traffic_wan720p_lam6.json")


def test_trace_summary_splits_one_run_per_configuration(tmp_path):
    d = str(tmp_path)
    _write(os.path.join(d, "run", "run_kernel_stats.csv"),
           ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"],
           [[RULE, 6, 600e6, 100e6, 60.0], [DENSE, 3, 300e6, 100e6, 40.0]])
    header = ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Scratch_Size",
              "LDS_Block_Size", "Workgroup_Size_X", "Grid_Size_X", "Grid_Size_Y"]
    rows, t = [], 0

    def launch(name, ms, grid_x=591 * 256):
        nonlocal t
        rows.append([name, t, t + int(ms * 1e6), 0, 66560, 256, grid_x, 40])
        t += int(ms * 1e6) + 1000

    for _ in range(3):
        launch(DENSE, 96.0)
    for _ in range(3):
        launch(RULE, 99.0)              # recall target: nothing skipped
    for _ in range(3):
        launch(RULE, 68.0)              # a threshold that skips: a new run
    launch(RULE, 68.5)                  # within 4 %: same run
    launch(RULE, 68.0, grid_x=256 * 256)  # another shape: a new run
    _write(os.path.join(d, "run", "run_kernel_trace.csv"), header, rows)
    text = bench.trace_summary(d, "cmd")
    runs = [l.split() for l in text.splitlines() if l[:4].strip().isdigit() and "fa_fwd" in l]
    assert [(int(r[1]), float(r[2])) for r in runs] == [
        (3, 96.0), (3, 99.0), (4, pytest.approx(68.125)), (1, 68.0)]
    assert [r[4] for r in runs] == ["591x40", "591x40", "591x40", "256x40"]
    assert all(r[5] == "0" and r[6] == "66560" for r in runs)


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""
