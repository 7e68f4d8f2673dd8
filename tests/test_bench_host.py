"""Host logic of bench.py on the CPU: the algorithmic flop counts per pair,
the traffic record (read back only for the kernel sources it was taken on,
scaled by the calibration copy), the exponential-rate figures, and the
refusal of more than one GPU."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_flops_per_pair():
    D, C = 64, 1
    assert bench.flops_per_pair(("fwd",), D, C, False) == 2 * D + 2 * C
    assert bench.flops_per_pair(("fwd", "dq"), D, C, True) == 4 * D + 4 * C
    assert bench.flops_per_pair(("fwd", "dq"), D, C, False) == (2 * D + 2 * C) + (4 * D + 2 * C)
    assert bench.flops_per_pair(("fwd", "dq", "dk", "dv"), 128, 128, True) == (
        (4 * 128 + 4 * 128) + (4 * 128 + 2 * 128) + (2 * 128 + 2 * 128))


def _write_counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, val in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": val})


def test_traffic_record_roundtrip(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "traffic_file", lambda w: str(tmp_path / ("traffic_%s.json" % w)))
    copy = 512 << 20
    fetch, write = str(tmp_path / "fetch"), str(tmp_path / "write")
    # the copy kernel reads half of its bytes in counter units (scale 2), the
    # dominant kernel's mean over dispatches is taken (as for its launch time)
    _write_counters(fetch, "FETCH_SIZE", [("void gs::k_dq<x>", 100.0), ("void gs::k_dq<x>", 400.0),
                                          ("void gs::k_dq<x>", 100.0), ("elementwise_copy_kernel", copy / 2048.0)])
    _write_counters(write, "WRITE_SIZE", [("void gs::k_dq<x>", 50.0), ("elementwise_copy_kernel", copy / 1024.0)])
    bench.traffic_from("wl", fetch, write, copy, "k_dq")
    rec = json.load(open(tmp_path / "traffic_wl.json"))
    assert rec["fetch"]["counter_kib_per_launch"] == 200.0
    assert rec["fetch"]["scale"] == pytest.approx(2.0)
    assert rec["bytes_per_launch"] == pytest.approx(200.0 * 1024 * 2 + 50.0 * 1024)
    assert bench.recorded_traffic("wl", "k_dq") == pytest.approx(rec["bytes_per_launch"])
    assert bench.recorded_traffic("wl", "k_fwd") is None           # another kernel
    rec["kernel_sources_sha256"] = "0" * 64                        # other sources
    json.dump(rec, open(tmp_path / "traffic_wl.json", "w"))
    assert bench.recorded_traffic("wl", "k_dq") is None


def test_exp_rate_and_measured_fractions(monkeypatch):
    monkeypatch.setattr(bench, "measured_peaks", lambda: {"exp2_per_s": 1.0e13,
                                                           "mfma_f16_16x16x32_flop_per_s": 2.0e15})
    e = bench.exp_rate(4.0e9, 1.0)            # 4e9 exponentials in 1 ms
    assert e["achieved"] == pytest.approx(4.0e12)
    assert e["frac_measured"] == pytest.approx(0.4)
    assert e["frac_nominal"] == pytest.approx(4.0e12 / (256 * 4 * 8 * 2.4e9))
    m = bench.measured_mfma(1000.0)           # TFLOP/s
    assert m["peak_measured"] == pytest.approx(2000.0) and m["frac_of_measured"] == pytest.approx(0.5)
    monkeypatch.setattr(bench, "measured_peaks", lambda: None)
    assert "peak_measured" not in bench.exp_rate(1.0, 1.0) and bench.measured_mfma(1.0) == {}


def test_committed_records_are_readable():
    pk = bench.measured_peaks()
    assert pk is not None and pk["mfma_f16_16x16x32_flop_per_s"] > 1e15 and pk["exp2_per_s"] > 1e13


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr + r.stdout


def test_algorithmic_step_flops():
    # forward alone, forward + dq on shared tiles, forward + full backward
    assert bench.algorithmic_flops_per_pair(("fwd",), 16, 1) == 2 * 16 + 2
    assert bench.algorithmic_flops_per_pair(("fwd", "dq"), 64, 1) == 4 * 64 + 4
    assert bench.algorithmic_flops_per_pair(("fwd", "dq", "dk", "dv"), 256, 16) == 8 * 256 + 6 * 16
    assert bench.algorithmic_flops_per_pair(("dq",), 64, 8) == 4 * 64 + 2 * 8
    assert bench.algorithmic_flops_per_pair(("dv",), 64, 8) == 2 * 64 + 2 * 8


def test_dominant_launch_flops_follow_the_fusion_rule():
    # D = 256, C = 16: forward fused into dq, dv into dk; 4D+4C each
    assert bench.dominant_flops(("fwd", "dq", "dk", "dv"), 256, 16, True) == 4 * 256 + 4 * 16
    # separate calls: the forward has its own pass, dv still rides in dk
    assert bench.dominant_flops(("fwd", "dq", "dk", "dv"), 256, 16, False) == 4 * 256 + 3 * 16
    # C = 128: nothing fused; dq and dk launches 4D+2C each
    assert bench.dominant_flops(("fwd", "dq", "dk", "dv"), 128, 128, True) == 4 * 128 + 2 * 128
    # single channel: forward fused into dq, dv into dk
    assert bench.dominant_flops(("fwd", "dq"), 64, 1, True) == 4 * 64 + 4
    assert bench.dominant_flops(("fwd", "dq"), 64, 1, False) == 4 * 64 + 2
    assert bench.dominant_flops(("fwd",), 32, 4, False) == 2 * 32 + 2 * 4


def test_sub_record_fields(monkeypatch):
    monkeypatch.setattr(bench, "measured_peaks", lambda: {"exp2_per_s": 1.0e13})
    res = {"config": {"workload": "mixture_d32: ...", "M": 1024, "N": 2048, "D": 32, "C": 4, "tau": 1.0,
                      "passes": "fwd", "api": "gauss_sum_fwd"},
           "steps": 5, "ms_per_step": 2.0, "value": 1024 * 2048 / 2e-3,
           "step_roofline": {"frac": 0.1},
           "roofline": {"kernel": "k_fwd", "avg_launch_ms": 1.0, "frac": 0.2, "exp": {"achieved": 1024 * 2048 / 1e-3}}}
    r = bench.sub_record(res)
    assert r["workload"] == "mixture_d32"
    assert r["exp_per_s_step"] == pytest.approx(1024 * 2048 / 2e-3)
    assert r["step_frac_of_measured_exp_rate"] == pytest.approx(1024 * 2048 / 2e-3 / 1e13)
    assert r["kernel_frac_of_measured_exp_rate"] == pytest.approx(1024 * 2048 / 1e-3 / 1e13)
