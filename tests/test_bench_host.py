"""Host-side logic of bench.py (CPU only): the algorithmic bytes and FLOPs behind the roofline,
the choice of the dominant kernel and its bound, the measured-traffic lookup keyed by the
kernel sources, and the single-GPU contract."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2208_05419_amd import synth  # noqa: E402


def test_algorithmic_work_of_the_headline():
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    w = bench.algorithmic_work(wl, 2)
    x = 4 * 90 * 180 * 768 * 2                  # bf16 fields
    s = 4 * 90 * 91 * 768 * 2 * 2               # kept half spectrum, complex bf16
    assert w["row_r2c"]["bytes"] == x + s
    assert w["column"]["bytes"] == 2 * s
    assert w["row_c2r"]["bytes"] == s + 2 * x
    # two complex layers of 96 x 96 per block and mode, 8 real FLOP per complex MAC
    assert w["column"]["flops"] == 8 * 2 * 96 * 96 * 8 * 4 * 90 * 91
    assert w["row_r2c"]["flops"] == w["row_c2r"]["flops"] == 0


def test_algorithmic_work_counts_only_kept_modes():
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_ens100_keep0.5"]
    w = bench.algorithmic_work(wl, 2)
    # keep 0.5: 45 kept columns of 91 and 45 kept rows of 90 (|signed k| < 23)
    s = 100 * 90 * 45 * 768 * 4
    assert w["column"]["bytes"] == 2 * s
    assert w["column"]["flops"] == 16 * 768 * 96 * 100 * 45 * 45


def test_roofline_takes_the_slowest_kernel_and_its_bound():
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    ms = {"prep": 0.0, "row_r2c": 0.0355, "column": 0.0922, "row_c2r": 0.0483}
    roof, per = bench.roofline(wl, ms, 2)
    work = bench.algorithmic_work(wl, 2)
    assert roof["kernel"] == "column"
    # 201 MB at 8 TB/s (25 us) outlasts 38.6 GFLOP at 2.5 PFLOP/s (15.5 us): HBM-bound
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    gbs = work["column"]["bytes"] / 0.0922e-3 / 1e9
    assert roof["achieved"] == pytest.approx(gbs, rel=1e-4)
    assert roof["frac"] == pytest.approx(gbs / 8000.0, abs=1e-4)
    # a preparation inside the W-axis launch: its bytes move to that launch's row
    assert per["prep"]["folded_into"] == "row_r2c"
    assert per["row_r2c"]["bytes"] == work["row_r2c"]["bytes"] + work["prep"]["bytes"]


def test_roofline_of_an_arithmetic_bound_kernel():
    # fp32 storage: 9.7 GFLOP against 157.3 TFLOP/s (61 us) outlasts 100 MB at 8 TB/s (13 us)
    wl = synth.WORKLOADS["afno90x180_c768_nb8_fp32"]
    roof, _ = bench.roofline(wl, {"prep": 0.0, "row_r2c": 0.02, "column": 0.1, "row_c2r": 0.03}, 4)
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == 157.3


def test_measured_traffic_only_for_the_sources_it_was_taken_on(tmp_path, monkeypatch):
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    ms = {"prep": 0.0, "row_r2c": 0.0355, "column": 0.0922, "row_c2r": 0.0483}
    f = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    f.write_text(json.dumps({"source_sha256": bench.kernel_source_hash(),
                             "kernels": {"column": {"hbm_bytes_per_launch": 123}}}))
    assert bench.roofline(wl, ms, 2)[0]["traffic"] == 123
    f.write_text(json.dumps({"source_sha256": "0" * 64,
                             "kernels": {"column": {"hbm_bytes_per_launch": 123}}}))
    assert bench.roofline(wl, ms, 2)[0]["traffic"] is None
    f.unlink()
    assert bench.roofline(wl, ms, 2)[0]["traffic"] is None


def test_only_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr
