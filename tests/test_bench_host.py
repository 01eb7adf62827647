"""Host logic of bench.py on the CPU: the one-GPU guard, the counter arithmetic that turns two
rocprofv3 --pmc CSVs into per-launch HBM bytes, the stored-traffic hash check and the roofline
fractions."""
from __future__ import annotations

import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def _csv(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_write_traffic_scales_by_the_copy(tmp_path, monkeypatch):
    # the copy of the 54.4 MB feature matrix reads half its KiB under FETCH_SIZE (factor 2) and
    # writes all of them (factor 1); the scoring dispatches' mean is scaled by the same factors
    copy_kib = 100_000 * 136 * 4 / 1024
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [("__amd_rocclr_copyBuffer", copy_kib / 2),
                                             ("score_kernel<64, 4, true, true, false, 0>", 30000.0),
                                             ("score_kernel<64, 4, true, true, false, 0>", 32000.0),
                                             ("reduce_partials_thread_kernel", 7.0)])
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", copy_kib),
                                             ("score_kernel<64, 4, true, true, false, 0>", 600.0)])
    out = tmp_path / "traffic.json"
    assert bench.write_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "rank_1kx32", str(out)) == 0
    rec = json.loads(out.read_text())
    ent = rec["workloads"]["rank_1kx32"]
    assert ent["calibration"]["fetch_factor"] == pytest.approx(2.0)
    assert ent["hbm_read_bytes_per_launch"] == round(31000.0 * 1024 * 2)
    assert ent["hbm_write_bytes_per_launch"] == round(600.0 * 1024)
    assert rec["kernel_hash"] == bench.kernel_hash()
    # the stored figure is used only while the kernel sources hash the same
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    assert bench.load_traffic("rank_1kx32") == ent["hbm_bytes_per_launch"]
    # a second workload's entry is added beside the first
    copy5 = 1_000_000 * 700 * 4 / 1024
    _csv(tmp_path / "f5.csv", "FETCH_SIZE", [("__amd_rocclr_copyBuffer", copy5 / 2),
                                              ("score_kernel<64, 1, false, false, true, 0>", 1e6)])
    _csv(tmp_path / "w5.csv", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", copy5),
                                              ("score_kernel<64, 1, false, false, true, 0>", 4000.0)])
    assert bench.write_traffic(str(tmp_path / "f5.csv"), str(tmp_path / "w5.csv"), "large_5kx256_f700_1M",
                               str(out)) == 0
    rec = json.loads(out.read_text())
    assert set(rec["workloads"]) == {"rank_1kx32", "large_5kx256_f700_1M"}
    assert bench.load_traffic("large_5kx256_f700_1M") == round(1e6 * 1024 * 2) + round(4000.0 * 1024)
    rec["kernel_hash"] = "0" * 16
    out.write_text(json.dumps(rec))
    assert bench.load_traffic("rank_1kx32") is None


def test_roofline_fractions():
    rl, rl_hbm, rl_issue = bench.roofline(1e-3, 157.2864e9 / 2, 8e9 / 4, None)
    assert rl["frac"] == pytest.approx(0.5, abs=1e-4) and rl["bound"] == "lds"
    assert rl_hbm["frac"] == pytest.approx(0.25, abs=1e-4)
    assert rl_issue["peak"] == pytest.approx(256 * 2.4e9 * 512 / 4.4 / 1e9, rel=1e-6)
