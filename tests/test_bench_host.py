"""Host-only checks of bench.py's contract (no GPU needed)."""
import json
import os
import subprocess
import sys

import bench
from paper_2309_15812_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_algorithmic_bytes_of_the_step():
    wl = synth.WORKLOADS["metric"]
    T = 64 * 96 * 56 * 56 * 4
    b = bench.algorithmic_bytes(wl)
    assert T == 77070336
    assert b["fwd"] == 2 * T and b["bwd_input"] == 2 * T
    assert b["bwd"] == 3 * T + 96 * 31 * 4           # reads x and dy, writes dx and dw
    assert b["bwd_weight"] == 2 * T + 96 * 31 * 4
    assert b["fwd"] + b["bwd"] == 385363584           # the step: 5T + C*K*4
    bf = bench.algorithmic_bytes(synth.WORKLOADS["c4"])
    assert bf["fwd"] == 2 * 64 * 384 * 14 * 14 * 2   # bfloat16 storage


def test_traffic_is_used_only_for_the_current_kernel_sources(tmp_path, monkeypatch):
    rec = {"kernel_source_hash": bench.kernel_source_hash(), "ops": {"bwd": {"hbm_bytes_per_launch": 123}}}
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.traffic_for("bwd") == 123
    assert bench.traffic_for("fwd") is None
    rec["kernel_source_hash"] = "0" * 16
    f.write_text(json.dumps(rec))
    assert bench.traffic_for("bwd") is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.json"))
    assert bench.traffic_for("bwd") is None


def test_every_workload_angle_mode_is_described():
    for wl in synth.WORKLOADS.values():
        assert wl.theta in bench.THETA_TEXT, wl.theta
