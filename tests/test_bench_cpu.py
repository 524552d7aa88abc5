"""bench.py's command-line contract and its use of the committed counters,
checked on the CPU (no GPU needed)."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_defaults(monkeypatch):
    import bench
    monkeypatch.setattr(sys, "argv", ["bench.py"])
    a = bench.parse()
    assert (a.gpus, a.steps, a.warmup, a.workload) == (1, 20, 5, 2)
    assert not a.graph and not a.block and not a.fno


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_counters_resolve_for_the_default_workload():
    import bench
    with open(os.path.join(ROOT, "profiles", "hbm_counters.json")) as f:
        c = json.load(f)
    assert set(c["workloads"]) >= {"2", "5"}
    for role in c["workloads"]["2"]["kernels"]:
        t = bench.traffic_entry(2, role)
        # None only when the kernel's source changed after the counters were taken
        if t is not None:
            assert t > 0
    fwd = bench.traffic_entry(2, "stream_fwd_tzy")
    if fwd is None:
        pytest.skip("fused forward source changed since the counters were taken")
    # the 128^3 x 32 slab of 16: 537 MB read + 16.8 MB written, algorithmically
    assert abs(fwd - 553648128) / 553648128 < 0.01
    assert bench.traffic_entry(3, "stream_fwd_tzy") is None  # no counters for that workload
