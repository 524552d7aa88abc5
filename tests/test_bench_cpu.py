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
    # the 64x256x256x32 shard of 256^3x32 (B2 C32), the largest single-GPU forward configuration
    assert (a.gpus, a.steps, a.warmup, a.workload) == (1, 20, 5, 3)
    assert not a.graph and not a.block and not a.fno


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_unfused_block_needs_a_block_workload():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--unfused-block"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "--unfused-block applies to --block and --fno" in r.stderr
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


def test_counters_resolve_for_the_default_workload_3():
    """The default workload's HBM counters and MFMA counters are committed
    and match the current kernel sources (otherwise the bench line's traffic
    and counter fractions would be null)."""
    import bench
    for role in ("stream_fwd_tzy", "stream_inv_yzt"):
        t = bench.traffic_entry(3, role)
        assert t is not None, f"no current FETCH/WRITE counters for {role} at workload 3"
        # 64x256x256x32, B2 C32: 34.36 GB of shard + 0.27 GB of y-contracted rows, algorithmically
        alg = bench.work(_w3(), 32)[role]["bytes"]
        assert abs(t - alg) / alg < 0.02, (role, t, alg)
        f = bench.counter_flops(3, role)
        assert f is not None, f"no current MFMA counters for {role} at workload 3"
        ex = bench.work(_w3(), 32)[role]["mfma_flops"]
        # the counters include padded products; the accounting counts none
        assert 0.99 * ex <= f <= 1.25 * ex, (role, f, ex)


def _w3():
    import synth
    return synth.geometry(3)


def _table3():
    rows = {}
    with open(os.path.join(ROOT, "tests", "golden", "table3_gemm_flops.txt")) as f:
        for ln in f:
            if ln.startswith("#") or not ln.strip():
                continue
            parts = ln.split()
            rows["total" if parts[0] == "total" else parts[1]] = float(parts[4])
    return rows


def test_stage_flops_reproduce_table3():
    """Sec. V-B Table 3: per-stage GEMM flops of one forward on a 128 x 128 x 64
    grid with T = 30, modes (8, 8, 8, 16) and width 20, counted by the paper
    as 2 flops per complex multiply-add, stages T, Z, Y, X.  bench.stage_flops
    counts real flops: 4 per real x complex multiply-add (the T stage, real
    input) and 8 per complex x complex one, so its counts are 2x (T) and 4x
    (Z, Y, X) the printed ones."""
    import bench
    g = {"batch": 1, "n_local": (128, 128, 64, 30), "kmax": (8, 8, 8), "kt": 16}
    sf = bench.stage_flops(g, 20)
    tab = _table3()
    per_mac = {"T": 2, "Z": 4, "Y": 4, "X": 4}
    for st in "TZYX":
        got = sf[st.lower()] / per_mac[st] / 1e9
        assert abs(got - tab[st]) <= 0.05, (st, got, tab[st])
    total = sum(sf[st.lower()] / per_mac[st] for st in "TZYX") / 1e9
    assert abs(total - tab["total"]) <= 0.05, (total, tab["total"])


def test_work_uses_stage_flops_and_folds():
    """work(): the fused forward's direct flops are the t, z and y stages, the
    x contraction's the x stage; executed flops divide each folded stage."""
    import bench
    g = _w3()
    sf = bench.stage_flops(g, 32)
    w = bench.work(g, 32)
    assert w["stream_fwd_tzy"]["flops"] == sf["t"] + sf["z"] + sf["y"]
    assert w["axis_fwd_x"]["flops"] == sf["x"]
    # workload 3: y folds (whole N_y), x does not (a slab), z folds in classes, t does not (k_t = 8);
    # the axis kernels take complex products in three real products instead of four
    assert w["axis_fwd_x"]["mfma_flops"] == sf["x"] * 0.75
    zc = bench._z_classes(g)
    assert w["stream_fwd_tzy"]["mfma_flops"] == sf["t"] + sf["z"] / zc + sf["y"] / 2
    # the backward workload keeps K_y = 64 of the whole N_y = 256: y folds in four classes
    import synth
    g5 = synth.geometry(5)
    assert bench._axis_classes(g5, 1) == 4 and bench._axis_classes(g5, 0) == 1
    sf5 = bench.stage_flops(g5, 32)
    w5 = bench.work(g5, 32)
    assert w5["axis_fwd_y"]["mfma_flops"] == sf5["y"] / 4 * 0.75 == w5["axis_inv_y"]["mfma_flops"]
    # K = 32 per dimension (workload 3) would leave half-empty tiles: two classes only
    assert bench._axis_classes(g, 1) == 2
    # the accumulating x contraction also reads the spectrum back
    wa = bench.work(g, 32, acc_share=1.0)
    spec = g["batch"] * 32 * 32 * 32 * 32 * 8 * 8
    assert wa["axis_fwd_x"]["bytes"] - w["axis_fwd_x"]["bytes"] == spec
