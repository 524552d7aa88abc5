#!/usr/bin/env python3
"""Benchmark of one DTST spectral layer (forward partial DFT + mode-wise
channel mix + inverse partial DFT) on one MI355X.

A step is one pass of the whole layer over one batch of synthetic input
already resident in HBM.  The default workload is one GPU's share of a
256^3 x 32 grid split 4 ways along x: the 64 x 256 x 256 x 32 shard at x
offset 64, B = 2, C_in = C_out = 32, modes 32/32/32/8 -- the largest
single-GPU forward configuration.  The workloads that cover a whole
decomposition (--workload 2: 128^3 x 32 in 8 x-slabs) run the shards one
after another on this GPU: the shard forwards accumulate into one spectrum
(the sum that replaces the AllReduce), the mix runs over the mode ranges S_p
in turn (which assembles the spectrum the AllGather would), and every shard
is then expanded back.

Prints one JSON line with the step time, the layer's GB/s and TFLOP/s
(executed flops after the exact folds, and the direct-definition count of
Table 3's stages), an HBM roofline entry for the kernel that takes the most
time and an fp32-MFMA roofline entry for the contraction kernel that
executes the most matrix work (average launch times measured here with HIP
events on the launch stream; rocprof counter figures from profiles/ where
they match the kernel source), and the fp64 CPU oracle timed on a bounded
sample of the same workload on this host.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
FP32_MFMA_PEAK_TFS = 157.3   # MI355X dense fp32 matrix
COUNTERS_FILE = os.path.join(ROOT, "profiles", "hbm_counters.json")
MFMA_COUNTERS_FILE = os.path.join(ROOT, "profiles", "mfma_counters.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4, 5, 6, 7],
                    help="workload table entry (default 3: the 64x256x256x32 shard of 256^3x32, B2 C32, the "
                         "largest single-GPU forward configuration; 2: 128^3x32 in 8 x-slabs; 5 times the "
                         "backward; 6: 128^3x32 in 2x4 (x, y) pencils)")
    ap.add_argument("--block", action="store_true",
                    help="time the whole block of Algorithm 1: after every shard's inverse, the point-wise "
                         "bypass of the shard's input and GELU (forward workloads only)")
    ap.add_argument("--fno", action="store_true",
                    help="time the whole FNO forward (lift, 4 Fourier layers, projection) on workload 7, the "
                         "paper's model shape (d_v 20, modes (8, 8, 8, 16)) on 128^3 x 32 in 4 x-slabs")
    ap.add_argument("--unfused-block", action="store_true",
                    help="with --block or --fno: plans made with PLAN_UNFUSED_BLOCK, so that every block "
                         "epilogue runs as the inverse followed by the separate epilogue kernel (for comparison)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph after the warm-up and replay it in the timed "
                         "region (the same kernels; removes the host's per-launch cost)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-times", action="store_true",
                    help="skip the per-kernel event pass (used under rocprofv3)")
    ap.add_argument("--hbm-warmup-gb", type=int, default=96,
                    help="allocate, zero and release this much device memory before building the "
                         "workload (HBM that has not been written since the device came up streams "
                         "measurably slower; 0 disables)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (the known-size "
                         "reference for the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# Algorithmic work of each kernel role.  Flops are real flops: a real x complex
# multiply-add is 4, complex x complex 8.  "flops" are the direct-definition
# counts of each per-dimension contraction (Table 3's stages, in its order
# T, Z, Y, X), "mfma_flops" the products the kernels execute after the exact
# even / odd and four-class folds (no padding).  Bytes are the tensors each
# kernel must read and write once.
# ---------------------------------------------------------------------------
def stage_flops(g, channels):
    """Direct-definition real flops of the four per-dimension contractions of
    one forward (Sec. V-B, Table 3), contracting t, then z, y, x:
      t: 4 K_t N_t per (b, c, x, y, z) line (real input, complex basis)
      z: 8 K_z N_z per (b, c, x, y, k_t) line
      y: 8 K_y N_y per (b, c, x, k_z, k_t) line
      x: 8 K_x N_x per (b, c, k_y, k_z, k_t) line
    The inverse expansions mirror them."""
    B = g["batch"]
    Nx, Ny, Nz, Nt = g["n_local"]
    k = g["kmax"]
    Kx, Ky, Kz, Kt = 2 * k[0], 2 * k[1], 2 * k[2], g["kt"]
    lines = B * channels
    return {"t": lines * Nx * Ny * Nz * 4 * Kt * Nt,
            "z": lines * Nx * Ny * Kt * 8 * Kz * Nz,
            "y": lines * Nx * Kz * Kt * 8 * Ky * Ny,
            "x": lines * Ky * Kz * Kt * 8 * Kx * Nx}


def work(g, channels, m_count=None, acc_share=0.0):
    """Per-launch work of every kernel role.  acc_share: the share of the
    x-contraction launches that accumulate into the spectrum (they also read
    it back)."""
    B = g["batch"]
    Nx, Ny, Nz, Nt = g["n_local"]
    k = g["kmax"]
    Kx, Ky, Kz, Kt = 2 * k[0], 2 * k[1], 2 * k[2], g["kt"]
    C = channels
    M = Kx * Ky * Kz * Kt
    rows = B * C * Nx * Ny
    sf = stage_flops(g, C)
    fy = 1.0 / _axis_classes(g, 1)
    fx = 1.0 / _axis_classes(g, 0)
    w = {}
    # the t-folded kernels take the complex z products in three real products instead of four
    z_prod = 0.75 if _t_classes(g) == 2 else 1.0
    w["stream_fwd_tz"] = dict(
        bytes=rows * (Nz * Nt * 4 + Kz * Kt * 8),
        flops=sf["t"] + sf["z"],
        mfma_flops=sf["t"] / _t_classes(g) + sf["z"] / _z_classes(g) * z_prod)
    # the axis kernels take every complex product in three real products instead of four
    ax = 0.75
    w["axis_fwd_y"] = dict(bytes=B * C * Nx * (Ny + Ky) * Kz * Kt * 8, flops=sf["y"], mfma_flops=sf["y"] * fy * ax)
    # t + z + y in one launch: reads the shard once, writes the y-contracted rows
    w["stream_fwd_tzy"] = dict(
        bytes=rows * Nz * Nt * 4 + B * C * Nx * Ky * Kz * Kt * 8,
        flops=w["stream_fwd_tz"]["flops"] + sf["y"],
        mfma_flops=w["stream_fwd_tz"]["mfma_flops"] + sf["y"] * fy)
    spec = B * C * M * 8
    w["axis_fwd_x"] = dict(bytes=B * C * Nx * Ky * Kz * Kt * 8 + spec + acc_share * spec, flops=sf["x"],
                           mfma_flops=sf["x"] * fx * ax)
    w["axis_inv_x"] = dict(bytes=B * C * Nx * Ky * Kz * Kt * 8 + spec, flops=sf["x"], mfma_flops=sf["x"] * fx * ax)
    w["axis_inv_y"] = dict(bytes=w["axis_fwd_y"]["bytes"], flops=sf["y"], mfma_flops=sf["y"] * fy * ax)
    w["stream_inv_zt"] = dict(bytes=w["stream_fwd_tz"]["bytes"], flops=w["stream_fwd_tz"]["flops"],
                              mfma_flops=w["stream_fwd_tz"]["mfma_flops"])
    # y + z + t in one launch: reads the x-expanded spectrum, writes the shard
    w["stream_inv_yzt"] = dict(bytes=w["stream_fwd_tzy"]["bytes"], flops=w["stream_fwd_tzy"]["flops"],
                               mfma_flops=w["stream_fwd_tzy"]["mfma_flops"])
    mc = M if m_count is None else m_count
    ci, co = g["c_in"], g["c_out"]
    w["mix"] = dict(bytes=mc * ci * co * 8 + B * (ci + co) * mc * 8, flops=8 * B * mc * ci * co)
    for v in w.values():
        v.setdefault("mfma_flops", v["flops"])
    return w


def _block_zt_work(g):
    """The fused inverse z + t expansion and block epilogue: reads the
    y-expanded spectrum (B, C_out, N_x, N_y, K_z, K_t) and the block input x,
    writes y once.  Executed flops: the z expansion with z folded in two
    classes where that saves padded slots (three real products per
    complex one when t folds), the t expansion (halved when t folds), and the
    bypass (C_out x C_in per point) on the matrix cores."""
    B, ci, co = g["batch"], g["c_in"], g["c_out"]
    Nx, Ny, Nz, Nt = g["n_local"]
    Kz, Kt = 2 * g["kmax"][2], g["kt"]
    V = _vol(g)
    sf = stage_flops(g, co)
    zc = _block_z_classes(g)
    tc = _t_classes(g)
    byp = 2 * B * V * ci * co
    return dict(bytes=B * co * Nx * Ny * Kz * Kt * 8 + B * (ci + co) * V * 4, flops=sf["t"] + sf["z"] + byp,
                mfma_flops=sf["t"] / tc + sf["z"] / zc * (0.75 if tc == 2 else 1.0) + byp)


# Kernel roles whose products run on the matrix cores (the per-dimension
# contractions); the mix, its gradients and the point-wise layers run on the
# vector ALUs.
CONTRACTION_ROLES = ("stream_fwd_tzy", "stream_fwd_tz", "axis_fwd_y", "axis_fwd_x", "axis_inv_x", "axis_inv_y",
                     "stream_inv_zt", "stream_inv_yzt", "stream_inv_zt_block")


def _folded(g, dim):
    """The library folds a dimension whose whole even extent is local."""
    return g["n_local"][dim] == g["n_global"][dim] and g["n_global"][dim] % 2 == 0


def _axis_classes(g, dim):
    """Mode classes of the separate x / y contractions: 4 when the whole
    extent is local with N % 4 == 0 and the K = 2 k_max retained modes fill
    whole 16-mode tiles per class (K % 64 == 0, K <= 128), 2 when the
    dimension only folds in halves, else 1; their MFMA work divides by it."""
    if not _folded(g, dim):
        return 1
    K = 2 * g["kmax"][dim]
    return 4 if g["n_global"][dim] % 4 == 0 and K % 64 == 0 and K <= 128 else 2


def _t_classes(g):
    """2 when the streaming kernels fold t (8 < k_t <= 16 and the whole
    N_t = 32 local: even k_t from the sums of t and t + N_t/2, odd k_t from
    the differences), else 1; the t MFMA work divides by it."""
    nt = g["n_local"][3]
    return 2 if 8 < g["kt"] <= 16 and nt == 32 and g["n_global"][3] == nt else 1


def _z_classes(g):
    """z mode classes of the streaming kernels.  z folds only where the shard
    holds the whole even N_z; the class count is the one with the fewest
    padded slots per class (the z products per row are those slots x N_z for
    any count), the smaller one on a tie: 4 (k mod 4: N_z % 4 == 0, even
    k_max, and at most 16 modes per class with k_t > 8 or 8 with k_t <= 8),
    2 (parity) or 1.  The z MFMA work divides by it."""
    if not _folded(g, 2):
        return 1
    Kz = 2 * g["kmax"][2]
    ct = 2 if g["kt"] > 8 else 1

    def padded(n):
        if n == 4 and ct == 1:
            return 8
        k = -(-(-(-Kz // n)) // 16) * 16
        return 64 if k == 48 else k

    n = 1
    if padded(2) < padded(n):
        n = 2
    four = g["n_global"][2] % 4 == 0 and g["kmax"][2] % 2 == 0 and Kz <= (64 if ct == 2 else 32)
    if four and padded(4) < padded(n):
        n = 4
    return n


def _block_z_classes(g):
    """z classes of the fused inverse + block epilogue kernel: 2 where z folds
    and the parity classes pad to fewer slots than one class, else 1."""
    if not _folded(g, 2):
        return 1
    Kz = 2 * g["kmax"][2]
    return 2 if -(-(-(-Kz // 2)) // 16) < -(-Kz // 16) else 1


def _sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


# ---------------------------------------------------------------------------
class Workload:
    """One benchmark step and its accounting.

    step()      launches the whole step on the current stream
    launches    kernel role -> launches per step
    work        kernel role -> algorithmic bytes / flops of one launch
    bytes, flops, mfma_flops   the whole step
    cpu_sample()  runs the fp64 oracle on a sample of the step and returns
                  (seconds, fraction of the step's bytes it covered, description)
    """


def _geo(O, g, batch=None, c_in=None, c_out=None):
    return O.Geometry(g["n_global"], g["n_local"], g["offset"], g["kmax"], g["kt"],
                      g["batch"] if batch is None else batch, g["c_in"] if c_in is None else c_in,
                      g["c_out"] if c_out is None else c_out)


def _vol(g):
    v = 1
    for n in g["n_local"]:
        v *= n
    return v


def _mix_work(g, m_count, kind):
    B, ci, co = g["batch"], g["c_in"], g["c_out"]
    spectra = B * (ci + co) * m_count * 8
    return dict(bytes=m_count * ci * co * 8 + spectra, flops=8 * B * m_count * ci * co,
                mfma_flops=8 * B * m_count * ci * co)


def forward_workload(torch, D, synth, cfg, device, block=False, flags=0):
    """Forward partial DFT + mix + inverse over every shard of the workload.
    Workload 2 runs its 8 slabs one after another: the forwards accumulate
    into one spectrum, the mix runs over the 8 mode ranges in turn, and every
    slab is then expanded back."""
    c = synth.WORKLOADS[cfg]
    shards = []
    if cfg in synth.ALL_SHARDS:
        full = synth.full_domain(cfg)
        x_full = synth.torch_input(cfg, full, device)
        for p in range(c["shards"]):
            g = synth.geometry(cfg, p)
            (x0, y0, _, _), (lx, ly, _, _) = g["offset"], g["n_local"]
            shards.append((g, x_full[:, :, x0:x0 + lx, y0:y0 + ly].contiguous()))
        del x_full
        torch.cuda.empty_cache()
    else:
        g = synth.geometry(cfg)
        shards.append((g, synth.torch_input(cfg, g, device)))
    g0 = shards[0][0]
    plans = [D.Plan(g, device, flags) for g, _ in shards]
    M = plans[0].n_modes
    W = synth.torch_weights(M, g0["c_in"], g0["c_out"], synth.seed_of(cfg, "weights"), device)
    xhat = torch.empty(plans[0].spectral_shape(g0["c_in"]), dtype=torch.complex64, device=device)
    yhat = torch.empty(plans[0].spectral_shape(g0["c_out"]), dtype=torch.complex64, device=device)
    ys = [torch.empty(p.spatial_shape(g0["c_out"]), dtype=torch.float32, device=device) for p in plans]
    P = len(plans)
    bounds = [(M * r) // P for r in range(P + 1)]
    ranges = [(bounds[r], bounds[r + 1]) for r in range(P)]
    Wb = synth.torch_bypass(g0["c_out"], g0["c_in"], synth.seed_of(cfg, "bypass"), device) if block else None

    w = Workload()

    def step():
        for p, (plan, (_, x)) in enumerate(zip(plans, shards)):
            plan.forward(x, xhat, accumulate=p > 0)
        for m0, m1 in ranges:
            plans[0].mix(xhat, W[m0:m1], yhat, m0, m1)
        for plan, y, (_, x) in zip(plans, ys, shards):
            if block:
                plan.inverse_block(yhat, x, Wb, y)
            else:
                plan.inverse(yhat, y)

    w.step = step
    # every shard's forward after the first accumulates into the spectrum
    per = work(g0, g0["c_in"], acc_share=(P - 1) / P)
    per["mix"] = _mix_work(g0, M // P, "mix")
    B0, ci0, co0, V0 = g0["batch"], g0["c_in"], g0["c_out"], _vol(g0)
    per["block_epilogue"] = dict(bytes=B0 * V0 * (ci0 + 2 * co0) * 4, flops=2 * B0 * V0 * ci0 * co0,
                                 mfma_flops=2 * B0 * V0 * ci0 * co0)
    per["stream_inv_zt_block"] = _block_zt_work(g0)
    w.work = per
    B, ci, co = g0["batch"], g0["c_in"], g0["c_out"]
    w.bytes = P * B * (ci + co) * _vol(g0) * 4 + M * ci * co * 8   # read x, write y, read W
    w.metric = ("DRIFT block ms and GB/s + TFLOP/s per MI355X (fwd partial DFT+mix+inverse, bypass + GELU)"
                if block else "spectral-layer ms and GB/s + TFLOP/s per MI355X (fwd partial DFT+mix+inverse)")
    w.config = {"workload": synth.WORKLOADS[cfg]["name"], "global_grid": list(g0["n_global"]),
                "local_shard": list(g0["n_local"]), "shards_run_in_sequence": P, "batch": B,
                "c_in": ci, "c_out": co,
                "modes": [2 * g0["kmax"][0], 2 * g0["kmax"][1], 2 * g0["kmax"][2], g0["kt"]]}

    def cpu_sample(min_seconds=10.0):
        """Whole fp64 oracle layers of this workload when a layer is small
        (repeated until min_seconds), else the first channels of shard 0
        through forward, mix on a mode range, inverse."""
        import numpy as np
        import oracle as O
        if w.bytes <= 16e9:
            geos = [_geo(O, g) for g, _ in shards]
            xs = [x.cpu().numpy() for _, x in shards]
            Ws = W.cpu().numpy()
            Wbs = Wb.cpu().numpy() if block else None
            layers = 0
            t0 = time.perf_counter()
            while True:
                X = None
                for x, geo in zip(xs, geos):
                    part = O.forward(x, geo)
                    X = part if X is None else X + part
                Y = O.mix(X, Ws, 0, M, c_out=co).reshape((X.shape[0], co) + geos[0].K)
                for geo, x in zip(geos, xs):
                    y = O.inverse(Y, geo)
                    if block:
                        O.block_epilogue(x, Wbs, y)
                layers += 1
                dt = time.perf_counter() - t0
                if dt >= min_seconds:
                    break
            what = "block(s)" if block else "layer(s)"
            extra = ", each followed by the bypass and GELU" if block else ""
            return dt, float(layers), (f"fp64 oracle, {layers} whole {what} of this workload ({P} shard forwards "
                                       f"summed, mix over all {M} modes, {P} shard inverses{extra}), inputs in "
                                       f"host memory")
        # one (b, c) slice after another of shard 0 through the forward and
        # the inverse, each with the mix over a block of modes, until
        # min_seconds have passed
        ms = 8192
        g, x = shards[0]
        geo = _geo(O, g, batch=1, c_in=1, c_out=1)
        Ws = W[:ms, :, :].cpu().numpy()
        Xs = synth.np_complex_normal((B, ci, ms), 12345)
        Ys = synth.np_complex_normal((1, 1) + geo.K, 12346)
        slices = []
        dt = 0.0
        for s_i in range(B * ci):
            b, c = divmod(s_i, ci)
            xs = x[b:b + 1, c:c + 1].cpu().numpy()
            Wbs = Wb[c:c + 1, c:c + 1].cpu().numpy() if block else None
            t0 = time.perf_counter()
            O.forward(xs, geo)
            O.mix(Xs, Ws, 0, ms, c_out=co)
            ys = O.inverse(Ys, geo)
            if block:
                O.block_epilogue(xs, Wbs, ys)
            dt += time.perf_counter() - t0
            slices.append((b, c))
            if dt >= min_seconds:
                break
        n = len(slices)
        frac = n * (2 * _vol(g) * 4 + ms * ci * co * 8) / w.bytes
        return dt, frac, (f"fp64 oracle: {n} (b, c) slices of shard 0, each through the forward and the inverse "
                          f"with the mix over {ms} modes; GB/s scaled by the share of the layer's bytes they "
                          f"cover ({frac:.2e})")

    w.cpu_sample = cpu_sample
    return w


def backward_workload(torch, D, synth, cfg, device):
    """Backward of the spectral layer on one shard: inverse_adj of the
    upstream gradient, the mix data gradient (W^H), the weight gradient and
    forward_adj, over the full mode set."""
    g = synth.geometry(cfg)
    plan = D.Plan(g, device)
    M = plan.n_modes
    B, ci, co = g["batch"], g["c_in"], g["c_out"]
    x = synth.torch_input(cfg, g, device)
    xhat = torch.empty(plan.spectral_shape(ci), dtype=torch.complex64, device=device)
    plan.forward(x, xhat)            # set-up: the saved forward spectrum
    torch.cuda.synchronize()
    del x
    torch.cuda.empty_cache()
    W = synth.torch_weights(M, ci, co, synth.seed_of(cfg, "weights"), device)
    gy = synth.torch_normal(tuple(plan.spatial_shape(co)), synth.seed_of(cfg, "upstream"), device)
    gyh = torch.empty(plan.spectral_shape(co), dtype=torch.complex64, device=device)
    gxh = torch.empty(plan.spectral_shape(ci), dtype=torch.complex64, device=device)
    gW = torch.empty_like(W)
    gx = torch.empty(plan.spatial_shape(ci), dtype=torch.float32, device=device)

    w = Workload()

    def step():
        plan.inverse_adj(gy, gyh)
        plan.mix(gyh, W, gxh, 0, M, op=1)
        plan.wgrad(xhat, gyh, gW, 0, M)
        plan.forward_adj(gxh, gx)

    w.step = step
    per_o = work(g, co)       # inverse_adj runs the forward-direction kernels on C_out channels
    per_i = work(g, ci)       # forward_adj runs the inverse-direction kernels on C_in channels
    per = {k: per_o[k] for k in ("stream_fwd_tzy", "stream_fwd_tz", "axis_fwd_y", "axis_fwd_x")}
    per.update({k: per_i[k] for k in ("axis_inv_x", "axis_inv_y", "stream_inv_zt", "stream_inv_yzt")})
    per["mix_h"] = _mix_work(g, M, "mix_h")
    per["wgrad"] = _mix_work(g, M, "wgrad")
    w.work = per
    w.bytes = B * (ci + co) * _vol(g) * 4 + 2 * M * ci * co * 8   # read g_y, write g_x, read W, write g_W
    w.metric = ("spectral-layer backward ms and GB/s + TFLOP/s per MI355X "
                "(inverse_adj + mix data grad + wgrad + forward_adj)")
    w.config = {"workload": synth.WORKLOADS[cfg]["name"], "global_grid": list(g["n_global"]),
                "local_shard": list(g["n_local"]), "shards_run_in_sequence": 1, "batch": B,
                "c_in": ci, "c_out": co,
                "modes": [2 * g["kmax"][0], 2 * g["kmax"][1], 2 * g["kmax"][2], g["kt"]]}

    def cpu_sample(min_seconds=10.0):
        """One (b, c) slice through inverse_adj and forward_adj, and the
        data and weight gradients over a mode range, on the fp64 oracle."""
        import oracle as O
        ms = 4096
        geo = _geo(O, g, batch=1, c_in=1, c_out=1)
        Ws = W[:ms].cpu().numpy()
        Xs = synth.np_complex_normal((B, ci, ms), 12345)
        Gs = synth.np_complex_normal((B, co, ms), 12346)
        GXs = synth.np_complex_normal((1, 1) + geo.K, 12347)
        n = 0
        dt = 0.0
        for s_i in range(B * co):
            b, c = divmod(s_i, co)
            gys = gy[b:b + 1, c:c + 1].cpu().numpy()
            t0 = time.perf_counter()
            O.inverse_adj(gys, geo)
            O.mix_data_grad(Gs, Ws, 0, ms)
            O.mix_wgrad(Xs, Gs, 0, ms)
            O.forward_adj(GXs, geo)
            dt += time.perf_counter() - t0
            n += 1
            if dt >= min_seconds:
                break
        frac = n * (2 * _vol(g) * 4 + 2 * ms * ci * co * 8) / w.bytes
        return dt, frac, (f"fp64 oracle: {n} (b, c) slices through inverse_adj and forward_adj, each with the "
                          f"data and weight gradients over {ms} modes; GB/s scaled by the share of the step's "
                          f"bytes they cover ({frac:.2e})")

    w.cpu_sample = cpu_sample
    return w


def fno_workload(torch, D, synth, cfg, device, flags=0):
    """FNO forward (lift, Fourier layers as Algorithm 1, projection) over
    every shard of the workload, run one after another on this GPU."""
    from paper_2607_14394_amd.fno import FNO
    c = synth.WORKLOADS[cfg]
    spec = c["fno"]
    cin, cout, L = spec["c_data_in"], spec["c_data_out"], spec["layers"]
    shards = [synth.geometry(cfg, p) for p in range(c["shards"])]
    g0 = shards[0]
    dv, B = g0["c_in"], g0["batch"]
    M = synth.n_modes(g0)
    lift, layers, proj = synth.fno_params_np(M, dv, cin, cout, L, 1000 * cfg)
    t = lambda a: torch.from_numpy(a).to(device)
    fno = FNO(shards, (t(lift[0]), t(lift[1])), [(t(r), t(wb)) for r, wb in layers], (t(proj[0]), t(proj[1])),
              device, flags)
    xs = [synth.torch_normal(tuple(fno.input_shape(p)), synth.seed_of(cfg, "input") + p, device)
          for p in range(len(shards))]
    outs = [torch.empty(fno.output_shape(p), dtype=torch.float32, device=device) for p in range(len(shards))]
    P = len(shards)

    w = Workload()
    w.step = lambda: fno.forward(xs, outs)
    per = work(g0, dv)
    per["mix"] = _mix_work(g0, M // P, "mix")
    V = _vol(g0)
    per["block_epilogue"] = dict(bytes=B * V * 3 * dv * 4, flops=2 * B * V * dv * dv, mfma_flops=2 * B * V * dv * dv)
    per["stream_inv_zt_block"] = _block_zt_work(g0)
    # lift (C_in -> d_v) and projection (d_v -> C_out) move and compute the same per point when C_in = C_out
    pw = [B * V * (cin + dv) * 4, B * V * (dv + cout) * 4]
    per["pointwise"] = dict(bytes=sum(pw) / 2, flops=B * V * dv * (cin + cout), mfma_flops=B * V * dv * (cin + cout))
    w.work = per
    # Minimum traffic of the network: the input and output fields once, and per Fourier layer its
    # input activation read once, its output written once and its spectral weights read once.
    w.bytes = P * B * V * (cin + cout) * 4 + L * (2 * P * B * V * dv * 4 + M * dv * dv * 8)
    w.metric = "FNO forward ms and GB/s per MI355X (lift, 4 Fourier layers of Algorithm 1, projection)"
    w.config = {"workload": c["name"], "global_grid": list(g0["n_global"]), "local_shard": list(g0["n_local"]),
                "shards_run_in_sequence": P, "batch": B, "d_v": dv, "c_data_in": cin, "c_data_out": cout,
                "fourier_layers": L, "modes": [2 * g0["kmax"][0], 2 * g0["kmax"][1], 2 * g0["kmax"][2], g0["kt"]]}

    def cpu_sample(min_seconds=10.0):
        """One Fourier layer of one (b, c) slice of shard 0 (forward, inverse,
        bypass and GELU of that channel) and the mix over a mode range, on the
        fp64 oracle."""
        import numpy as np
        import oracle as O
        ms = 4096
        geo = _geo(O, g0, batch=1, c_in=1, c_out=1)
        Rs = layers[0][0][:ms]
        Xs = synth.np_complex_normal((B, dv, ms), 12345)
        Ys = synth.np_complex_normal((1, 1) + geo.K, 12346)
        n = 0
        dt = 0.0
        for it in range(64):
            c = it % xs[0].shape[1]
            xs0 = xs[0][0:1, c:c + 1].cpu().numpy()
            t0 = time.perf_counter()
            O.forward(xs0, geo)
            O.mix(Xs, Rs, 0, ms, c_out=dv)
            O.block_epilogue(xs0, np.eye(1), O.inverse(Ys, geo))
            dt += time.perf_counter() - t0
            n += 1
            if dt >= min_seconds:
                break
        frac = n * (2 * V * 4 + ms * dv * dv * 8) / w.bytes
        return dt, frac, (f"fp64 oracle: {n} channel slices of shard 0, each through one Fourier layer (forward, "
                          f"inverse, bypass and GELU) with the mix over {ms} modes; GB/s scaled by the share of "
                          f"the forward's bytes they cover ({frac:.2e})")

    w.cpu_sample = cpu_sample
    return w


def cpu_baseline(w):
    """Times the fp64 oracle on the workload's sample with the BLAS threads
    set to the cores this process may use."""
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
    except Exception:  # pragma: no cover
        threadpool_limits = None
    cores = len(os.sched_getaffinity(0))
    ctx = threadpool_limits(limits=cores) if threadpool_limits else None
    try:
        dt, frac, desc = w.cpu_sample()
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1) if threadpool_limits else cores
    finally:
        if ctx is not None:
            ctx.__exit__(None, None, None)
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    blas = None
    if threadpool_limits:
        libs = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        blas = ", ".join(sorted({"%s %s" % (i.get("internal_api"), i.get("version")) for i in libs})) or None
    return {"value": round(w.bytes * frac / dt / 1e9, 3), "unit": "GB/s", "cores": int(threads),
            "kind": "oracle", "seconds": round(dt, 2), "sample": desc, "cpu_model": cpu_model, "blas": blas}


def counter_flops(cfg, kernel):
    """fp32 MFMA flops per launch of one kernel role of workload cfg from
    committed rocprof counters (SQ_INSTS_VALU_MFMA_MOPS_F32 x 512); None when
    there are none or the kernel source changed since they were taken."""
    try:
        with open(MFMA_COUNTERS_FILE) as f:
            c = json.load(f)
    except Exception:
        return None
    ent = c.get("workloads", {}).get(str(cfg), {}).get("kernels", {}).get(kernel)
    if not ent:
        return None
    src = os.path.join(ROOT, "paper_2607_14394_amd", "csrc", ent.get("source", "k_stream.hip"))
    if ent.get("source_sha") != _sha(src):
        return None
    return ent["mfma_flops_per_launch"]


def traffic_entry(cfg, kernel):
    """HBM bytes per launch of one kernel role of workload cfg from committed
    FETCH_SIZE / WRITE_SIZE counters, scaled by the copy-kernel calibration;
    None when the workload has no counters or the kernel source changed
    since they were taken."""
    try:
        with open(COUNTERS_FILE) as f:
            c = json.load(f)
    except Exception:
        return None
    ent = c.get("workloads", {}).get(str(cfg), {}).get("kernels", {}).get(kernel)
    if not ent:
        return None
    src = os.path.join(ROOT, "paper_2607_14394_amd", "csrc", ent.get("source", "k_stream.hip"))
    if ent.get("source_sha") != _sha(src):
        return None
    return ent["fetch_kib"] * 1024 * c["fetch_scale"] + ent["write_kib"] * 1024 * c["write_scale"]


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: every shard of the decomposition runs one after "
              "another on a single MI355X (no collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.fno and args.block:
        print("--fno already includes every block's bypass and GELU", file=sys.stderr)
        sys.exit(2)
    if args.unfused_block and not (args.block or args.fno):
        print("--unfused-block applies to --block and --fno", file=sys.stderr)
        sys.exit(2)

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy:
        n = 1 << 28                      # 2^28 floats = 1 GiB
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": n * 4, "copies": 3}), flush=True)
        return

    import paper_2607_14394_amd as D
    import synth

    device = "cuda"
    cfg = 7 if args.fno else args.workload
    if args.hbm_warmup_gb > 0:
        # Set-up only, outside every timed region: the stream kernels run up to
        # 13% slower on the first large buffers a fresh process places in HBM;
        # touching and releasing one large block first removes that.
        free_b, _ = torch.cuda.mem_get_info()
        nbytes = min(args.hbm_warmup_gb << 30, int(free_b * 0.8))
        log(f"touching {nbytes >> 30} GiB of HBM once")
        blk = torch.empty(nbytes, dtype=torch.uint8, device=device)
        blk.zero_()
        torch.cuda.synchronize()
        del blk
        torch.cuda.empty_cache()
    log(f"building workload {cfg}")
    if args.block and cfg == 5:
        print("--block applies to the forward workloads (1-4)", file=sys.stderr)
        sys.exit(2)
    if cfg == 7 and not args.fno:
        print("workload 7 is the FNO forward: run it with --fno", file=sys.stderr)
        sys.exit(2)
    flags = D.PLAN_UNFUSED_BLOCK if args.unfused_block else 0
    if args.fno:
        w = fno_workload(torch, D, synth, cfg, device, flags)
    else:
        w = (backward_workload(torch, D, synth, cfg, device) if cfg == 5
             else forward_workload(torch, D, synth, cfg, device, block=args.block, flags=flags))
    log(f"warmup {args.warmup} steps")

    # ---- warmup ----
    for _ in range(args.warmup):
        w.step()
    torch.cuda.synchronize()

    # The kernels one step launches (the plan picks the forward schedule):
    # one untimed step under the library's own launch records.
    D.dtst_profile_collect()
    D.dtst_profile_enable(True)
    w.step()
    torch.cuda.synchronize()
    w.launches = {k: n for k, (n, _) in D.dtst_profile_collect().items() if n > 0}
    D.dtst_profile_enable(False)
    missing = [k for k in w.launches if k not in w.work]
    assert not missing, f"no work accounting for kernel roles {missing}"
    w.flops = sum(w.work[k]["flops"] * n for k, n in w.launches.items())
    w.mfma_flops = sum(w.work[k]["mfma_flops"] * n for k, n in w.launches.items())
    log(f"kernels per step: {w.launches}")

    # ---- optional HIP graph of one step (the execute calls are capturable:
    # kernel launches only) ----
    run = w.step
    if args.graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            w.step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            w.step()
        run = graph.replay
        run()
        torch.cuda.synchronize()

    log(f"timing {args.steps} steps")
    # ---- timed region: K steps bracketed by events on the launch stream ----
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        run()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps

    # ---- per-step pass: each step bracketed by its own events (median, min) ----
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record(stream)
        run()
        e1.record(stream)
    torch.cuda.synchronize()
    per_step = sorted(e0.elapsed_time(e1) for e0, e1 in evs)

    # ---- per-kernel pass: every launch bracketed by HIP events ----
    kernel_ms = {}
    if not args.no_kernel_times:
        D.dtst_profile_enable(True)
        D.dtst_profile_collect()
        torch.cuda.synchronize()
        for _ in range(args.steps):
            w.step()
        torch.cuda.synchronize()
        prof = D.dtst_profile_collect()
        D.dtst_profile_enable(False)
        kernel_ms = {k: (n, tot / n) for k, (n, tot) in prof.items()}

    # ---- accounting ----
    sec = ms_per_step / 1e3
    gbs = w.bytes / sec / 1e9
    roof = None
    roof_mfma = None
    stages = {}
    if kernel_ms:
        for k, (n, avg) in kernel_ms.items():
            wk = w.work.get(k)
            if wk is None:
                continue
            st = {"launches_per_step": n // args.steps, "avg_ms": round(avg, 4),
                  "bytes_per_launch": int(wk["bytes"]), "executed_flops_per_launch": int(wk["mfma_flops"]),
                  "direct_flops_per_launch": int(wk["flops"]),
                  "GB_s": round(wk["bytes"] / (avg / 1e3) / 1e9, 1),
                  "TFLOP_s": round(wk["mfma_flops"] / (avg / 1e3) / 1e12, 2),
                  "direct_TFLOP_s": round(wk["flops"] / (avg / 1e3) / 1e12, 2)}
            if k in CONTRACTION_ROLES:
                st["mfma_frac"] = round(wk["mfma_flops"] / (avg / 1e3) / 1e12 / FP32_MFMA_PEAK_TFS, 4)
                cf = counter_flops(cfg, k)
                if cf is not None and not (args.block or args.fno):
                    st["counter_TFLOP_s"] = round(cf / (avg / 1e3) / 1e12, 2)
                    st["counter_mfma_frac"] = round(cf / (avg / 1e3) / 1e12 / FP32_MFMA_PEAK_TFS, 4)
            stages[k] = st
        dom = max((k for k in kernel_ms if k in w.work), key=lambda k: kernel_ms[k][0] * kernel_ms[k][1])
        n, avg = kernel_ms[dom]
        wk = w.work[dom]
        ach = wk["bytes"] / (avg / 1e3) / 1e9
        tr = None if args.block or args.fno else traffic_entry(cfg, dom)
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None if tr is None else int(tr),
                "algorithmic_bytes_per_launch": int(wk["bytes"]), "avg_launch_ms": round(avg, 4)}
        # The contraction kernel that executes the most MFMA work per step,
        # against the fp32 matrix peak: executed flops (after the folds) per
        # launch over its event-timed launch, and, where committed rocprof
        # counters of the same kernel source exist, the counted MFMA flops.
        cons = [k for k in kernel_ms if k in w.work and k in CONTRACTION_ROLES]
        if cons:
            dm = max(cons, key=lambda k: kernel_ms[k][0] * w.work[k]["mfma_flops"])
            n, avg = kernel_ms[dm]
            ex = w.work[dm]["mfma_flops"] / (avg / 1e3) / 1e12
            cf = None if args.block or args.fno else counter_flops(cfg, dm)
            roof_mfma = {"kernel": dm, "bound": "mfma", "achieved": round(ex, 2), "peak": FP32_MFMA_PEAK_TFS,
                         "unit": "TFLOP/s", "frac": round(ex / FP32_MFMA_PEAK_TFS, 4),
                         "executed_flops_per_launch": int(w.work[dm]["mfma_flops"]),
                         "counter_flops_per_launch": None if cf is None else int(cf),
                         "counter_frac": None if cf is None else round(cf / (avg / 1e3) / 1e12 / FP32_MFMA_PEAK_TFS, 4),
                         "avg_launch_ms": round(avg, 4)}
            # every contraction kernel together: executed MFMA flops over their summed time
            tot_f = sum(w.work[k]["mfma_flops"] * kernel_ms[k][0] for k in cons)
            tot_s = sum(kernel_ms[k][0] * kernel_ms[k][1] / 1e3 for k in cons)
            roof_mfma["all_contraction_kernels_frac"] = round(tot_f / tot_s / 1e12 / FP32_MFMA_PEAK_TFS, 4)

    out = {
        "metric": w.metric,
        "value": round(gbs, 2), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "launch": "hip_graph" if args.graph else "eager",
        "step_ms": {"mean": round(ms_per_step, 4), "median": round(per_step[len(per_step) // 2], 4),
                    "min": round(per_step[0], 4), "note": "median and min from a separate pass that brackets "
                                                          "each step with its own events"},
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "layer_ms": round(ms_per_step, 4),
        # executed flops: the products the kernels perform after the exact folds
        "layer_TFLOP_s": round(w.mfma_flops / sec / 1e12, 3),
        # the per-dimension contractions as defined (Table 3's stage counts, in real flops)
        "layer_direct_TFLOP_s": round(w.flops / sec / 1e12, 3),
        "layer_bytes": int(w.bytes), "layer_executed_flops": int(w.mfma_flops), "layer_direct_flops": int(w.flops),
        "config": w.config,
        "roofline": roof, "roofline_mfma": roof_mfma, "stages": stages,
    }
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
