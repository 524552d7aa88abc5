"""Seeded synthetic inputs for the DTST spectral-layer workloads.

This module is shared by the tests, the bench and the smoke check.  It holds
no arithmetic of the transform itself: it only describes the five workload
shapes and draws seeded random tensors (Gaussian shards, complex weights,
upstream gradients, a smooth random field built from a few random plane
waves).  Every array it returns is fed unchanged to both the HIP library and
the fp64 CPU oracle.

Seeds: input 1000*cfg, weights 1000*cfg + 1, upstream gradient 1000*cfg + 2,
synthetic spectra 1000*cfg + 3, bypass weights 1000*cfg + 4, lift 1000*cfg + 5,
projection 1000*cfg + 6 (the Fourier layer l of an FNO adds 10*l to the weight
and bypass seeds).

The paper's workload (PDEBench 3D compressible Navier-Stokes, 128^3 x 21
steps, d_v = 20, modes (8, 8, 8, 16)) is not available here; these fields
stand in for it with the shapes, channel counts and truncations listed
below.
"""

from __future__ import annotations

import math

import numpy as np

# ---------------------------------------------------------------------------
# Workload table.  Sizes are (x, y, z, t).  kmax = (kx, ky, kz): x, y, z keep
# 2*k indices; kt: t keeps 0..kt-1.
# ---------------------------------------------------------------------------
WORKLOADS = {
    1: dict(name="full-domain 32^3x8, B1 C8, modes 16/16/16/4",
            n_global=(32, 32, 32, 8), n_local=(32, 32, 32, 8), shards=1,
            kmax=(8, 8, 8), kt=4, batch=1, c_in=8, c_out=8, field="normal"),
    2: dict(name="128^3x32 in 8 x-slabs of 16, B1 C16, modes 32/32/32/8",
            n_global=(128, 128, 128, 32), n_local=(16, 128, 128, 32), shards=8,
            kmax=(16, 16, 16), kt=8, batch=1, c_in=16, c_out=16,
            field="normal+waves"),
    3: dict(name="shard 64x256x256x32 of 256^3x32 (x/4), B2 C32, modes 32/32/32/8",
            n_global=(256, 256, 256, 32), n_local=(64, 256, 256, 32), shards=4,
            shard=1, kmax=(16, 16, 16), kt=8, batch=2, c_in=32, c_out=32,
            field="normal"),
    4: dict(name="shard 32x512x512x32 of 512^3x32 (x/16), B1 C32, modes 32/32/32/8",
            n_global=(512, 512, 512, 32), n_local=(32, 512, 512, 32), shards=16,
            shard=1, kmax=(16, 16, 16), kt=8, batch=1, c_in=32, c_out=32,
            field="smooth"),
    5: dict(name="backward on the 64x256x256x32 shard, B2 C32, modes 64/64/64/16",
            n_global=(256, 256, 256, 32), n_local=(64, 256, 256, 32), shards=4,
            shard=1, kmax=(32, 32, 32), kt=16, batch=2, c_in=32, c_out=32,
            field="normal"),
    # Not one of the five reference workloads: the grid of workload 2 under the
    # paper's 2-D (pencil) decomposition, x and y both distributed.
    6: dict(name="128^3x32 in 2x4 (x, y) pencils of 64x32, B1 C16, modes 32/32/32/8",
            n_global=(128, 128, 128, 32), n_local=(64, 32, 128, 32), shards=8, grid=(2, 4),
            kmax=(16, 16, 16), kt=8, batch=1, c_in=16, c_out=16,
            field="normal+waves"),
    # The paper's model (Sec. VI-A): d_v = 20, 4 Fourier layers, modes (8, 8, 8, 16),
    # 128^3 grid in 4 x-slabs; 5 input and 5 output fields as in 3D compressible
    # Navier-Stokes; N_t = 32 so that k_t = 16 is a half spectrum.
    7: dict(name="FNO forward: 128^3x32 in 4 x-slabs of 32, B1, lift 5->20, 4 blocks, modes 16/16/16/16, proj 20->5",
            n_global=(128, 128, 128, 32), n_local=(32, 128, 128, 32), shards=4,
            kmax=(8, 8, 8), kt=16, batch=1, c_in=20, c_out=20, field="normal",
            fno=dict(c_data_in=5, c_data_out=5, layers=4)),
}

# Workloads whose every shard is run, one after another, on the one GPU.
ALL_SHARDS = (2, 6, 7)

# Plane waves planted in every channel of workload 2: (k, phase), amplitude 5.
# k is a signed (x, y, z, t) wavenumber.  The second wave sits on the -k_max
# boundary index with k_t = 0 (its partner +16 is not retained); the third on
# the last retained k_t.
CFG2_WAVES = (((3, -5, 7, 2), 0.0),
              ((-16, 15, 0, 0), math.pi / 3),
              ((9, 0, -12, 7), -math.pi / 4))
CFG2_AMPLITUDE = 5.0


def seed_of(cfg: int, what: str) -> int:
    return 1000 * cfg + {"input": 0, "weights": 1, "upstream": 2, "spectrum": 3, "bypass": 4, "lift": 5,
                         "proj": 6}[what]


def fno_params_np(M, dv, c_in, c_out, layers, seed):
    """Seeded FNO parameters as host arrays: lift (w (dv, c_in), b (dv,)),
    layers [(R (M, dv, dv) complex64 with E|R|^2 = 1/dv^2, W (dv, dv) float32
    ~ N(0, 1/dv))], projection (w (c_out, dv), b (c_out,)); the scales keep the
    activations of order one through the layers."""
    lift = (np_normal((dv, c_in), seed + 5, std=1.0 / math.sqrt(c_in)), np_normal((dv,), seed + 15, std=0.1))
    blocks = [(np_weights(M, dv, dv, seed + 1 + 10 * l), np_normal((dv, dv), seed + 4 + 10 * l, std=1.0 / math.sqrt(dv)))
              for l in range(layers)]
    proj = (np_normal((c_out, dv), seed + 6, std=1.0 / math.sqrt(dv)), np_normal((c_out,), seed + 16, std=0.1))
    return lift, blocks, proj


def geometry(cfg: int, shard: int | None = None) -> dict:
    """Plain-dict description of one shard of workload ``cfg``.  Shards are
    numbered row-major over the (x, y) shard grid (x slabs: grid (P, 1))."""
    c = WORKLOADS[cfg]
    p = c.get("shard", 0) if shard is None else shard
    gx, gy = c.get("grid", (c["shards"], 1))
    off = ((p // gy) * c["n_local"][0], (p % gy) * c["n_local"][1], 0, 0)
    return dict(n_global=tuple(c["n_global"]), n_local=tuple(c["n_local"]),
                offset=off, kmax=tuple(c["kmax"]), kt=c["kt"],
                batch=c["batch"], c_in=c["c_in"], c_out=c["c_out"])


def full_domain(cfg: int) -> dict:
    """The same workload as one shard covering the whole global grid."""
    g = geometry(cfg, 0)
    g["n_local"] = g["n_global"]
    g["offset"] = (0, 0, 0, 0)
    return g


def n_modes(g: dict) -> int:
    k = g["kmax"]
    return (2 * k[0]) * (2 * k[1]) * (2 * k[2]) * g["kt"]


# ---------------------------------------------------------------------------
# Host (numpy) generators for small cases
# ---------------------------------------------------------------------------
def np_normal(shape, seed, std=1.0, dtype=np.float32):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape) * std).astype(dtype)


def np_complex_normal(shape, seed, var=1.0):
    """Circular complex normal with E|w|^2 = var (each part var/2)."""
    rng = np.random.default_rng(seed)
    s = math.sqrt(var / 2.0)
    re = rng.standard_normal(shape) * s
    im = rng.standard_normal(shape) * s
    return (re + 1j * im).astype(np.complex64)


def np_weights(m_count, c_in, c_out, seed):
    """Spectral weights (m, C_in, C_out) with E|w|^2 = 1/(C_in C_out)."""
    return np_complex_normal((m_count, c_in, c_out), seed, var=1.0 / (c_in * c_out))


def plane_wave_np(g: dict, k, phase, amp=1.0):
    """amp * cos(2 pi sum_i k_i n_i / N_i + phase) on the shard's global
    coordinates, float64, shape n_local.  The phase k_i*n_i is reduced
    modulo N_i in integers before the angle is formed."""
    nl, off, ng = g["n_local"], g["offset"], g["n_global"]
    total = np.zeros(tuple(nl), dtype=np.float64)
    for i in range(4):
        n = off[i] + np.arange(nl[i], dtype=np.int64)
        frac = ((k[i] * n) % ng[i]).astype(np.float64) / ng[i]
        shp = [1, 1, 1, 1]
        shp[i] = nl[i]
        total = total + frac.reshape(shp)
    return amp * np.cos(2.0 * math.pi * total + phase)


# ---------------------------------------------------------------------------
# Device (torch) generators for full-size workloads
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def torch_normal(shape, seed, device, std=1.0):
    torch = _torch()
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(0.0, std, generator=gen)
    return t


def torch_complex_normal(shape, seed, device, var=1.0):
    torch = _torch()
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    t = torch.empty(tuple(shape) + (2,), dtype=torch.float32, device=device)
    t.normal_(0.0, math.sqrt(var / 2.0), generator=gen)
    return torch.view_as_complex(t)


def torch_weights(m_count, c_in, c_out, seed, device):
    return torch_complex_normal((m_count, c_in, c_out), seed, device,
                                var=1.0 / (c_in * c_out))


def torch_bypass(c_out, c_in, seed, device):
    """Real point-wise bypass weights (C_out x C_in), N(0, 1/C_in)."""
    return torch_normal((c_out, c_in), seed, device, std=1.0 / math.sqrt(c_in))


def torch_plane_wave_(out, g, k, phase, amp):
    """out[...] += amp*cos(2 pi k.n/N + phase) over the shard (float64 math)."""
    torch = _torch()
    nl, off, ng = g["n_local"], g["offset"], g["n_global"]
    total = torch.zeros((), dtype=torch.float64, device=out.device)
    for i in range(4):
        n = off[i] + torch.arange(nl[i], dtype=torch.int64, device=out.device)
        frac = ((k[i] * n) % ng[i]).to(torch.float64) / ng[i]
        shp = [1, 1, 1, 1]
        shp[i] = nl[i]
        total = total + frac.reshape(shp)
    out += (amp * torch.cos(2.0 * math.pi * total + phase)).to(out.dtype)


def torch_smooth_field(g, channels, seed, device, waves=48, width=8.0, noise_std=0.1):
    """Smooth random field per channel: a sum of ``waves`` random plane
    waves with integer wavenumbers |k_x,y,z| <= 24, 0 <= k_t <= 15 and
    Gaussian-spectrum amplitudes ~ N(0,1) exp(-|k|^2 / (2 width^2)),
    normalised to unit RMS, plus N(0, noise_std^2) noise.

    Evaluated as a rank-``waves`` product of per-axis phase factors on the
    shard's global coordinates.  Returns (channels, *n_local) float32.
    """
    torch = _torch()
    rng = np.random.default_rng(seed)
    nl, off, ng = g["n_local"], g["offset"], g["n_global"]
    out = torch.empty((channels,) + tuple(nl), dtype=torch.float32, device=device)
    axes = [off[i] + np.arange(nl[i], dtype=np.int64) for i in range(4)]
    for ch in range(channels):
        ks = np.stack([rng.integers(-24, 25, waves), rng.integers(-24, 25, waves),
                       rng.integers(-24, 25, waves), rng.integers(0, 16, waves)], 1)
        amp = rng.standard_normal(waves) * np.exp(-(ks ** 2).sum(1) / (2 * width ** 2))
        ph = rng.uniform(0, 2 * math.pi, waves)
        fac = []
        for i in range(4):
            frac = ((ks[:, i:i + 1] * axes[i][None, :]) % ng[i]) / ng[i]
            fac.append(np.exp(2j * math.pi * frac))            # (waves, n_i)
        u = (amp * np.exp(1j * ph))[:, None, None] * fac[0][:, :, None] * fac[1][:, None, :]
        v = fac[2][:, :, None] * fac[3][:, None, :]
        U = torch.from_numpy(u.reshape(waves, -1).T.astype(np.complex64)).to(device)
        V = torch.from_numpy(v.reshape(waves, -1).astype(np.complex64)).to(device)
        f = torch.matmul(U, V).real.reshape(tuple(nl))
        f = f / f.pow(2).mean().sqrt().clamp_min(1e-30)
        out[ch] = f
    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 7)
    noise = torch.empty_like(out)
    noise.normal_(0.0, noise_std, generator=gen)
    out += noise
    return out


def torch_input(cfg: int, g: dict, device, channels_first=True):
    """Input shard x (B, C_in, *n_local) float32 for workload ``cfg``."""
    torch = _torch()
    c = WORKLOADS[cfg]
    shape = (g["batch"], g["c_in"]) + tuple(g["n_local"])
    kind = c["field"]
    if kind == "smooth":
        x = torch.empty(shape, dtype=torch.float32, device=device)
        for b in range(g["batch"]):
            x[b] = torch_smooth_field(g, g["c_in"], seed_of(cfg, "input") + 17 * b, device)
        return x
    x = torch_normal(shape, seed_of(cfg, "input"), device)
    if kind == "normal+waves":
        for k, ph in CFG2_WAVES:
            torch_plane_wave_(x, g, k, ph, CFG2_AMPLITUDE)
    return x
