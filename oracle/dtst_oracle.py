"""Plain, slow, fp64 CPU oracle for the DTST spectral-layer path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, table or
constant with the HIP library; both sides only consume the same seeded
inputs.

What it computes (paper: "DRIFT: Direct Reduced Fourier Transforms for
Distributed Spectral Neural Operators", arXiv 2607.14394):

* retained index sets           -- Sec. III (definition of S_j), Fig. 5
* forward partial spectrum      -- Sec. IV-B, Eq. (full_dft) restricted to one
                                   shard dom(p) as in Eq. (dtst_decompose), with
                                   the offset basis of Sec. V-B Eq. (basis_matrix)
* shard sum                     -- Sec. IV-B, Eq. (dtst_reduce)
* mode-wise channel mix         -- Sec. V-A, Eq. (partitioned_conv)
* inverse partial DFT           -- Sec. V-A, Eq. (dtst_inverse), with the
                                   half-spectrum reading for t (see below)
* adjoints / weight gradient    -- Sec. V-C (backward pass), worked out with
                                   respect to <a, b> = Re sum conj(a) b
* block epilogue                -- Sec. V (block structure), Algorithm 1: the
                                   point-wise bypass W x added to the spectral
                                   output, through GELU
* FNO forward                   -- Sec. II: lift P, L Fourier layers (each as
                                   Algorithm 1), projection Q

Readings taken where the paper is silent:

* x, y, z keep {0..k-1} U {N-k..N-1} (Sec. III); t keeps {0..K_t-1} only, the
  half spectrum of a real signal (Table 3 contracts T 30 -> 16 for k_t = 16).
* The inverse of a half spectrum follows the real-inverse-FFT convention:
  y[n] = (1/prod N) Re sum_k w(k_t) Yhat[k] conj(phi_k(n)), w(0) = 1,
  w(N_t/2) = 1 for even N_t, w = 2 otherwise.
* Mix: Yhat[b,o,m] = sum_i Xhat[b,i,m] W[m,i,o], no conjugation.
* Phases are reduced as exact integers, (k * n) mod N, before any trig call.
* GELU is the exact form v Phi(v) (erf), the bypass W a real (C_out x C_in)
  matrix with no bias (Algorithm 1 names neither an approximation nor a bias).
* The point-wise networks P and Q of the FNO (Sec. II names them, not their
  depth) are single linear layers with a bias; every Fourier layer, the last
  included, ends in GELU as Algorithm 1 returns it.

Every routine works in float64 / complex128.  Contractions are done one
dimension at a time (the DFT kernel is a product over dimensions), in the
paper's order T, Z, Y, X for the forward and X, Y, Z, T for the inverse
(Algorithm 1).  The library primitives used are ``np.tensordot`` and
``np.einsum`` (contractions) and ``scipy.special.erf``.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

__all__ = [
    "Geometry", "retained_indices", "retained_t", "basis", "half_weights",
    "forward", "inverse", "forward_adj", "inverse_adj", "mix",
    "mix_data_grad", "mix_wgrad", "forward_at_modes", "inverse_at_points", "forward_adj_at_points",
    "n_modes", "mode_index", "gelu", "block_epilogue", "pointwise", "fno_forward",
]


# ---------------------------------------------------------------------------
# Geometry of one shard (Sec. IV-A problem setting, Sec. V-B offsets)
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class Geometry:
    """One shard of the global (x, y, z, t) grid and the retained modes.

    n_global, n_local, offset: per dimension (x, y, z, t).  The shard holds
    global indices offset[i] .. offset[i] + n_local[i] - 1 (Sec. IV-A: GPU p
    holds a contiguous block; Sec. V-B: offset p_i N_i^loc).
    kmax: (k_x, k_y, k_z) -- x, y, z keep 2*k indices each (Sec. III).
    kt: number of retained t indices 0..kt-1 (half spectrum).
    """
    n_global: tuple
    n_local: tuple
    offset: tuple
    kmax: tuple
    kt: int
    batch: int = 1
    c_in: int = 1
    c_out: int = 1

    @property
    def K(self):
        return (2 * self.kmax[0], 2 * self.kmax[1], 2 * self.kmax[2], self.kt)

    def validate(self):
        for i in range(4):
            if not (1 <= self.n_local[i] and 0 <= self.offset[i]
                    and self.offset[i] + self.n_local[i] <= self.n_global[i]):
                raise ValueError(f"dimension {i}: bad extent/offset")
        for i in range(3):
            if not (1 <= 2 * self.kmax[i] <= self.n_global[i]):
                raise ValueError(f"dimension {i}: need 1 <= 2k <= N")
        if not (1 <= self.kt <= self.n_global[3] // 2 + 1):
            raise ValueError("t: need 1 <= kt <= N_t/2 + 1")


def retained_indices(n: int, k: int) -> np.ndarray:
    """Stored indices of S_j = {0..k-1} U {N-k..N-1} in ascending order.

    Sec. III, definition of S_j; Fig. 5 caption (N = 128, K = 16 keeps rows
    0..7 and 120..127).
    """
    return np.array(list(range(k)) + list(range(n - k, n)), dtype=np.int64)


def retained_t(kt: int) -> np.ndarray:
    """t keeps 0..kt-1 (half spectrum; Table 3 reading)."""
    return np.arange(kt, dtype=np.int64)


def basis(n_global: int, offset: int, n_local: int, idx: np.ndarray) -> np.ndarray:
    """B[k, j] = W_N^{k (offset + j)}, W_N = exp(-2 pi i / N).

    Sec. V-B, Eq. (basis_matrix).  The exponent k*(offset+j) is reduced
    modulo N in exact integer arithmetic, then turned into an angle in fp64.
    """
    k = np.asarray(idx, dtype=np.int64)[:, None]
    n = offset + np.arange(n_local, dtype=np.int64)[None, :]
    r = (k * n) % n_global
    ang = -2.0 * math.pi * r.astype(np.float64) / float(n_global)
    return np.cos(ang) + 1j * np.sin(ang)


def half_weights(nt: int, kt: int) -> np.ndarray:
    """Real-inverse weights for the stored half spectrum in t.

    w(0) = 1; w(N_t/2) = 1 if N_t is even and that index is stored; else 2.
    (Reading of Sec. V-A Eq. (dtst_inverse) for a half spectrum.)
    """
    w = np.full(kt, 2.0)
    w[0] = 1.0
    if nt % 2 == 0 and kt > nt // 2:
        w[nt // 2] = 1.0
    return w


def _bases(g: Geometry):
    idx = [retained_indices(g.n_global[i], g.kmax[i]) for i in range(3)]
    idx.append(retained_t(g.kt))
    return [basis(g.n_global[i], g.offset[i], g.n_local[i], idx[i]) for i in range(4)]


def n_modes(g: Geometry) -> int:
    K = g.K
    return K[0] * K[1] * K[2] * K[3]


def mode_index(g: Geometry, ix, iy, iz, it):
    """Flattened mode index m = ((ix*Ky + iy)*Kz + iz)*Kt + it (row-major)."""
    K = g.K
    return ((ix * K[1] + iy) * K[2] + iz) * K[3] + it


# ---------------------------------------------------------------------------
# Forward partial spectrum of one shard (Eq. dtst_decompose, one term X_p)
# ---------------------------------------------------------------------------
def forward(x: np.ndarray, g: Geometry, scale_t=None) -> np.ndarray:
    """X_p[b,c,k] = sum_{n in dom(p)} x[b,c,n] prod_i W_{N_i}^{k_i n_i}.

    x: (B, C, Nx_loc, Ny_loc, Nz_loc, Nt_loc), real.  Returns complex128
    (B, C, Kx, Ky, Kz, Kt).  Contracts T, then Z, Y, X (Algorithm 1).
    ``scale_t`` (length Kt) multiplies the result along k_t; used by
    ``inverse_adj``.
    """
    x = np.asarray(x, dtype=np.float64)
    Bx, By, Bz, Bt = _bases(g)
    K = g.K
    out = np.empty(x.shape[:2] + tuple(K), dtype=np.complex128)
    for b in range(x.shape[0]):
        for c in range(x.shape[1]):
            v = x[b, c]                                  # (X, Y, Z, T)
            v = np.tensordot(v, Bt, axes=([3], [1]))     # (X, Y, Z, Kt)
            v = np.tensordot(v, Bz, axes=([2], [1]))     # (X, Y, Kt, Kz)
            v = np.tensordot(v, By, axes=([1], [1]))     # (X, Kt, Kz, Ky)
            v = np.tensordot(v, Bx, axes=([0], [1]))     # (Kt, Kz, Ky, Kx)
            v = v.transpose(3, 2, 1, 0)                  # (Kx, Ky, Kz, Kt)
            if scale_t is not None:
                v = v * np.asarray(scale_t)[None, None, None, :]
            out[b, c] = v
    return out


def forward_at_modes(x_bc: np.ndarray, g: Geometry, modes) -> np.ndarray:
    """Forward coefficients of one (b, c) slice at a list of (ix, iy, iz, it)
    positions, each evaluated as its own direct sum over the shard.

    Used to check outputs of very large shards one coefficient at a time.
    """
    x_bc = np.asarray(x_bc, dtype=np.float64)
    Bx, By, Bz, Bt = _bases(g)
    res = np.empty(len(modes), dtype=np.complex128)
    for q, (ix, iy, iz, it) in enumerate(modes):
        v = x_bc @ Bt[it]              # (X, Y, Z)
        v = v @ Bz[iz]                 # (X, Y)
        v = v @ By[iy]                 # (X,)
        res[q] = v @ Bx[ix]
    return res


# ---------------------------------------------------------------------------
# Inverse partial DFT onto the shard (Eq. dtst_inverse, half spectrum in t)
# ---------------------------------------------------------------------------
def _expand(yhat: np.ndarray, g: Geometry, wt: np.ndarray) -> np.ndarray:
    """Re sum_k wt[k_t] Yhat[k] conj(phi_k(n)) for n in dom(p).

    Expands X, then Y, Z, T (reverse of the forward order, Sec. V-B)."""
    yhat = np.asarray(yhat, dtype=np.complex128)
    Bx, By, Bz, Bt = _bases(g)
    Cx, Cy, Cz, Ct = (np.conj(B) for B in (Bx, By, Bz, Bt))
    Ct = Ct * wt[:, None]
    nl = g.n_local
    out = np.empty(yhat.shape[:2] + tuple(nl), dtype=np.float64)
    for b in range(yhat.shape[0]):
        for c in range(yhat.shape[1]):
            v = yhat[b, c]                               # (Kx, Ky, Kz, Kt)
            v = np.tensordot(v, Cx, axes=([0], [0]))     # (Ky, Kz, Kt, X)
            v = np.tensordot(v, Cy, axes=([0], [0]))     # (Kz, Kt, X, Y)
            v = np.tensordot(v, Cz, axes=([0], [0]))     # (Kt, X, Y, Z)
            v = np.tensordot(v, Ct, axes=([0], [0]))     # (X, Y, Z, T)
            out[b, c] = v.real
    return out


def inverse(yhat: np.ndarray, g: Geometry) -> np.ndarray:
    """y_p[n] = (1/prod N_i) Re sum_{k in S} w(k_t) Yhat[k] prod_i W^{-k_i n_i}.

    Sec. V-A, Eq. (dtst_inverse); the w(k_t) weights and the real part are
    the half-spectrum reading.  Output (B, C, Nx_loc, .., Nt_loc) float64.
    """
    ntot = float(np.prod(np.asarray(g.n_global, dtype=np.float64)))
    w = half_weights(g.n_global[3], g.kt) / ntot
    return _expand(yhat, g, w)


def inverse_at_points(yhat_bc: np.ndarray, g: Geometry, points) -> np.ndarray:
    """Inverse of one (b, c) slice at a list of local points (x, y, z, t),
    each one its own sum over all retained modes."""
    ntot = float(np.prod(np.asarray(g.n_global, dtype=np.float64)))
    return _expand_at_points(yhat_bc, g, points, half_weights(g.n_global[3], g.kt) / ntot)


def forward_adj_at_points(g_xhat_bc: np.ndarray, g: Geometry, points) -> np.ndarray:
    """``forward_adj`` of one (b, c) slice at a list of local points."""
    return _expand_at_points(g_xhat_bc, g, points, np.ones(g.kt))


def _expand_at_points(yhat_bc, g, points, w):
    yhat_bc = np.asarray(yhat_bc, dtype=np.complex128)
    Bx, By, Bz, Bt = _bases(g)
    res = np.empty(len(points), dtype=np.float64)
    for q, (px, py, pz, pt) in enumerate(points):
        v = np.tensordot(yhat_bc, np.conj(Bt[:, pt]) * w, axes=([3], [0]))
        v = np.tensordot(v, np.conj(Bz[:, pz]), axes=([2], [0]))
        v = np.tensordot(v, np.conj(By[:, py]), axes=([1], [0]))
        res[q] = np.dot(v, np.conj(Bx[:, px])).real
    return res


# ---------------------------------------------------------------------------
# Adjoints (Sec. V-C), inner product <a, b> = Re sum conj(a) b
# ---------------------------------------------------------------------------
def forward_adj(g_xhat: np.ndarray, g: Geometry) -> np.ndarray:
    """Adjoint of ``forward`` (real input -> complex modes):
    g_x[n] = Re sum_k G[k] conj(phi_k(n)); no 1/N, no half weights."""
    return _expand(g_xhat, g, np.ones(g.kt))


def inverse_adj(g_y: np.ndarray, g: Geometry) -> np.ndarray:
    """Adjoint of ``inverse``: G[k] = (w(k_t)/prod N) sum_n g_y[n] phi_k(n)."""
    ntot = float(np.prod(np.asarray(g.n_global, dtype=np.float64)))
    return forward(g_y, g, scale_t=half_weights(g.n_global[3], g.kt) / ntot)


# ---------------------------------------------------------------------------
# Mode-wise channel mix on a mode range (Sec. V-A, Eq. partitioned_conv)
# ---------------------------------------------------------------------------
def _flat(a):
    a = np.asarray(a)
    return a.reshape(a.shape[0], a.shape[1], -1)


def mix(xhat, w, m0, m1, yhat_in=None, c_out=None):
    """Yhat[b,o,m] = sum_i Xhat[b,i,m] W[m-m0,i,o] for m in [m0, m1).

    xhat: (B, C_in, M...) complex; w: (m1-m0, C_in, C_out).  Columns outside
    [m0, m1) are copied from ``yhat_in`` (zeros when it is None), so running
    the disjoint ranges S_p one after another assembles the whole Yhat (the
    reassembly of Eq. allgather on one device).
    """
    xf = _flat(xhat).astype(np.complex128)
    w = np.asarray(w, dtype=np.complex128)
    B, Ci, M = xf.shape
    Co = w.shape[2] if c_out is None else c_out
    if yhat_in is None:
        yf = np.zeros((B, Co, M), dtype=np.complex128)
    else:
        yf = _flat(yhat_in).astype(np.complex128).copy()
    for b in range(B):
        # (m, i) x (m, i, o) -> (m, o)
        xs = xf[b, :, m0:m1].T
        yf[b, :, m0:m1] = np.einsum("mi,mio->om", xs, w)
    return yf


def mix_data_grad(g_yhat, w, m0, m1, gx_in=None, c_in=None):
    """Adjoint of ``mix`` in Xhat: G_X[b,i,m] = sum_o G_Y[b,o,m] conj(W[m,i,o])."""
    gf = _flat(g_yhat).astype(np.complex128)
    w = np.asarray(w, dtype=np.complex128)
    B, Co, M = gf.shape
    Ci = w.shape[1] if c_in is None else c_in
    if gx_in is None:
        out = np.zeros((B, Ci, M), dtype=np.complex128)
    else:
        out = _flat(gx_in).astype(np.complex128).copy()
    for b in range(B):
        gs = gf[b, :, m0:m1].T                       # (m, o)
        out[b, :, m0:m1] = np.einsum("mo,mio->im", gs, np.conj(w))
    return out


def mix_wgrad(xhat, g_yhat, m0, m1, gw_in=None):
    """Weight gradient on the local mode range (Sec. V-A, Sec. V-C):
    G_W[m-m0,i,o] = sum_b conj(Xhat[b,i,m]) G_Y[b,o,m] (+ gw_in)."""
    xf = _flat(xhat).astype(np.complex128)
    gf = _flat(g_yhat).astype(np.complex128)
    gw = np.einsum("bim,bom->mio", np.conj(xf[:, :, m0:m1]), gf[:, :, m0:m1])
    if gw_in is not None:
        gw = gw + np.asarray(gw_in, dtype=np.complex128)
    return gw


# ---------------------------------------------------------------------------
# Block epilogue (Sec. V "Block Structure", Algorithm 1: first and last step)
# ---------------------------------------------------------------------------
def gelu(v):
    """GELU(v) = v Phi(v) with Phi the standard normal CDF,
    Phi(v) = (1 + erf(v / sqrt 2)) / 2 (the exact form, not an approximation)."""
    from scipy.special import erf
    v = np.asarray(v, dtype=np.float64)
    return 0.5 * v * (1.0 + erf(v / math.sqrt(2.0)))


def block_epilogue(x, w_bypass, y):
    """out[b,o,n] = GELU(sum_i W[o,i] x[b,i,n] + y[b,o,n]): the point-wise
    linear bypass W x of the block input added to the spectral output y (the
    inverse partial DFT of the mixed spectrum), through the activation.

    x: (B, C_in, ...) real, w_bypass: (C_out, C_in) real, y: (B, C_out, ...)."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w_bypass, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    y0 = np.tensordot(w, x, axes=([1], [1]))          # (C_out, B, ...)
    return gelu(np.moveaxis(y0, 0, 1) + y)


# ---------------------------------------------------------------------------
# FNO forward (Sec. II: lift P, L Fourier layers, projection Q)
# ---------------------------------------------------------------------------
def pointwise(x, w, bias=None, act=False):
    """y[b,o,n] = act(sum_i W[o,i] x[b,i,n] + bias[o]): a point-wise linear
    layer, the reading of the lift P and the projection Q; act applies GELU.

    x: (B, C_in, ...) real, w: (C_out, C_in) real, bias: (C_out,) or None."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    y = np.moveaxis(np.tensordot(w, x, axes=([1], [1])), 0, 1)   # (B, C_out, ...)
    if bias is not None:
        b = np.asarray(bias, dtype=np.float64)
        y = y + b.reshape((1, -1) + (1,) * (y.ndim - 2))
    return gelu(y) if act else y


def fno_forward(x, g: Geometry, lift, blocks, proj):
    """FNO forward on the whole domain g (offset 0, c_in = c_out = d_v):

        v_0     = P(x)                                   lift, (C_data_in -> d_v)
        v_{l+1} = GELU(W_l v_l + I(R_l F(v_l)))          Fourier layer l (Algorithm 1)
        out     = Q(v_L)                                 projection, (d_v -> C_data_out)

    F and I are the forward and inverse partial DFTs over the retained modes
    (``forward``, ``inverse``), R_l the mode-wise channel mix (``mix`` over all
    M modes), W_l the point-wise bypass.  lift = (w, bias), proj = (w, bias),
    blocks = [(R_l (M, d_v, d_v) complex, W_l (d_v, d_v) real), ...].  The
    result does not depend on how the domain is split into shards: the shard
    spectra sum to the whole-domain spectrum (Eq. dtst_reduce) and the inverse
    is evaluated point by point."""
    v = pointwise(x, lift[0], lift[1])
    M = n_modes(g)
    for r_l, w_l in blocks:
        xh = forward(v, g)
        yh = mix(xh, r_l, 0, M).reshape((v.shape[0], np.asarray(r_l).shape[2]) + g.K)
        v = block_epilogue(v, w_l, inverse(yh, g))
    return pointwise(v, proj[0], proj[1])
