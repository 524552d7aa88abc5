"""Pins for the fp64 oracle, each against something other than the oracle.

* brute-force direct sums written from Eq. (full_dft) with complex
  exponentials and no integer phase reduction (pure Python, tiny grids);
* numpy's FFT (rfftn / irfftn) followed by truncation, the route the paper
  compares against in Sec. VI-C;
* closed forms: single plane waves, and the Dirichlet sum on a slab;
* identities: linearity, shard additivity (Eq. dtst_reduce), F.I.F and the
  full-retention identity, dot-product adjoint identities;
* torch's own FFT + autograd for the whole layer backward.

A plausible slip in the oracle (dropped offset, conjugated basis, wrong
half-spectrum weight, transposed weight tensor) fails at least one case.
"""

import cmath
import math
import os

import numpy as np
import pytest

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# (n_global, n_local, offset, kmax, kt, B, C_in, C_out)
TINY = {
    "baseline": ((12, 10, 8, 8), (12, 10, 8, 8), (0, 0, 0, 0), (3, 2, 2), 3, 1, 2, 2),
    "slab": ((12, 10, 8, 8), (4, 10, 8, 8), (4, 0, 0, 0), (3, 2, 2), 3, 1, 2, 2),
    "pencil": ((12, 10, 8, 8), (4, 5, 8, 8), (8, 5, 0, 0), (3, 2, 2), 3, 2, 1, 3),
    "odd": ((9, 7, 5, 6), (9, 7, 5, 6), (0, 0, 0, 0), (2, 3, 1), 3, 1, 1, 1),
    "odd_shard": ((9, 7, 5, 6), (3, 7, 5, 6), (6, 0, 0, 0), (2, 3, 1), 4, 1, 1, 1),
    "nyquist_t": ((6, 6, 4, 6), (6, 6, 4, 6), (0, 0, 0, 0), (2, 2, 1), 4, 1, 1, 1),
    "k_gt_nloc": ((12, 6, 4, 4), (2, 6, 4, 4), (6, 0, 0, 0), (3, 1, 1), 2, 1, 1, 1),
    "all_modes": ((6, 4, 4, 6), (6, 4, 4, 6), (0, 0, 0, 0), (3, 2, 2), 4, 1, 1, 1),
    "t_shard": ((8, 6, 4, 10), (8, 6, 4, 5), (0, 0, 0, 5), (2, 2, 1), 4, 1, 2, 1),
}


def geo(name, **kw):
    ng, nl, off, k, kt, b, ci, co = TINY[name]
    g = O.Geometry(ng, nl, off, k, kt, b, ci, co)
    g.validate()
    return g


def rand_shard(g, seed, channels=None):
    c = g.c_in if channels is None else channels
    return synth.np_normal((g.batch, c) + tuple(g.n_local), seed, dtype=np.float64)


def rel(a, b):
    return np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(np.ravel(b)), 1e-300)


# ---------------------------------------------------------------------------
def test_fig5_retained_rows_golden():
    with open(os.path.join(GOLDEN, "fig5_retained_rows.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    n, k = int(rows[0][0]), int(rows[0][1])
    want = [int(v) for v in rows[1]]
    assert O.retained_indices(n, k).tolist() == want


def test_mode_index_flattening():
    """The flattened mode order m = ((ix Ky + iy) Kz + iz) Kt + it (ascending
    stored index per dimension, Fig. 5; the contiguous S_p ranges of the
    equal partition of Sec. V-A are ranges of this m): numpy's row-major
    ravel_multi_index over (2kx, 2ky, 2kz, kt), the reshape of a
    (B, C, Kx, Ky, Kz, Kt) spectrum to (B, C, M) that the tests and the mix
    use, and the coefficient stored at m equal to a brute-force direct sum at
    the stored frequencies of (ix, iy, iz, it)."""
    g = O.Geometry((12, 10, 14, 8), (5, 10, 14, 8), (3, 0, 0, 0), (3, 2, 4), 3, 1, 1, 1)
    g.validate()
    K = g.K
    M = O.n_modes(g)
    assert M == int(np.prod(K))
    ix, iy, iz, it = np.meshgrid(*[np.arange(k) for k in K], indexing="ij")
    m = O.mode_index(g, ix, iy, iz, it)
    assert np.array_equal(m, np.ravel_multi_index((ix, iy, iz, it), K))
    assert np.array_equal(np.sort(m.ravel()), np.arange(M))                  # a bijection onto 0..M-1
    assert np.array_equal(np.arange(M).reshape(K)[ix, iy, iz, it], m)        # the (B, C, M) reshape
    # t fastest, then z, y, x: neighbouring stored indices are stride 1, Kt, Kz Kt, Ky Kz Kt apart
    assert O.mode_index(g, 0, 0, 0, 1) == 1 and O.mode_index(g, 0, 0, 1, 0) == K[3]
    assert O.mode_index(g, 0, 1, 0, 0) == K[2] * K[3] and O.mode_index(g, 1, 0, 0, 0) == K[1] * K[2] * K[3]
    # the coefficient at flattened m is the direct sum at the stored frequencies of its indices
    x = rand_shard(g, 55)
    flat = O.forward(x, g).reshape(1, 1, M)
    idx = [O.retained_indices(g.n_global[i], g.kmax[i]) for i in range(3)] + [O.retained_t(g.kt)]
    rng = np.random.default_rng(56)
    pts = np.stack(np.meshgrid(*[np.arange(nl) for nl in g.n_local], indexing="ij"), -1).reshape(-1, 4)
    glob = pts + np.asarray(g.offset)
    xv = x[0, 0].reshape(-1)
    for _ in range(12):
        a = tuple(int(rng.integers(0, k)) for k in K)
        freq = [int(idx[d][a[d]]) for d in range(4)]
        ph = sum(freq[d] * glob[:, d] / g.n_global[d] for d in range(4))
        want = sum(v * cmath.exp(-2j * math.pi * p) for v, p in zip(xv, ph))
        got = flat[0, 0, O.mode_index(g, *a)]
        assert abs(got - want) <= 1e-10 * max(1.0, abs(want)), (a, got, want)


def _brute_forward(x, g):
    """Eq. (full_dft) over dom(p) with plain complex exponentials."""
    K = g.K
    idx = [O.retained_indices(g.n_global[i], g.kmax[i]).tolist() for i in range(3)]
    idx.append(list(range(g.kt)))
    B, C = x.shape[:2]
    out = np.zeros((B, C) + tuple(K), dtype=np.complex128)
    nl, off, ng = g.n_local, g.offset, g.n_global
    for b in range(B):
        for c in range(C):
            for a0, k0 in enumerate(idx[0]):
                for a1, k1 in enumerate(idx[1]):
                    for a2, k2 in enumerate(idx[2]):
                        for a3, k3 in enumerate(idx[3]):
                            s = 0j
                            for j0 in range(nl[0]):
                                for j1 in range(nl[1]):
                                    for j2 in range(nl[2]):
                                        for j3 in range(nl[3]):
                                            ph = (k0 * (off[0] + j0) / ng[0] + k1 * (off[1] + j1) / ng[1]
                                                  + k2 * (off[2] + j2) / ng[2] + k3 * (off[3] + j3) / ng[3])
                                            s += x[b, c, j0, j1, j2, j3] * cmath.exp(-2j * math.pi * ph)
                            out[b, c, a0, a1, a2, a3] = s
    return out


@pytest.mark.parametrize("name", ["odd_shard", "k_gt_nloc"])
def test_forward_brute_force(name):
    g = geo(name)
    x = rand_shard(g, 11)
    ref = _brute_forward(x, g)
    got = O.forward(x, g)
    assert rel(got, ref) < 1e-12


def _fft_forward(x, g):
    """Embed the shard in the zero global grid, FFT, truncate (Sec. VI-C)."""
    B, C = x.shape[:2]
    full = np.zeros((B, C) + tuple(g.n_global))
    sl = tuple(slice(g.offset[i], g.offset[i] + g.n_local[i]) for i in range(4))
    full[(slice(None), slice(None)) + sl] = x
    F = np.fft.rfftn(full, axes=(2, 3, 4, 5))
    for ax in range(3):
        F = np.take(F, O.retained_indices(g.n_global[ax], g.kmax[ax]), axis=2 + ax)
    return F[..., :g.kt]


def _fft_inverse(yhat, g):
    B, C = yhat.shape[:2]
    ng = g.n_global
    spec = np.zeros((B, C, ng[0], ng[1], ng[2], ng[3] // 2 + 1), dtype=np.complex128)
    ix = [O.retained_indices(ng[a], g.kmax[a]) for a in range(3)]
    spec[np.ix_(range(B), range(C), ix[0], ix[1], ix[2], range(g.kt))] = yhat
    y = np.fft.irfftn(spec, s=ng, axes=(2, 3, 4, 5))
    sl = tuple(slice(g.offset[i], g.offset[i] + g.n_local[i]) for i in range(4))
    return y[(slice(None), slice(None)) + sl]


@pytest.mark.parametrize("name", sorted(TINY))
def test_forward_matches_fft_then_truncate(name):
    g = geo(name)
    x = rand_shard(g, 12)
    assert rel(O.forward(x, g), _fft_forward(x, g)) < 1e-13


@pytest.mark.parametrize("name", sorted(TINY))
def test_inverse_matches_irfftn_of_padded_spectrum(name):
    g = geo(name)
    K = g.K
    yhat = synth.np_complex_normal((g.batch, g.c_out) + tuple(K), 13).astype(np.complex128)
    assert rel(O.inverse(yhat, g), _fft_inverse(yhat, g)) < 1e-13


def test_exactness_level_moderate_grid():
    """Sec. VI-C reports a 3.2e-14 relative Frobenius error between FFT +
    truncation and the partial DFT in fp64; the oracle must reach that
    level too."""
    g = O.Geometry((48, 40, 32, 16), (48, 40, 32, 16), (0, 0, 0, 0), (8, 8, 8), 8, 1, 1, 1)
    x = synth.np_normal((1, 1, 48, 40, 32, 16), 14, dtype=np.float64)
    assert rel(O.forward(x, g), _fft_forward(x, g)) < 1e-13


def test_plane_wave_single_coefficient():
    """A cos(2 pi k0.n/N + phi) with 0 < k0_t < K_t puts A prod(N)/2 e^{i phi}
    on mode k0 and nothing anywhere else in the stored half spectrum."""
    g = geo("baseline")
    k0 = (2, -1, 1, 2)
    amp, ph = 1.7, 0.4
    gd = dict(n_global=g.n_global, n_local=g.n_local, offset=g.offset)
    x = synth.plane_wave_np(gd, k0, ph, amp)[None, None]
    X = O.forward(x, g)
    idx = [O.retained_indices(g.n_global[a], g.kmax[a]).tolist() for a in range(3)]
    pos = tuple(idx[a].index(k0[a] % g.n_global[a]) for a in range(3)) + (k0[3],)
    want = amp * np.prod(g.n_global) / 2 * cmath.exp(1j * ph)
    assert abs(X[(0, 0) + pos] - want) < 1e-10 * abs(want)
    X[(0, 0) + pos] = 0
    assert np.abs(X).max() < 1e-10 * abs(want)


def test_plane_wave_kt0_partner():
    """With k0_t = 0 the conjugate value also appears at -k0 when -k0 is
    retained, and is absent when it is not (the -k_max boundary)."""
    g = geo("baseline")
    gd = dict(n_global=g.n_global, n_local=g.n_local, offset=g.offset)
    N = np.prod(g.n_global)
    idx = [O.retained_indices(g.n_global[a], g.kmax[a]).tolist() for a in range(3)]
    for k0, partner_kept in (((1, -2, 1, 0), False), ((2, 1, -1, 0), True)):
        x = synth.plane_wave_np(gd, k0, 0.3, 1.0)[None, None]
        X = O.forward(x, g)
        p = tuple(idx[a].index(k0[a] % g.n_global[a]) for a in range(3)) + (0,)
        assert abs(X[(0, 0) + p] - N / 2 * cmath.exp(0.3j)) < 1e-9 * N
        negk = tuple((-k0[a]) % g.n_global[a] for a in range(3))
        if partner_kept:
            q = tuple(idx[a].index(negk[a]) for a in range(3)) + (0,)
            assert abs(X[(0, 0) + q] - N / 2 * cmath.exp(-0.3j)) < 1e-9 * N
        else:
            assert any(negk[a] not in idx[a] for a in range(3))
        nz = np.abs(X[0, 0]) > 1e-8 * N
        assert nz.sum() == (2 if partner_kept else 1)


def test_plane_wave_on_slab_dirichlet_closed_form():
    """On an x-slab, the x-sum of a plane wave is a geometric (Dirichlet)
    sum; the other dimensions contribute their full extent."""
    g = geo("slab")
    k0 = (5, 1, -1, 1)
    gd = dict(n_global=g.n_global, n_local=g.n_local, offset=g.offset)
    x = synth.plane_wave_np(gd, k0, 0.0, 1.0)[None, None]
    X = O.forward(x, g)
    Nx, o, L = g.n_global[0], g.offset[0], g.n_local[0]
    idx = [O.retained_indices(g.n_global[a], g.kmax[a]).tolist() for a in range(3)]
    rest = g.n_global[1] * g.n_global[2] * g.n_global[3] / 2
    for a0, kx in enumerate(idx[0]):
        d = (k0[0] - kx) % Nx
        if d == 0:
            s = L
        else:
            z = cmath.exp(2j * math.pi * d / Nx)
            s = z ** o * (1 - z ** L) / (1 - z)
        p = (a0, idx[1].index(k0[1] % g.n_global[1]), idx[2].index(k0[2] % g.n_global[2]), k0[3])
        assert abs(X[(0, 0) + p] - rest * s) < 1e-9 * rest * L


def test_linearity():
    g = geo("pencil")
    x = rand_shard(g, 21)
    y = rand_shard(g, 22)
    a, b = 0.7, -1.9
    assert rel(O.forward(a * x + b * y, g), a * O.forward(x, g) + b * O.forward(y, g)) < 1e-13


@pytest.mark.parametrize("split", ["x_slabs", "pencil_xy"])
def test_shard_additivity(split):
    """Eq. (dtst_reduce): the per-shard partial spectra sum to the full one."""
    ng = (12, 10, 8, 8)
    full = O.Geometry(ng, ng, (0, 0, 0, 0), (3, 2, 2), 3, 1, 2, 2)
    x = synth.np_normal((1, 2) + ng, 31, dtype=np.float64)
    parts = [(4, 10, 0, 0)] if split == "x_slabs" else [(4, 5, 0, 0)]
    px, py = (3, 1) if split == "x_slabs" else (3, 2)
    lx, ly = ng[0] // px, ng[1] // py
    acc = 0
    for i in range(px):
        for j in range(py):
            g = O.Geometry(ng, (lx, ly, 8, 8), (i * lx, j * ly, 0, 0), (3, 2, 2), 3, 1, 2, 2)
            acc = acc + O.forward(x[:, :, i * lx:(i + 1) * lx, j * ly:(j + 1) * ly], g)
    assert parts
    assert rel(acc, O.forward(x, full)) < 1e-13


def test_forward_inverse_forward():
    """F(I(F(x))) = F(x) except on k_t = 0 modes whose Hermitian partner is
    not retained, which come back exactly halved."""
    g = geo("baseline")
    x = rand_shard(g, 41)
    X = O.forward(x, g)
    X2 = O.forward(O.inverse(X, g), g)
    idx = [O.retained_indices(g.n_global[a], g.kmax[a]) for a in range(3)]
    expect = X.copy()
    for a0, kx in enumerate(idx[0]):
        for a1, ky in enumerate(idx[1]):
            for a2, kz in enumerate(idx[2]):
                kept = ((-kx) % g.n_global[0] in idx[0] and (-ky) % g.n_global[1] in idx[1]
                        and (-kz) % g.n_global[2] in idx[2])
                if not kept:
                    expect[:, :, a0, a1, a2, 0] *= 0.5
    assert rel(X2, expect) < 1e-12


def test_full_retention_identity():
    g = geo("all_modes")
    assert g.K[:3] == g.n_global[:3] and g.kt == g.n_global[3] // 2 + 1
    x = rand_shard(g, 42)
    assert rel(O.inverse(O.forward(x, g), g), x) < 1e-13


def _dot(a, b):
    return float(np.real(np.vdot(np.ravel(a), np.ravel(b))))


@pytest.mark.parametrize("name", ["pencil", "odd_shard", "nyquist_t", "t_shard"])
def test_adjoint_identities(name):
    g = geo(name)
    K = g.K
    x = rand_shard(g, 51)
    G = synth.np_complex_normal((g.batch, g.c_in) + tuple(K), 52).astype(np.complex128)
    assert abs(_dot(G, O.forward(x, g)) - _dot(O.forward_adj(G, g), x)) < 1e-10 * abs(_dot(G, O.forward(x, g)))
    Y = synth.np_complex_normal((g.batch, g.c_out) + tuple(K), 53).astype(np.complex128)
    gy = synth.np_normal((g.batch, g.c_out) + tuple(g.n_local), 54, dtype=np.float64)
    lhs = _dot(gy, O.inverse(Y, g))
    rhs = _dot(O.inverse_adj(gy, g), Y)
    assert abs(lhs - rhs) < 1e-10 * abs(lhs)


def test_mix_identities_and_loops():
    B, Ci, Co, M = 2, 3, 4, 10
    m0, m1 = 3, 8
    X = synth.np_complex_normal((B, Ci, M), 61).astype(np.complex128)
    W = synth.np_complex_normal((m1 - m0, Ci, Co), 62).astype(np.complex128)
    Y = O.mix(X, W, m0, m1)
    for b in range(B):
        for o in range(Co):
            for m in range(M):
                s = 0j
                if m0 <= m < m1:
                    for i in range(Ci):
                        s += X[b, i, m] * W[m - m0, i, o]
                assert abs(Y[b, o, m] - s) < 1e-13
    G = synth.np_complex_normal((B, Co, M), 63).astype(np.complex128)
    G_in = np.zeros_like(G)
    G_in[:, :, m0:m1] = G[:, :, m0:m1]
    lhs = _dot(G_in, Y)
    assert abs(lhs - _dot(O.mix_data_grad(G, W, m0, m1), X)) < 1e-12 * abs(lhs)
    assert abs(lhs - _dot(O.mix_wgrad(X, G, m0, m1), W)) < 1e-12 * abs(lhs)
    # B = C = 1 reduces to an elementwise product.
    x1, w1 = X[:1, :1], W[:, :1, :1]
    y1 = O.mix(x1, w1, m0, m1)
    assert np.allclose(y1[0, 0, m0:m1], x1[0, 0, m0:m1] * w1[:, 0, 0], rtol=0, atol=1e-14)
    # mode ranges pieced together equal the full-range mix
    Wfull = synth.np_complex_normal((M, Ci, Co), 64).astype(np.complex128)
    y_full = O.mix(X, Wfull, 0, M)
    y_pieces = None
    for a, b in ((0, 4), (4, 7), (7, 10)):
        y_pieces = O.mix(X, Wfull[a:b], a, b, yhat_in=y_pieces, c_out=Co)
    assert rel(y_pieces, y_full) < 1e-15


def test_backward_matches_torch_autograd():
    """Whole layer y = I(mix(F(x), W)) built from torch.fft (fp64, CPU);
    torch's autograd gives dL/dx and dL/dW for L = <g_y, y>.  The oracle's
    chain inverse_adj -> mix_data_grad / mix_wgrad -> forward_adj must
    agree (PyTorch's complex-gradient convention is dL/dRe + i dL/dIm)."""
    torch = pytest.importorskip("torch")
    g = geo("pencil")
    K = g.K
    M = int(np.prod(K))
    x = rand_shard(g, 71)
    W = synth.np_complex_normal((M, g.c_in, g.c_out), 72).astype(np.complex128)
    gy = synth.np_normal((g.batch, g.c_out) + tuple(g.n_local), 73, dtype=np.float64)

    xt = torch.tensor(x, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    ng = g.n_global
    pad = []
    for i in reversed(range(4)):
        pad += [g.offset[i], ng[i] - g.offset[i] - g.n_local[i]]
    full = torch.nn.functional.pad(xt, pad)
    F = torch.fft.rfftn(full, dim=(2, 3, 4, 5))
    ix = [torch.tensor(O.retained_indices(ng[a], g.kmax[a])) for a in range(3)]
    F = F.index_select(2, ix[0]).index_select(3, ix[1]).index_select(4, ix[2])[..., :g.kt]
    Xf = F.reshape(g.batch, g.c_in, M)
    Yf = torch.einsum("bim,mio->bom", Xf, Wt)
    Yr = Yf.reshape((g.batch, g.c_out) + tuple(K))
    spec = torch.zeros((g.batch, g.c_out, ng[0], ng[1], ng[2], ng[3] // 2 + 1), dtype=torch.complex128)
    I0, I1, I2 = torch.meshgrid(ix[0], ix[1], ix[2], indexing="ij")
    spec[:, :, I0, I1, I2, :g.kt] = Yr
    y = torch.fft.irfftn(spec, s=ng, dim=(2, 3, 4, 5))
    sl = [slice(None), slice(None)] + [slice(g.offset[i], g.offset[i] + g.n_local[i]) for i in range(4)]
    y = y[tuple(sl)]
    L = (y * torch.tensor(gy)).sum()
    L.backward()

    X = O.forward(x, g)
    assert rel(Xf.detach().numpy().reshape(X.shape), X) < 1e-12
    GY = O.inverse_adj(gy, g)
    GX = O.mix_data_grad(GY, W, 0, M).reshape(X.shape)
    GW = O.mix_wgrad(X, GY, 0, M)
    gx = O.forward_adj(GX, g)
    assert rel(gx, xt.grad.numpy()) < 1e-11
    assert rel(GW, Wt.grad.numpy()) < 1e-11


def _dirichlet(d, o, L, N):
    """sum_{n=o}^{o+L-1} exp(2 pi i d n / N)."""
    d %= N
    if d == 0:
        return complex(L)
    z = cmath.exp(2j * math.pi * d / N)
    return z ** o * (1 - z ** L) / (1 - z)


def wave_spectrum_closed_form(g, k0, phase, amp):
    """Forward of amp*cos(2 pi k0.n/N + phase) on shard g, mode by mode:
    (amp/2) [e^{i phase} prod_i D_i(k0_i - k_i) + e^{-i phase} prod_i D_i(-k0_i - k_i)]
    with D_i the Dirichlet sum over the shard's extent in dimension i."""
    idx = [O.retained_indices(g.n_global[a], g.kmax[a]) for a in range(3)] + [np.arange(g.kt)]
    out = np.zeros(tuple(g.K), dtype=np.complex128)
    for sgn, ph in ((1, phase), (-1, -phase)):
        fac = [np.array([_dirichlet(sgn * k0[a] - int(k), g.offset[a], g.n_local[a], g.n_global[a])
                         for k in idx[a]]) for a in range(4)]
        out += (amp / 2) * cmath.exp(1j * ph) * np.einsum("a,b,c,d->abcd", *fac)
    return out


def test_planted_waves_closed_form_on_slab():
    """Workload-2 style pin at tiny size: F(noise + waves) - F(noise) equals
    the closed-form spectrum of the planted waves (Dirichlet sums on the
    slab, including a wave on the -k_max boundary with k_t = 0)."""
    ng = (32, 32, 32, 8)
    g = O.Geometry(ng, (8, 32, 32, 8), (8, 0, 0, 0), (4, 4, 4), 3, 1, 1, 1)
    gd = dict(n_global=ng, n_local=g.n_local, offset=g.offset)
    noise = synth.np_normal((1, 1) + g.n_local, 81, dtype=np.float64)
    waves = np.zeros(g.n_local)
    expect = 0
    for k, ph in (((1, -2, 3, 1), 0.0), ((-4, 3, 0, 0), math.pi / 3), ((2, 0, -3, 2), -math.pi / 4)):
        waves = waves + synth.plane_wave_np(gd, k, ph, 5.0)
        expect = expect + wave_spectrum_closed_form(g, k, ph, 5.0)
    d = O.forward(noise + waves[None, None], g) - O.forward(noise, g)
    assert rel(d[0, 0], expect) < 1e-11


def test_point_evaluators_match_pinned_full_transforms():
    """The per-coefficient / per-point evaluators used for very large shards
    agree with the full transforms pinned above (FFT, irfftn, adjoint)."""
    g = geo("pencil")
    x = rand_shard(g, 91)
    X = O.forward(x, g)
    modes = [(0, 1, 2, 0), (5, 3, 0, 2), (2, 0, 3, 1)]
    got = O.forward_at_modes(x[1, 0], g, modes)
    assert np.allclose(got, [X[1, 0][m] for m in modes], rtol=1e-12, atol=1e-12)
    Y = synth.np_complex_normal((g.batch, g.c_out) + g.K, 92).astype(np.complex128)
    pts = [(0, 0, 0, 0), (3, 4, 7, 5), (1, 2, 5, 7)]
    y = O.inverse(Y, g)
    assert np.allclose(O.inverse_at_points(Y[1, 2], g, pts), [y[1, 2][p] for p in pts], rtol=1e-12, atol=1e-14)
    ga = O.forward_adj(Y, g)
    assert np.allclose(O.forward_adj_at_points(Y[0, 1], g, pts), [ga[0, 1][p] for p in pts], rtol=1e-12,
                       atol=1e-12)


# ---------------------------------------------------------------------------
# Block epilogue: GELU(W x + y) (Sec. V block structure, Algorithm 1)
# ---------------------------------------------------------------------------
def test_gelu_matches_normal_cdf_table():
    """GELU(v) = v Phi(v) at tabulated values of the normal CDF."""
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "normal_cdf.txt")) if ln.strip() and ln[0] != "#"]
    v = np.array([float(r[0]) for r in rows])
    phi = np.array([float(r[1]) for r in rows])
    assert np.allclose(O.gelu(v), v * phi, rtol=0, atol=2e-15)


def test_gelu_identities():
    """GELU(v) - GELU(-v) = v (Phi(v) + Phi(-v) = 1), GELU(0) = 0, and the
    activation is the identity / zero far out on either side."""
    v = np.linspace(-6.0, 6.0, 241)
    assert np.allclose(O.gelu(v) - O.gelu(-v), v, rtol=0, atol=1e-15)
    assert O.gelu(np.array([0.0]))[0] == 0.0
    assert abs(O.gelu(np.array([12.0]))[0] - 12.0) < 1e-15
    assert abs(O.gelu(np.array([-12.0]))[0]) < 1e-15


def test_block_epilogue_special_cases_and_brute_force():
    """W = I and y = 0 give GELU(x); W = 0 gives GELU(y); a random case
    equals the per-point, per-channel loop written out."""
    rng = np.random.default_rng(31)
    B, ci, co, shape = 2, 3, 4, (2, 3, 2, 5)
    x = rng.standard_normal((B, ci) + shape)
    y = rng.standard_normal((B, co) + shape)
    w = rng.standard_normal((co, ci))
    eye = np.eye(ci)
    assert np.allclose(O.block_epilogue(x, eye, np.zeros_like(x)), O.gelu(x), rtol=0, atol=1e-15)
    assert np.allclose(O.block_epilogue(x, np.zeros((co, ci)), y), O.gelu(y), rtol=0, atol=1e-15)
    got = O.block_epilogue(x, w, y)
    ref = np.empty_like(y)
    for b in range(B):
        for o in range(co):
            for n in np.ndindex(*shape):
                s = y[(b, o) + n]
                for i in range(ci):
                    s += w[o, i] * x[(b, i) + n]
                ref[(b, o) + n] = 0.5 * s * (1.0 + math.erf(s / math.sqrt(2.0)))
    assert np.allclose(got, ref, rtol=0, atol=1e-14)


def test_pointwise_brute_force_and_special_cases():
    """The point-wise layer equals the per-point loop written out; with the
    identity matrix and no bias it returns x, and with act it returns GELU."""
    rng = np.random.default_rng(41)
    B, ci, co, shape = 2, 3, 2, (2, 3, 2, 4)
    x = rng.standard_normal((B, ci) + shape)
    w = rng.standard_normal((co, ci))
    b = rng.standard_normal(co)
    got = O.pointwise(x, w, b)
    ref = np.empty((B, co) + shape)
    for bb in range(B):
        for o in range(co):
            for n in np.ndindex(*shape):
                s = b[o]
                for i in range(ci):
                    s += w[o, i] * x[(bb, i) + n]
                ref[(bb, o) + n] = s
    assert np.allclose(got, ref, rtol=0, atol=1e-14)
    assert np.allclose(O.pointwise(x, np.eye(ci)), x, rtol=0, atol=0)
    g = O.pointwise(x, np.eye(ci), act=True)
    assert np.allclose(g, [[[[[[0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in r3] for r3 in r2] for r2 in r1]
                             for r1 in c] for c in bx] for bx in x], rtol=0, atol=1e-15)


def _fno_fft(x, g, lift, blocks, proj):
    """The FNO forward written with numpy's FFT: rfftn, gather of the
    retained modes, per-mode channel mix, scatter into the zero spectrum,
    irfftn; bypass and GELU (math.erf) per point; lift and projection as
    matrix products over the channel axis."""
    erf = np.vectorize(math.erf)
    act = lambda v: 0.5 * v * (1.0 + erf(v / math.sqrt(2.0)))
    chan = lambda w, v: np.einsum("oi,bi...->bo...", w, v)
    v = chan(lift[0], x) + lift[1][None, :, None, None, None, None]
    for r, wb in blocks:
        F = _fft_forward(v, g)                                   # (B, C, Kx, Ky, Kz, Kt)
        B, C = F.shape[:2]
        Fm = F.reshape(B, C, -1)                                  # m = flattened mode index
        Y = np.einsum("bim,mio->bom", Fm, r).reshape((B, r.shape[2]) + g.K)
        v = act(chan(wb, v) + _fft_inverse(Y, g))
    return chan(proj[0], v) + proj[1][None, :, None, None, None, None]


@pytest.mark.parametrize("n_global,kmax,kt", [((8, 6, 4, 6), (2, 2, 1), 3), ((6, 5, 8, 8), (3, 2, 3), 5)])
def test_fno_forward_matches_fft_formulation(n_global, kmax, kt):
    """The oracle's FNO forward (direct partial DFTs) equals the same network
    evaluated through numpy's FFT, four Fourier layers deep; with no Fourier
    layer it is the projection of the lift."""
    rng = np.random.default_rng(43)
    dv, cin, cout, B = 3, 2, 2, 2
    g = O.Geometry(n_global, n_global, (0, 0, 0, 0), kmax, kt, B, dv, dv)
    M = O.n_modes(g)
    x = rng.standard_normal((B, cin) + tuple(n_global))
    lift = (rng.standard_normal((dv, cin)), rng.standard_normal(dv))
    proj = (rng.standard_normal((cout, dv)), rng.standard_normal(cout))
    blocks = [((rng.standard_normal((M, dv, dv)) + 1j * rng.standard_normal((M, dv, dv))) / dv,
               rng.standard_normal((dv, dv)) / math.sqrt(dv)) for _ in range(4)]
    got = O.fno_forward(x, g, lift, blocks, proj)
    ref = _fno_fft(x, g, lift, blocks, proj)
    assert got.shape == (B, cout) + tuple(n_global)
    assert rel(got, ref) < 1e-12
    direct = np.einsum("oi,bi...->bo...", proj[0] @ lift[0], x) + (proj[0] @ lift[1] + proj[1])[None, :, None, None, None, None]
    assert rel(O.fno_forward(x, g, lift, [], proj), direct) < 1e-13
