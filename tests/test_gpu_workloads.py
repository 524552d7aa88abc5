"""GPU parity at the full sizes of the five workloads, in the launch
configuration the benchmark uses, checked on outputs the fp64 oracle can
compute one at a time (whole (b, c) slices, sampled modes, sampled points)
and on properties that hold at any size (planted plane waves, shard sums).

Every stage gets its own seeded synthetic input; no oracle input comes from
the GPU.  Sizes: shard 64x256x256x32 with B2 C32 is 34.4 GB per spatial
tensor, so these tests need most of the device's 288 GB.
"""

import math

import numpy as np
import pytest

import oracle as O
import synth
from gpu_common import check, np_of, say, torch_gpu

pytestmark = pytest.mark.gpu


def geo_of(g):
    return O.Geometry(g["n_global"], g["n_local"], g["offset"], g["kmax"], g["kt"], g["batch"], g["c_in"],
                      g["c_out"])


def free(torch):
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def sampled_modes(M, n, seed):
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(M, size=min(n, M), replace=False))


def sampled_points(nl, n, seed):
    rng = np.random.default_rng(seed)
    pts = [tuple(int(rng.integers(0, nl[d])) for d in range(4)) for _ in range(n)]
    # always include both corners of the shard
    return pts + [(0, 0, 0, 0), tuple(v - 1 for v in nl)]


def _mix_sampled(torch, D, plan, g, cfg, M, name):
    """mix (op 0 and 1) and wgrad on the full mode range, checked on sampled modes."""
    B, ci, co = g["batch"], g["c_in"], g["c_out"]
    X = synth.torch_complex_normal((B, ci) + plan.K, synth.seed_of(cfg, "spectrum"), "cuda",
                                   var=float(np.prod(g["n_local"])))
    GY = synth.torch_complex_normal((B, co) + plan.K, synth.seed_of(cfg, "spectrum") + 10, "cuda",
                                    var=float(np.prod(g["n_local"])))
    W = synth.torch_weights(M, ci, co, synth.seed_of(cfg, "weights"), "cuda")
    idx = sampled_modes(M, 768, 5 + cfg)
    tidx = torch.from_numpy(idx).cuda()
    Wn = np_of(W.index_select(0, tidx))
    Xn = np_of(X.reshape(B, ci, M).index_select(2, tidx))
    GYn = np_of(GY.reshape(B, co, M).index_select(2, tidx))

    Y = torch.empty((B, co) + plan.K, dtype=torch.complex64, device="cuda")
    plan.mix(X, W, Y, 0, M, op=0)
    got = np_of(Y.reshape(B, co, M).index_select(2, tidx))
    ref = np.einsum("bim,mio->bom", Xn.astype(np.complex128), Wn.astype(np.complex128))
    check(got, ref, f"{name} mix (sampled modes)")
    del Y

    GX = torch.empty((B, ci) + plan.K, dtype=torch.complex64, device="cuda")
    plan.mix(GY, W, GX, 0, M, op=1)
    got = np_of(GX.reshape(B, ci, M).index_select(2, tidx))
    ref = np.einsum("bom,mio->bim", GYn.astype(np.complex128), np.conj(Wn.astype(np.complex128)))
    check(got, ref, f"{name} mix data grad (sampled modes)")
    del GX

    GW = torch.empty_like(W)
    del W
    plan.wgrad(X, GY, GW, 0, M)
    got = np_of(GW.index_select(0, tidx))
    ref = np.einsum("bim,bom->mio", np.conj(Xn.astype(np.complex128)), GYn.astype(np.complex128))
    check(got, ref, f"{name} wgrad (sampled modes)")
    del GW, X, GY
    free(torch)


@pytest.mark.parametrize("cfg", [3, 4])
def test_layer_full_size(cfg):
    """Forward on whole sampled (b, c) slices, mix / wgrad on sampled modes,
    inverse and forward_adj on sampled points and on one whole slice each."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = synth.geometry(cfg)
    go = geo_of(g)
    say(f"[workload {cfg}] {synth.WORKLOADS[cfg]['name']}")
    plan = D.Plan(g)
    M = plan.n_modes
    B, ci, co = g["batch"], g["c_in"], g["c_out"]

    x = synth.torch_input(cfg, g, "cuda")
    xh = torch.empty((B, ci) + plan.K, dtype=torch.complex64, device="cuda")
    plan.forward(x, xh)
    for (b, c) in ((0, 0), (B - 1, ci - 1)):
        xs = np_of(x[b:b + 1, c:c + 1])
        check(np_of(xh[b:b + 1, c:c + 1]), O.forward(xs, go), f"forward b={b} c={c}")
    del x, xh
    free(torch)

    _mix_sampled(torch, D, plan, g, cfg, M, f"workload {cfg}")

    yh = synth.torch_complex_normal((B, co) + plan.K, synth.seed_of(cfg, "spectrum") + 20, "cuda")
    y = torch.empty((B, co) + tuple(g["n_local"]), dtype=torch.float32, device="cuda")
    plan.inverse(yh, y)
    pts = sampled_points(g["n_local"], 48, 11 + cfg)
    for (b, c) in ((0, 1), (B - 1, co - 2)):
        ref = O.inverse_at_points(np_of(yh[b, c]), go, pts)
        got = np.array([y[(b, c) + p].item() for p in pts])
        check(got, ref, f"inverse b={b} c={c} (sampled points)")
    # one whole (b, c) slice of the shard against the oracle's inverse
    b, c = B - 1, co - 2
    check(np_of(y[b:b + 1, c:c + 1]), O.inverse(np_of(yh[b:b + 1, c:c + 1]), go),
          f"inverse b={b} c={c} (whole slice)")
    del y
    gx = torch.empty((B, ci) + tuple(g["n_local"]), dtype=torch.float32, device="cuda")
    gxh = yh if ci == co else synth.torch_complex_normal((B, ci) + plan.K, 77, "cuda")
    plan.forward_adj(gxh, gx)
    for (b, c) in ((0, 2),):
        ref = O.forward_adj_at_points(np_of(gxh[b, c]), go, pts)
        got = np.array([gx[(b, c) + p].item() for p in pts])
        check(got, ref, f"forward_adj b={b} c={c} (sampled points)")
        check(np_of(gx[b:b + 1, c:c + 1]), O.forward_adj(np_of(gxh[b:b + 1, c:c + 1]), go),
              f"forward_adj b={b} c={c} (whole slice)")
    del gx, yh, gxh
    plan.close()
    free(torch)


@pytest.mark.parametrize("cfg", [2, 6])
def test_decomposition_128cubed(cfg):
    """Workload 2 (8 x-slabs) and 6 (2x4 (x, y) pencils): the shards run one
    after another and accumulated equal the full-domain spectrum; two
    channels are checked against the oracle, and the three planted plane
    waves sit at their closed-form values."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    full = synth.full_domain(cfg)
    say(f"[workload {cfg}] {synth.WORKLOADS[cfg]['name']}")
    x = synth.torch_input(cfg, full, "cuda")
    P = synth.WORKLOADS[cfg]["shards"]
    pf = D.Plan(full)
    K = pf.K
    B, C = full["batch"], full["c_in"]
    acc = torch.empty((B, C) + K, dtype=torch.complex64, device="cuda")
    for p in range(P):
        g = synth.geometry(cfg, p)
        (x0, y0, _, _), (lx, ly, _, _) = g["offset"], g["n_local"]
        plan = D.Plan(g)
        plan.forward(x[:, :, x0:x0 + lx, y0:y0 + ly].contiguous(), acc, accumulate=p > 0)
        plan.close()
    ref_full = torch.empty_like(acc)
    pf.forward(x, ref_full)
    # Two fp32 results compared with each other: each carries its own rounding
    # (about 3e-7 relative at the planted spikes, which are ~300x the RMS),
    # so the max-abs bound is twice the oracle bar.
    check(np_of(acc), np_of(ref_full), f"sum over {P} shards vs one full-domain call", maxabs_rms=2e-4)
    go = geo_of(full)
    for c in (0, 9):
        check(np_of(acc[:, c:c + 1]), O.forward(np_of(x[:, c:c + 1]), go), f"shard sum vs oracle c={c}")
    # planted waves: 5 cos(2 pi k.n/N + phi) -> (5 prod N / 2) e^{i phi} at +k on top of
    # Gaussian noise whose coefficients have standard deviation sqrt(prod N)
    ng = full["n_global"]
    ntot = float(np.prod(ng))
    noise = math.sqrt(ntot)
    idx = [list(O.retained_indices(ng[a], full["kmax"][a])) for a in range(3)]
    A = np_of(acc)
    for k, ph in synth.CFG2_WAVES:
        pos = tuple(idx[a].index(k[a] % ng[a]) for a in range(3)) + (k[3],)
        want = synth.CFG2_AMPLITUDE * ntot / 2 * complex(math.cos(ph), math.sin(ph))
        for c in range(C):
            err = abs(A[(0, c) + pos] - want)
            assert err < 8 * noise, (k, c, err, noise)
    say(f"  planted waves: |spike| = {abs(want):.4e}, noise sigma = {noise:.1f}")
    del x, acc, ref_full
    free(torch)
    # every shard's inverse of one spectrum is its block of the full-domain
    # inverse; one shard is also checked against the oracle on sampled points
    yh = synth.torch_complex_normal((B, C) + K, synth.seed_of(cfg, "spectrum") + 50, "cuda")
    y_full = torch.empty((B, C) + tuple(full["n_global"]), dtype=torch.float32, device="cuda")
    pf.inverse(yh, y_full)
    for p in range(P):
        g = synth.geometry(cfg, p)
        (x0, y0, _, _), (lx, ly, _, _) = g["offset"], g["n_local"]
        plan = D.Plan(g)
        y = torch.empty((B, C) + tuple(g["n_local"]), dtype=torch.float32, device="cuda")
        plan.inverse(yh, y)
        check(np_of(y), np_of(y_full[:, :, x0:x0 + lx, y0:y0 + ly]), f"shard {p} inverse vs full-domain block")
        if p == P - 1:
            pts = sampled_points(g["n_local"], 32, 29)
            ref = O.inverse_at_points(np_of(yh[0, 5]), geo_of(g), pts)
            check(np.array([y[(0, 5) + q].item() for q in pts]), ref, f"shard {p} inverse vs oracle (points)")
            check(np_of(y[:, 5:6]), O.inverse(np_of(yh[:, 5:6]), geo_of(g)),
                  f"shard {p} inverse vs oracle (whole channel)")
        plan.close()
        del y
    pf.close()
    del yh, y_full
    free(torch)


def test_backward_full_size():
    """Workload 5 (modes 64/64/64/16 on the 64x256x256x32 shard): the
    inverse adjoint on whole sampled slices, the mix data gradient and the
    weight gradient (34.4 GB each) on sampled modes, forward_adj on points
    and on a whole slice, and the inverse at these modes on a whole slice."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    cfg = 5
    g = synth.geometry(cfg)
    go = geo_of(g)
    say(f"[workload 5] {synth.WORKLOADS[cfg]['name']}")
    plan = D.Plan(g)
    M = plan.n_modes
    B, ci, co = g["batch"], g["c_in"], g["c_out"]
    gy = synth.torch_normal((B, co) + tuple(g["n_local"]), synth.seed_of(cfg, "upstream"), "cuda")
    gyh = torch.empty((B, co) + plan.K, dtype=torch.complex64, device="cuda")
    plan.inverse_adj(gy, gyh)
    for (b, c) in ((0, 3), (B - 1, co - 1)):
        check(np_of(gyh[b:b + 1, c:c + 1]), O.inverse_adj(np_of(gy[b:b + 1, c:c + 1]), go),
              f"inverse_adj b={b} c={c}")
    del gy, gyh
    free(torch)

    _mix_sampled(torch, D, plan, g, cfg, M, "workload 5")

    gxh = synth.torch_complex_normal((B, ci) + plan.K, synth.seed_of(cfg, "spectrum") + 30, "cuda")
    gx = torch.empty((B, ci) + tuple(g["n_local"]), dtype=torch.float32, device="cuda")
    plan.forward_adj(gxh, gx)
    pts = sampled_points(g["n_local"], 32, 17)
    ref = O.forward_adj_at_points(np_of(gxh[1, 7]), go, pts)
    got = np.array([gx[(1, 7) + p].item() for p in pts])
    check(got, ref, "forward_adj b=1 c=7 (sampled points)")
    # whole (b, c) slices of forward_adj and of the inverse at these modes against the oracle
    check(np_of(gx[1:2, 7:8]), O.forward_adj(np_of(gxh[1:2, 7:8]), go), "forward_adj b=1 c=7 (whole slice)")
    plan.inverse(gxh, gx)
    check(np_of(gx[0:1, 30:31]), O.inverse(np_of(gxh[0:1, 30:31]), go), "inverse b=0 c=30 (whole slice)")
    del gxh, gx
    plan.close()
    free(torch)


def test_block_epilogue_full_size():
    """Block epilogue GELU(W x + y) on one 16x128x128x32 slab of workload 2
    (B1, C16, the launch the block benchmark times), checked on sampled
    points; the spectral output y is a seeded stand-in."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    cfg = 2
    g = synth.geometry(cfg, 3)
    say(f"[workload 2 block epilogue] slab 3, n_local={g['n_local']}")
    plan = D.Plan(g)
    B, ci, co = g["batch"], g["c_in"], g["c_out"]
    x = synth.torch_input(cfg, g, "cuda")
    y = synth.torch_normal((B, co) + tuple(g["n_local"]), synth.seed_of(cfg, "spectrum") + 40, "cuda")
    wb = synth.torch_bypass(co, ci, synth.seed_of(cfg, "bypass"), "cuda")
    pts = sampled_points(g["n_local"], 4096, 23)
    idx = torch.tensor([list(p) for p in pts], device="cuda").T
    xs = np_of(x[:, :, idx[0], idx[1], idx[2], idx[3]])
    ys = np_of(y[:, :, idx[0], idx[1], idx[2], idx[3]])
    plan.block_epilogue(x, wb, y)
    got = np_of(y[:, :, idx[0], idx[1], idx[2], idx[3]])
    check(got, O.block_epilogue(xs, np_of(wb), ys), "block epilogue (sampled points)")
    del x, y
    plan.close()
    free(torch)
