"""GPU parity of every C-ABI call against the fp64 oracle, element by element,
on the same fp32 inputs, at sizes the oracle handles in seconds.  The cases
cover several MFMA tiles plus ragged tails in every dimension, odd extents,
the folded and unfolded z paths, both k_t column layouts, shards with
offsets (slab, pencil, t-shard), retained counts above the local extent,
full retention, and empty calls."""

import numpy as np
import pytest

import oracle as O
from gpu_common import (Guarded, check, desc_of, dev, geometry, np_of, rand_cplx, rand_real, say,
                        torch_gpu)

pytestmark = pytest.mark.gpu

# name: (n_global, n_local, offset, kmax, kt, B, C_in, C_out)
CASES = {
    "tiny_baseline": ((12, 10, 8, 8), (12, 10, 8, 8), (0, 0, 0, 0), (3, 2, 2), 3, 1, 2, 2),
    "tiny_slab": ((12, 10, 8, 8), (4, 10, 8, 8), (4, 0, 0, 0), (3, 2, 2), 3, 1, 2, 2),
    "tiny_pencil": ((12, 10, 8, 8), (4, 5, 8, 8), (8, 5, 0, 0), (3, 2, 2), 3, 2, 1, 3),
    "odd_extents": ((9, 7, 5, 6), (9, 7, 5, 6), (0, 0, 0, 0), (2, 3, 1), 3, 1, 1, 1),
    "odd_shard": ((9, 7, 5, 6), (3, 7, 5, 6), (6, 0, 0, 0), (2, 3, 1), 4, 1, 1, 1),
    "nyquist_t": ((6, 6, 4, 6), (6, 6, 4, 6), (0, 0, 0, 0), (2, 2, 1), 4, 1, 1, 1),
    "k_above_nloc": ((12, 6, 4, 4), (2, 6, 4, 4), (6, 0, 0, 0), (3, 1, 1), 2, 1, 1, 1),
    "all_modes": ((6, 4, 4, 6), (6, 4, 4, 6), (0, 0, 0, 0), (3, 2, 2), 4, 1, 1, 1),
    "t_shard_odd": ((8, 6, 4, 10), (8, 6, 4, 5), (0, 0, 0, 5), (2, 2, 1), 4, 1, 2, 1),
    "fold_ragged": ((24, 40, 48, 32), (24, 40, 48, 32), (0, 0, 0, 0), (5, 9, 11), 7, 2, 3, 5),
    "slab_like_cfg2": ((64, 64, 64, 32), (16, 64, 64, 32), (32, 0, 0, 0), (16, 16, 16), 8, 1, 3, 2),
    "z_shard_unfolded": ((16, 20, 64, 16), (16, 20, 30, 16), (0, 0, 17, 0), (4, 5, 9), 5, 1, 2, 2),
    "kt16_two_col_tiles": ((16, 16, 32, 32), (16, 16, 32, 32), (0, 0, 0, 0), (4, 4, 8), 16, 1, 2, 2),
    "kz64_unfolded_odd_nz": ((8, 8, 129, 8), (8, 8, 129, 8), (0, 0, 0, 0), (2, 2, 32), 5, 1, 1, 2),
    "nt64_kt12": ((8, 12, 20, 64), (8, 12, 20, 64), (0, 0, 0, 0), (2, 3, 5), 12, 1, 2, 1),
    "nt21_pdebench_like": ((16, 16, 16, 21), (16, 16, 16, 21), (0, 0, 0, 0), (4, 4, 4), 8, 1, 2, 2),
    "cfg1_full": ((32, 32, 32, 8), (32, 32, 32, 8), (0, 0, 0, 0), (8, 8, 8), 4, 1, 8, 8),
    # largest tiles the stream kernels take: 64 folded z modes per class, k_t = 16, N_t = 64
    "max_tiles": ((4, 4, 128, 64), (4, 4, 128, 64), (0, 0, 0, 0), (2, 2, 64), 16, 1, 2, 2),
    # four-class z fold (N_z % 4 == 0, even k_max(z), k_t > 8): ragged z tile with masked
    # 16-byte t chunks, scalar t (N_t = 21), complete tiles with every z mode kept
    "radix4_ragged": ((6, 8, 40, 24), (6, 8, 40, 24), (0, 0, 0, 0), (2, 3, 6), 10, 2, 2, 3),
    "radix4_scalar_t": ((4, 6, 24, 21), (4, 6, 24, 21), (0, 0, 0, 0), (1, 2, 4), 11, 1, 1, 2),
    "radix4_full_tiles": ((4, 4, 64, 32), (4, 4, 64, 32), (0, 0, 0, 0), (2, 2, 32), 16, 1, 2, 2),
    # (with at most 16 z modes every class count pads to one tile, so the kernels take one class;
    # 17-64 modes keep four): ragged quarter N_z / 4 = 22 with masked 16-byte t, and scalar t
    "radix4_kz40_ragged": ((4, 6, 88, 24), (4, 6, 88, 24), (0, 0, 0, 0), (1, 2, 20), 10, 1, 2, 2),
    "radix4_kz36_scalar_t": ((4, 4, 72, 21), (4, 4, 72, 21), (0, 0, 0, 0), (1, 1, 18), 11, 1, 1, 2),
    # odd k_max(z) with N_z % 4 == 0 and k_t > 8 keeps the two-class fold
    "fold2_odd_kz_kt9": ((4, 4, 24, 16), (4, 4, 24, 16), (0, 0, 0, 0), (1, 1, 5), 9, 1, 2, 1),
    # t fold (k_t > 8, whole N_t = 32): two z classes with a ragged z tile and an odd k_t count,
    # 64 slots of unfolded sharded z, 32 slots per class in an x slab; with N_t = 32 of a
    # sharded t the unfolded two-tile kernels run instead
    "tfold_two_class_ragged": ((6, 8, 36, 32), (6, 8, 36, 32), (0, 0, 0, 0), (2, 3, 9), 13, 1, 2, 3),
    "tfold_z_shard_mt8": ((4, 6, 96, 32), (4, 6, 40, 32), (0, 0, 24, 0), (1, 2, 20), 16, 1, 1, 2),
    "tfold_mt4_slab": ((8, 6, 90, 32), (4, 6, 90, 32), (4, 0, 0, 0), (2, 2, 20), 16, 2, 1, 1),
    "t_shard_nt32_kt16": ((4, 4, 16, 64), (4, 4, 16, 32), (0, 0, 0, 32), (1, 2, 4), 16, 1, 2, 2),
    # four-class x and y folds of the separate axis launches (whole N % 4 == 0, K % 64 == 0):
    # x and y both folded (x forward accumulating into the spectrum), then a ragged quarter
    # (N_y / 4 = 50) with two k tiles per class and two K steps of the inverse class sums
    "axis_four_class": ((64, 128, 8, 8), (64, 128, 8, 8), (0, 0, 0, 0), (32, 32, 2), 3, 1, 2, 2),
    "axis_four_class_ragged": ((8, 200, 8, 8), (4, 200, 8, 8), (4, 0, 0, 0), (2, 64, 2), 3, 2, 1, 2),
    # more (b, c, x) planes than the fused t+z+y kernel has resident workgroups
    "many_planes": ((48, 8, 16, 8), (48, 8, 16, 8), (0, 0, 0, 0), (4, 2, 4), 3, 2, 4, 3),
    # N_y = N_z = 512: the fused kernels' y basis images do not fit next to the z image and the
    # row exchange in LDS and are read from global memory
    "y_image_global": ((2, 512, 512, 8), (2, 512, 512, 8), (0, 0, 0, 0), (1, 16, 16), 4, 1, 1, 1),
}

# Geometries whose plan takes the fused t + z + y forward kernel (K_t <= 8, at
# most 16 z modes per class, N_t <= 32 and a multiple of 4, K_y <= 32,
# K_z K_t <= 256): folded y with a ragged last slot group, unfolded y (pencil),
# K above the local extent, several slot groups, many planes, y basis images
# read from global memory.
FUSED_CASES = ["tiny_baseline", "tiny_slab", "tiny_pencil", "k_above_nloc", "fold_ragged", "slab_like_cfg2",
               "cfg1_full", "many_planes", "y_image_global"]


def _setup(name, split=False):
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry(*CASES[name])
    g.validate()
    say(f"[case {name}] n_global={g.n_global} n_local={g.n_local} offset={g.offset} "
        f"kmax={g.kmax} kt={g.kt} B={g.batch} Cin={g.c_in} Cout={g.c_out} split={split}")
    plan = D.Plan(desc_of(g), flags=D.PLAN_SPLIT_SCHEDULE if split else 0)
    return torch, D, g, plan


@pytest.mark.parametrize("name", list(CASES))
def test_forward_and_accumulate(name):
    torch, D, g, plan = _setup(name)
    x = rand_real((g.batch, g.c_in) + g.n_local, 101)
    ref = O.forward(x, g)
    out = Guarded(torch, plan.spectral_shape(g.c_in), torch.complex64)
    plan.forward(dev(torch, x), out.t)
    torch.cuda.synchronize()
    check(np_of(out.t), ref, "forward")
    assert out.guards_intact()
    plan.forward(dev(torch, x), out.t, accumulate=True)
    torch.cuda.synchronize()
    check(np_of(out.t), 2 * ref, "forward accumulate")
    assert out.guards_intact()


@pytest.mark.parametrize("name", list(CASES))
def test_inverse(name):
    torch, D, g, plan = _setup(name)
    yh = rand_cplx((g.batch, g.c_out) + g.K, 102)
    ref = O.inverse(yh, g)
    out = Guarded(torch, plan.spatial_shape(g.c_out), torch.float32)
    plan.inverse(dev(torch, yh), out.t)
    torch.cuda.synchronize()
    check(np_of(out.t), ref, "inverse")
    assert out.guards_intact()


@pytest.mark.parametrize("name", list(CASES))
def test_adjoints(name):
    torch, D, g, plan = _setup(name)
    G = rand_cplx((g.batch, g.c_in) + g.K, 103)
    out = Guarded(torch, plan.spatial_shape(g.c_in), torch.float32)
    plan.forward_adj(dev(torch, G), out.t)
    torch.cuda.synchronize()
    check(np_of(out.t), O.forward_adj(G, g), "forward_adj")
    assert out.guards_intact()
    gy = rand_real((g.batch, g.c_out) + g.n_local, 104)
    ref = O.inverse_adj(gy, g)
    out2 = Guarded(torch, plan.spectral_shape(g.c_out), torch.complex64)
    plan.inverse_adj(dev(torch, gy), out2.t)
    torch.cuda.synchronize()
    check(np_of(out2.t), ref, "inverse_adj")
    plan.inverse_adj(dev(torch, gy), out2.t, accumulate=True)
    torch.cuda.synchronize()
    check(np_of(out2.t), 2 * ref, "inverse_adj accumulate")
    assert out2.guards_intact()


@pytest.mark.parametrize("name", ["tiny_pencil", "fold_ragged", "cfg1_full", "kt16_two_col_tiles"])
def test_mix_ranges_and_wgrad(name):
    torch, D, g, plan = _setup(name)
    M = plan.n_modes
    X = rand_cplx((g.batch, g.c_in) + g.K, 105)
    W = rand_cplx((M, g.c_in, g.c_out), 106, var=1.0 / (g.c_in * g.c_out))
    Xd, Wd = dev(torch, X), dev(torch, W)
    # full range
    Y = Guarded(torch, plan.spectral_shape(g.c_out), torch.complex64)
    plan.mix(Xd, Wd, Y.t, 0, M, op=0)
    torch.cuda.synchronize()
    check(np_of(Y.t).reshape(g.batch, g.c_out, M), O.mix(X, W, 0, M), "mix full")
    assert Y.guards_intact()
    # a middle range leaves every other column untouched
    m0, m1 = M // 3, (2 * M) // 3 + 1
    sentinel = rand_cplx((g.batch, g.c_out) + g.K, 107)
    Y2 = Guarded(torch, plan.spectral_shape(g.c_out), torch.complex64, fill=dev(torch, sentinel))
    plan.mix(Xd, Wd[m0:m1].contiguous(), Y2.t, m0, m1, op=0)
    torch.cuda.synchronize()
    ref = O.mix(X, W[m0:m1], m0, m1, yhat_in=sentinel)
    got = np_of(Y2.t).reshape(g.batch, g.c_out, M)
    check(got[:, :, m0:m1], ref[:, :, m0:m1], "mix range")
    assert np.array_equal(got[:, :, :m0], sentinel.reshape(g.batch, g.c_out, M)[:, :, :m0])
    assert np.array_equal(got[:, :, m1:], sentinel.reshape(g.batch, g.c_out, M)[:, :, m1:])
    assert Y2.guards_intact()
    # ranges run one after another assemble the full mix (replaces the AllGather)
    Y3 = torch.zeros(plan.spectral_shape(g.c_out), dtype=torch.complex64, device="cuda")
    bounds = np.linspace(0, M, 5).astype(int)
    for a, b in zip(bounds[:-1], bounds[1:]):
        plan.mix(Xd, Wd[a:b].contiguous(), Y3, int(a), int(b), op=0)
    torch.cuda.synchronize()
    check(np_of(Y3).reshape(g.batch, g.c_out, M), O.mix(X, W, 0, M), "mix pieced")
    # data gradient (op = 1)
    GY = rand_cplx((g.batch, g.c_out) + g.K, 108)
    GX = Guarded(torch, plan.spectral_shape(g.c_in), torch.complex64)
    plan.mix(dev(torch, GY), Wd, GX.t, 0, M, op=1)
    torch.cuda.synchronize()
    check(np_of(GX.t).reshape(g.batch, g.c_in, M), O.mix_data_grad(GY, W, 0, M), "mix data grad")
    assert GX.guards_intact()
    # weight gradient on a range, with accumulate
    GW = Guarded(torch, (m1 - m0, g.c_in, g.c_out), torch.complex64)
    plan.wgrad(Xd, dev(torch, GY), GW.t, m0, m1)
    torch.cuda.synchronize()
    refw = O.mix_wgrad(X, GY, m0, m1)
    check(np_of(GW.t), refw, "wgrad")
    plan.wgrad(Xd, dev(torch, GY), GW.t, m0, m1, accumulate=True)
    torch.cuda.synchronize()
    check(np_of(GW.t), 2 * refw, "wgrad accumulate")
    assert GW.guards_intact()


# (B, C_in, C_out): row groups of 1..64 lanes, one to eight columns per lane
# (C_out = 512 is the largest the mix kernels take), batch chunks beyond the
# register chunk, w row chunks beyond 16, odd counts.
MIX_SHAPES = [(2, 32, 32), (1, 16, 16), (3, 5, 64), (2, 7, 65), (1, 40, 130), (5, 2, 3), (1, 1, 1),
              (1, 3, 512)]


@pytest.mark.parametrize("shape", MIX_SHAPES, ids=lambda s: "B%d_ci%d_co%d" % s)
def test_mix_channel_shapes(shape):
    """mix, its data gradient and the weight gradient (with accumulate) on
    channel and batch counts that exercise every lane layout of the mix
    kernels, over the full mode set and a ragged middle range."""
    B, ci, co = shape
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry((8, 8, 6, 8), (8, 8, 6, 8), (0, 0, 0, 0), (2, 3, 2), 3, B, ci, co)
    say(f"[mix shape] B={B} Cin={ci} Cout={co}")
    plan = D.Plan(desc_of(g))
    M = plan.n_modes
    X = rand_cplx((B, ci) + g.K, 120)
    GY = rand_cplx((B, co) + g.K, 121)
    W = rand_cplx((M, ci, co), 122, var=1.0 / (ci * co))
    Xd, GYd, Wd = dev(torch, X), dev(torch, GY), dev(torch, W)
    for m0, m1 in ((0, M), (M // 3 + 1, M - 5)):
        Wr = Wd[m0:m1].clone()  # its own (aligned) allocation
        sentinel = rand_cplx((B, co) + g.K, 123)
        Y = Guarded(torch, plan.spectral_shape(co), torch.complex64, fill=dev(torch, sentinel))
        plan.mix(Xd, Wr, Y.t, m0, m1, op=0)
        gx_sent = rand_cplx((B, ci) + g.K, 124)
        GX = Guarded(torch, plan.spectral_shape(ci), torch.complex64, fill=dev(torch, gx_sent))
        plan.mix(GYd, Wr, GX.t, m0, m1, op=1)
        GW = Guarded(torch, (m1 - m0, ci, co), torch.complex64)
        plan.wgrad(Xd, GYd, GW.t, m0, m1)
        torch.cuda.synchronize()
        y_ref = O.mix(X, W[m0:m1], m0, m1, yhat_in=sentinel)
        check(np_of(Y.t).reshape(B, co, M), y_ref, f"mix [{m0},{m1})")
        gx_ref = O.mix_data_grad(GY, W[m0:m1], m0, m1, gx_in=gx_sent)
        check(np_of(GX.t).reshape(B, ci, M), gx_ref, f"mix data grad [{m0},{m1})")
        gw_ref = O.mix_wgrad(X, GY, m0, m1)
        check(np_of(GW.t), gw_ref, f"wgrad [{m0},{m1})")
        plan.wgrad(Xd, GYd, GW.t, m0, m1, accumulate=True)
        torch.cuda.synchronize()
        check(np_of(GW.t), 2 * gw_ref, f"wgrad accumulate [{m0},{m1})")
        for t in (Y, GX, GW):
            assert t.guards_intact()
    plan.close()


def test_slab_sum_equals_full_domain():
    """Eq. (dtst_reduce) on one GPU: per-slab forwards accumulated into one
    output equal the full-domain coefficients (and the oracle)."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    ng, k, kt, B, C = (32, 24, 16, 8), (6, 5, 4), 5, 1, 3
    x = rand_real((B, C) + ng, 109)
    full = geometry(ng, ng, (0, 0, 0, 0), k, kt, B, C, C)
    ref = O.forward(x, full)
    acc = torch.zeros((B, C) + full.K, dtype=torch.complex64, device="cuda")
    for p in range(4):
        g = geometry(ng, (8,) + ng[1:], (8 * p, 0, 0, 0), k, kt, B, C, C)
        plan = D.Plan(desc_of(g))
        plan.forward(dev(torch, x[:, :, 8 * p:8 * p + 8]), acc, accumulate=(p > 0))
    torch.cuda.synchronize()
    check(np_of(acc), ref, "sum over x-slabs")
    # pencil split over x and y, accumulated
    acc2 = torch.zeros_like(acc)
    first = True
    for px in range(2):
        for py in range(2):
            g = geometry(ng, (16, 12, 16, 8), (16 * px, 12 * py, 0, 0), k, kt, B, C, C)
            plan = D.Plan(desc_of(g))
            plan.forward(dev(torch, x[:, :, 16 * px:16 * px + 16, 12 * py:12 * py + 12]), acc2, accumulate=not first)
            first = False
    torch.cuda.synchronize()
    check(np_of(acc2), ref, "sum over pencils")


def test_gpu_adjoint_dot_products():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry(*CASES["fold_ragged"])
    plan = D.Plan(desc_of(g))
    x = dev(torch, rand_real((g.batch, g.c_in) + g.n_local, 110)).double()
    G = dev(torch, rand_cplx((g.batch, g.c_in) + g.K, 111))
    Fx = torch.empty(plan.spectral_shape(g.c_in), dtype=torch.complex64, device="cuda")
    plan.forward(x.float(), Fx)
    FtG = torch.empty(plan.spatial_shape(g.c_in), dtype=torch.float32, device="cuda")
    plan.forward_adj(G, FtG)
    lhs = torch.real(torch.vdot(G.flatten().to(torch.complex128), Fx.flatten().to(torch.complex128))).item()
    rhs = torch.dot(FtG.double().flatten(), x.flatten()).item()
    assert abs(lhs - rhs) <= 1e-5 * abs(lhs)


def test_empty_batch_and_empty_range_are_noops():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry((8, 8, 8, 8), (8, 8, 8, 8), (0, 0, 0, 0), (2, 2, 2), 3, 0, 2, 2)
    plan = D.Plan(desc_of(g))
    assert plan.ws_bytes == 0
    x = torch.empty((0, 2, 8, 8, 8, 8), dtype=torch.float32, device="cuda")
    xh = torch.empty((0, 2) + g.K, dtype=torch.complex64, device="cuda")
    plan.forward(x, xh)
    plan.inverse(xh, x)
    g1 = geometry((8, 8, 8, 8), (8, 8, 8, 8), (0, 0, 0, 0), (2, 2, 2), 3, 1, 2, 2)
    plan1 = D.Plan(desc_of(g1))
    X = torch.ones((1, 2) + g1.K, dtype=torch.complex64, device="cuda")
    Y = torch.full((1, 2) + g1.K, 3.0, dtype=torch.complex64, device="cuda")
    W = torch.empty((0, 2, 2), dtype=torch.complex64, device="cuda")
    D.dtst_mix(plan1.handle, X, W, Y, 5, 5, 0)
    torch.cuda.synchronize()
    assert bool((Y == 3.0).all().item())


def test_errors_launch_nothing():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry(*CASES["tiny_slab"])
    plan = D.Plan(desc_of(g))
    x = dev(torch, rand_real((g.batch, g.c_in) + g.n_local, 112))
    out = torch.full(plan.spectral_shape(g.c_in), 5.0, dtype=torch.complex64, device="cuda")
    small_ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(D.DtstError) as e:
        D.dtst_forward(plan.handle, x, out, 0, small_ws)
    assert e.value.status == 1 and "workspace" in str(e.value)
    with pytest.raises(D.DtstError):
        D.dtst_mix(plan.handle, out, out, out, 0, plan.n_modes + 1, 0)
    with pytest.raises(D.DtstError):
        D.dtst_mix(plan.handle, out, out, out, 0, 1, 2)
    with pytest.raises(D.DtstError):
        D.dtst_forward(plan.handle, x, out, 2, plan.ws)
    mis = torch.empty(plan.spectral_shape(g.c_in)[0] * 1000 + 8, dtype=torch.uint8, device="cuda")[4:]
    with pytest.raises(D.DtstError) as e:
        D.dtst_forward(plan.handle, x, mis, 0, plan.ws)
    assert "aligned" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 5.0).all().item())
    h = plan.handle
    plan.close()
    with pytest.raises(D.DtstError) as e:
        D.dtst_forward(h, x, out, 0, small_ws)
    assert "destroyed" in str(e.value)


# (n_local, B, C_in, C_out): 16-byte path with one chunk of 16 output channels,
# chunks of 16 with a ragged last one (37), chunks of 12 (C_out = 20, the FNO's
# width d_v, and 17 with a ragged last chunk), the scalar path (point count not
# a multiple of 4) and narrow outputs, C_in != C_out.
EPILOGUE_SHAPES = [((4, 6, 8, 8), 2, 16, 16), ((3, 5, 4, 8), 1, 3, 37), ((4, 6, 8, 8), 1, 20, 20),
                   ((3, 5, 4, 8), 2, 7, 17), ((3, 5, 7, 3), 1, 20, 20), ((3, 5, 7, 3), 2, 5, 2),
                   ((2, 2, 2, 2), 1, 1, 1),
                   # one pass over the input channels for 24 < C_out <= 32
                   ((3, 5, 4, 8), 1, 32, 32), ((4, 6, 8, 8), 2, 9, 25)]


@pytest.mark.parametrize("shape", EPILOGUE_SHAPES, ids=lambda s: "nl%s_B%d_ci%d_co%d" % (
    "x".join(map(str, s[0])), s[1], s[2], s[3]))
def test_block_epilogue(shape):
    """y <- GELU(W x + y) (Algorithm 1, first and last step) against the
    oracle, element by element."""
    nl, B, ci, co = shape
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry(nl, nl, (0, 0, 0, 0), (1, 1, 1), 1, B, ci, co)
    say(f"[block epilogue] n_local={nl} B={B} Cin={ci} Cout={co}")
    plan = D.Plan(desc_of(g))
    x = rand_real((B, ci) + nl, 130)
    y = rand_real((B, co) + nl, 131)
    w = (rand_real((co, ci), 132) / np.sqrt(ci)).astype(np.float32)
    Y = Guarded(torch, plan.spatial_shape(co), torch.float32, fill=dev(torch, y))
    plan.block_epilogue(dev(torch, x), dev(torch, w), Y.t)
    torch.cuda.synchronize()
    check(np_of(Y.t), O.block_epilogue(x, w, y), "block epilogue")
    assert Y.guards_intact()
    plan.close()


def test_block_forward_small():
    """The whole block of Algorithm 1 on one shard: forward, mix, inverse, then
    the bypass and GELU, against the oracle composed from the same input."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry((16, 12, 24, 16), (16, 12, 24, 16), (0, 0, 0, 0), (4, 3, 5), 6, 2, 3, 4)
    plan = D.Plan(desc_of(g))
    M = plan.n_modes
    x = rand_real((g.batch, g.c_in) + g.n_local, 133)
    W = rand_cplx((M, g.c_in, g.c_out), 134, var=1.0 / (g.c_in * g.c_out))
    wb = (rand_real((g.c_out, g.c_in), 135) / np.sqrt(g.c_in)).astype(np.float32)
    xd = dev(torch, x)
    xh = torch.empty(plan.spectral_shape(g.c_in), dtype=torch.complex64, device="cuda")
    yh = torch.empty(plan.spectral_shape(g.c_out), dtype=torch.complex64, device="cuda")
    y = torch.empty(plan.spatial_shape(g.c_out), dtype=torch.float32, device="cuda")
    plan.forward(xd, xh)
    plan.mix(xh, dev(torch, W), yh, 0, M)
    plan.inverse(yh, y)
    plan.block_epilogue(xd, dev(torch, wb), y)
    torch.cuda.synchronize()
    spec = O.mix(O.forward(x, g), W, 0, M, c_out=g.c_out).reshape((g.batch, g.c_out) + g.K)
    ref = O.block_epilogue(x, wb, O.inverse(spec, g))
    check(np_of(y), ref, "block forward (spectral path + bypass + GELU)")
    plan.close()


def test_block_epilogue_rejects_overlap():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry((4, 4, 4, 4), (4, 4, 4, 4), (0, 0, 0, 0), (1, 1, 1), 1, 1, 2, 2)
    plan = D.Plan(desc_of(g))
    buf = torch.zeros((1, 2) + g.n_local, dtype=torch.float32, device="cuda")
    w = torch.zeros((2, 2), dtype=torch.float32, device="cuda")
    with pytest.raises(D.DtstError) as e:
        D.dtst_block_epilogue(plan.handle, buf, w, buf)
    assert e.value.status == 1
    plan.close()


# (n_global, n_local, offset, kmax, kt, B, C_in, C_out), and whether the
# fused z + t expansion and epilogue kernel covers the shape: folded and
# sharded z, many input channels, both k_t column layouts, scalar t, the
# FNO's width d_v = 20; for the fused kernel every instance form: one and two
# k_t tiles (t folded or not), one and two t tiles, 16 and 32 z slots per
# class, one and two z classes, each channel class (<= 16, <= 20, <= 32),
# ragged z tiles and t extents that are not a multiple of 16.
INVERSE_BLOCK_CASES = {
    "fold": (((8, 6, 32, 32), (8, 6, 32, 32), (0, 0, 0, 0), (2, 2, 8), 5, 2, 3, 6), True),
    "z_shard": (((8, 6, 64, 16), (8, 6, 32, 16), (0, 0, 16, 0), (2, 2, 4), 4, 1, 20, 16), True),
    "many_inputs": (((4, 4, 32, 32), (4, 4, 32, 32), (0, 0, 0, 0), (1, 1, 4), 3, 1, 64, 16), False),
    "kt12": (((4, 4, 16, 32), (4, 4, 16, 32), (0, 0, 0, 0), (1, 2, 4), 12, 1, 2, 3), True),
    "nt21": (((4, 6, 8, 21), (4, 6, 8, 21), (0, 0, 0, 0), (2, 2, 2), 6, 2, 2, 2), False),
    "dv20": (((8, 6, 32, 32), (8, 6, 32, 32), (0, 0, 0, 0), (2, 2, 8), 5, 1, 20, 20), True),
    "dv20_tfold": (((8, 8, 32, 32), (8, 8, 32, 32), (0, 0, 0, 0), (4, 4, 8), 16, 1, 20, 20), True),
    "mt4_fold": (((4, 4, 64, 16), (4, 4, 64, 16), (0, 0, 0, 0), (1, 2, 24), 3, 1, 5, 7), True),
    "mt4_z_shard": (((4, 4, 64, 16), (4, 4, 48, 16), (0, 0, 8, 0), (1, 2, 12), 3, 2, 4, 3), True),
    "ct2_th1": (((4, 6, 16, 16), (4, 6, 16, 16), (0, 0, 0, 0), (2, 2, 4), 9, 1, 3, 5), True),
    "ct2_t_shard": (((4, 4, 16, 64), (4, 4, 16, 32), (0, 0, 0, 32), (1, 1, 4), 12, 1, 6, 4), True),
    "c32": (((4, 4, 32, 16), (4, 4, 32, 16), (0, 0, 0, 0), (1, 1, 4), 3, 1, 32, 24), True),
    # more than 20 channels: two passes of 16 output channels per chunk (t folded, one z class)
    "c28_tfold": (((8, 4, 32, 32), (8, 4, 32, 32), (0, 0, 0, 0), (2, 2, 8), 16, 1, 20, 28), True),
    "c32_z_shard": (((4, 4, 64, 16), (4, 4, 32, 16), (0, 0, 16, 0), (1, 1, 4), 3, 2, 32, 32), True),
    "ragged_z": (((4, 4, 40, 8), (4, 4, 40, 8), (0, 0, 0, 0), (1, 1, 6), 2, 1, 4, 4), True),
    "nt12_ragged": (((4, 4, 24, 12), (4, 4, 24, 12), (0, 0, 0, 0), (2, 2, 5), 4, 1, 3, 2), True),
    "nt20": (((4, 6, 32, 20), (4, 6, 32, 20), (0, 0, 0, 0), (2, 2, 6), 7, 1, 5, 5), True),
    "batch3": (((4, 6, 32, 32), (2, 6, 32, 32), (2, 0, 0, 0), (2, 2, 8), 6, 3, 5, 9), True),
    # a last tile of 1 or 2 output channels (one pass of two tiles; second pass of two)
    "c17": (((4, 6, 32, 32), (4, 6, 32, 32), (0, 0, 0, 0), (2, 2, 8), 5, 1, 17, 17), True),
    "c25_18": (((4, 4, 32, 16), (4, 4, 32, 16), (0, 0, 0, 0), (1, 1, 4), 3, 1, 25, 18), True),
    # whole tiles (C_in = C_out = 16 or 32, N_t = 32) over 1024 rows: several rows per
    # workgroup, so that the unconditional passes run between the first and last steps
    "full_c16": (((16, 64, 64, 32), (16, 64, 64, 32), (0, 0, 0, 0), (2, 4, 8), 5, 1, 16, 16), True),
    "full_c32": (((16, 64, 32, 32), (16, 64, 32, 32), (0, 0, 0, 0), (2, 4, 8), 6, 1, 32, 32), True),
    "full_c20": (((16, 64, 64, 32), (16, 64, 64, 32), (0, 0, 0, 0), (2, 4, 8), 5, 1, 20, 20), True),
    "full_c20_tfold": (((16, 64, 32, 32), (16, 64, 32, 32), (0, 0, 0, 0), (4, 4, 8), 16, 1, 20, 20), True),
    # 992 rows: workgroups own 3 or 4 rows, so their counts of unconditional passes differ
    "full_c16_ragged_rows": (((16, 62, 64, 32), (16, 62, 64, 32), (0, 0, 0, 0), (2, 4, 8), 5, 1, 16, 16), True),
    "full_c20_tfold_ragged_rows": (((16, 62, 32, 32), (16, 62, 32, 32), (0, 0, 0, 0), (4, 4, 8), 16, 1, 20, 20), True),
}


@pytest.mark.parametrize("unfused", [False, True], ids=["default", "unfused"])
@pytest.mark.parametrize("name", list(INVERSE_BLOCK_CASES))
def test_inverse_block(name, unfused):
    """y = GELU(W x + inverse(yhat)) in one call against the oracle's
    inverse followed by its block epilogue: the fused z + t expansion and
    epilogue kernel where the plan covers the shape, and the two launches of
    a plan made with PLAN_UNFUSED_BLOCK."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    spec, fusable = INVERSE_BLOCK_CASES[name]
    g = geometry(*spec)
    say(f"[inverse block {name} unfused={unfused}] n_global={g.n_global} n_local={g.n_local} kmax={g.kmax} "
        f"kt={g.kt} B={g.batch} Cin={g.c_in} Cout={g.c_out}")
    plan = D.Plan(desc_of(g), flags=D.PLAN_UNFUSED_BLOCK if unfused else 0)
    assert plan.block_fused == (fusable and not unfused)
    assert plan.block_ws_bytes >= plan.ws_bytes
    yh = rand_cplx((g.batch, g.c_out) + g.K, 140)
    x = rand_real((g.batch, g.c_in) + g.n_local, 141)
    wb = (rand_real((g.c_out, g.c_in), 142) / np.sqrt(g.c_in)).astype(np.float32)
    Y = Guarded(torch, plan.spatial_shape(g.c_out), torch.float32)
    plan.inverse_block(dev(torch, yh), dev(torch, x), dev(torch, wb), Y.t)
    torch.cuda.synchronize()
    check(np_of(Y.t), O.block_epilogue(x, wb, O.inverse(yh, g)), "inverse + block epilogue")
    assert Y.guards_intact()
    plan.close()


@pytest.mark.parametrize("name", ["fold", "dv20_tfold"])
def test_inverse_block_gelu_range(name):
    """The fused kernel's GELU over a wide range of arguments: a zero
    spectrum and W = I give y = GELU(x) exactly, with x swept over
    [-40, 40] (both tails, where the exponential underflows, and the region
    around zero).  The kernel's erf approximation is within 1.5e-7 of erf
    (Abramowitz & Stegun 7.1.26), i.e. Phi within 7.5e-8; the fp32 evaluation
    of q = Phi(-|x|) <= 1/2 (reciprocal, exponential, five FMAs, about ten
    roundings) adds at most 1e-6 relative to q; so |y - GELU(x)| <=
    (7.5e-8 + 5e-7) |x| plus one rounding of the result."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    spec, fusable = INVERSE_BLOCK_CASES[name]
    n_global, n_local, off, kmax, kt, B, _, _ = spec
    g = geometry(n_global, n_local, off, kmax, kt, B, 4, 4)
    say(f"[inverse block gelu range {name}] n_local={g.n_local} kt={g.kt}")
    plan = D.Plan(desc_of(g))
    assert plan.block_fused == 1
    yh = np.zeros((g.batch, g.c_out) + g.K, dtype=np.complex64)
    n = int(np.prod((g.batch, g.c_in) + g.n_local))
    v = np.linspace(-40.0, 40.0, n)
    v[: n // 2] = np.sign(v[: n // 2]) * np.abs(v[: n // 2]) ** 3 / 1600.0  # dense around zero too
    x = np.random.default_rng(143).permutation(v).astype(np.float32).reshape((g.batch, g.c_in) + g.n_local)
    wb = np.eye(g.c_out, g.c_in, dtype=np.float32)
    Y = Guarded(torch, plan.spatial_shape(g.c_out), torch.float32)
    plan.inverse_block(dev(torch, yh), dev(torch, x), dev(torch, wb), Y.t)
    torch.cuda.synchronize()
    ref = O.gelu(x.astype(np.float64))
    err = np.abs(np_of(Y.t).astype(np.float64) - ref)
    tol = 5.75e-7 * np.abs(x) + 6e-8 * np.abs(ref) + 1e-30
    assert np.all(err <= tol), float(np.max(err / tol))
    assert Y.guards_intact()
    plan.close()


def test_inverse_block_workspace_too_small():
    """A workspace below dtst_plan_block_info's size is rejected before any
    launch (the fused kernel also needs the y-expanded intermediate)."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry(*INVERSE_BLOCK_CASES["fold"][0])
    plan = D.Plan(desc_of(g))
    assert plan.block_fused == 1 and plan.block_ws_bytes > plan.ws_bytes
    yh = torch.zeros(plan.spectral_shape(g.c_out), dtype=torch.complex64, device="cuda")
    x = torch.zeros(plan.spatial_shape(g.c_in), dtype=torch.float32, device="cuda")
    wb = torch.zeros((g.c_out, g.c_in), dtype=torch.float32, device="cuda")
    y = torch.full(plan.spatial_shape(g.c_out), 3.0, dtype=torch.float32, device="cuda")
    small = torch.empty(plan.block_ws_bytes - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(D.DtstError) as e:
        D.dtst_inverse_block(plan.handle, yh, x, wb, y, small)
    assert e.value.status == 1
    torch.cuda.synchronize()
    assert bool((y == 3.0).all().item())
    plan.close()


@pytest.mark.parametrize("schedule", ["fused", "split"])
@pytest.mark.parametrize("name", FUSED_CASES)
def test_forward_schedules(name, schedule):
    """Both forward schedules (one t+z+y launch, or t+z then y, chosen by the
    plan option) against the oracle; the library's own per-kernel timing
    names the kernels that ran."""
    torch, D, g, plan = _setup(name, split=schedule == "split")
    x = rand_real((g.batch, g.c_in) + g.n_local, 111)
    ref = O.forward(x, g)
    out = Guarded(torch, plan.spectral_shape(g.c_in), torch.complex64)
    D.dtst_profile_collect()
    D.dtst_profile_enable(True)
    try:
        plan.forward(dev(torch, x), out.t)
        plan.forward(dev(torch, x), out.t, accumulate=True)
        torch.cuda.synchronize()
        ran = {k for k, (n, _) in D.dtst_profile_collect().items() if n > 0}
    finally:
        D.dtst_profile_enable(False)
    check(np_of(out.t), 2 * ref, f"forward ({schedule}) + accumulate")
    assert out.guards_intact()
    if schedule == "fused":
        assert "stream_fwd_tzy" in ran and "stream_fwd_tz" not in ran and "axis_fwd_y" not in ran, ran
    else:
        assert "stream_fwd_tz" in ran and "axis_fwd_y" in ran and "stream_fwd_tzy" not in ran, ran
    gy = rand_real((g.batch, g.c_out) + g.n_local, 112)
    out2 = Guarded(torch, plan.spectral_shape(g.c_out), torch.complex64)
    plan.inverse_adj(dev(torch, gy), out2.t)
    torch.cuda.synchronize()
    check(np_of(out2.t), O.inverse_adj(gy, g), f"inverse_adj ({schedule})")
    assert out2.guards_intact()


@pytest.mark.parametrize("schedule", ["fused", "split"])
@pytest.mark.parametrize("name", FUSED_CASES)
def test_inverse_schedules(name, schedule):
    """Both inverse schedules (y + z + t in one launch, or y then z + t,
    chosen by the plan option) for the inverse and forward_adj against the
    oracle, with the kernels that ran."""
    torch, D, g, plan = _setup(name, split=schedule == "split")
    yh = rand_cplx((g.batch, g.c_out) + g.K, 113)
    out = Guarded(torch, plan.spatial_shape(g.c_out), torch.float32)
    D.dtst_profile_collect()
    D.dtst_profile_enable(True)
    try:
        plan.inverse(dev(torch, yh), out.t)
        torch.cuda.synchronize()
        ran = {k for k, (n, _) in D.dtst_profile_collect().items() if n > 0}
    finally:
        D.dtst_profile_enable(False)
    check(np_of(out.t), O.inverse(yh, g), f"inverse ({schedule})")
    assert out.guards_intact()
    if schedule == "fused":
        assert "stream_inv_yzt" in ran and "stream_inv_zt" not in ran and "axis_inv_y" not in ran, ran
    else:
        assert "stream_inv_zt" in ran and "axis_inv_y" in ran and "stream_inv_yzt" not in ran, ran
    G = rand_cplx((g.batch, g.c_in) + g.K, 114)
    out2 = Guarded(torch, plan.spatial_shape(g.c_in), torch.float32)
    plan.forward_adj(dev(torch, G), out2.t)
    torch.cuda.synchronize()
    check(np_of(out2.t), O.forward_adj(G, g), f"forward_adj ({schedule})")
    assert out2.guards_intact()


@pytest.mark.parametrize("name", ["fold_ragged", "kt16_two_col_tiles"])
def test_one_plan_two_streams(name):
    """A plan used from two streams at once, each call with its own
    workspace (the concurrency contract of the C ABI): forward and inverse
    calls interleaved on two default-priority streams give each stream's
    oracle result."""
    torch, D, g, plan = _setup(name)
    xs = [rand_real((g.batch, g.c_in) + g.n_local, 120 + s) for s in range(2)]
    yhs = [rand_cplx((g.batch, g.c_out) + g.K, 130 + s) for s in range(2)]
    xd = [dev(torch, a) for a in xs]
    yd = [dev(torch, a) for a in yhs]
    wss = [torch.empty(max(plan.ws_bytes, 16), dtype=torch.uint8, device="cuda") for _ in range(2)]
    outs = [torch.empty(plan.spectral_shape(g.c_in), dtype=torch.complex64, device="cuda") for _ in range(2)]
    backs = [torch.empty(plan.spatial_shape(g.c_out), dtype=torch.float32, device="cuda") for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    cur = torch.cuda.current_stream()
    for st in streams:
        st.wait_stream(cur)
    for _ in range(3):
        for s, st in enumerate(streams):
            D.dtst_forward(plan.handle, xd[s], outs[s], 0, wss[s], stream=st.cuda_stream)
            D.dtst_inverse(plan.handle, yd[s], backs[s], wss[s], stream=st.cuda_stream)
    for st in streams:
        cur.wait_stream(st)
    torch.cuda.synchronize()
    for s in range(2):
        check(np_of(outs[s]), O.forward(xs[s], g), f"forward on stream {s}")
        check(np_of(backs[s]), O.inverse(yhs[s], g), f"inverse on stream {s}")


@pytest.mark.parametrize("name", ["fold_ragged", "kt16_two_col_tiles"])
def test_graph_capture_replays(name):
    """The execute calls allocate nothing, synchronise nothing and record
    no memset, so a layer step (forward, mix, inverse) can be captured in a
    HIP graph.  The graph is replayed several times, with eager work and
    synchronisation between the replays, and every replay is checked
    against the eager result."""
    torch, D, g, plan = _setup(name)
    M = plan.n_modes
    x = dev(torch, rand_real((g.batch, g.c_in) + g.n_local, 140))
    W = dev(torch, rand_cplx((M, g.c_in, g.c_out), 141, var=1.0 / (g.c_in * g.c_out)))
    xhat = torch.empty(plan.spectral_shape(g.c_in), dtype=torch.complex64, device="cuda")
    yhat = torch.empty(plan.spectral_shape(g.c_out), dtype=torch.complex64, device="cuda")
    y = torch.empty(plan.spatial_shape(g.c_out), dtype=torch.float32, device="cuda")

    def step():
        plan.forward(x, xhat)
        plan.mix(xhat, W, yhat, 0, M, op=0)
        plan.inverse(yhat, y)

    step()
    torch.cuda.synchronize()
    eager = np_of(y).copy()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    for r in range(3):
        y.fill_(-3.0)
        xhat.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = np_of(y)
        assert np.array_equal(got, eager), f"replay {r} differs from the eager step"
    check(eager, O.inverse(O.mix(O.forward(np_of(x), g), np_of(W), 0, M).reshape(plan.spectral_shape(g.c_out)), g),
          "eager step vs oracle")


@pytest.mark.parametrize("name", ["fold", "full_c16"])
def test_graph_capture_replays_block(name):
    """The block of Algorithm 1 (forward, mix, fused inverse + bypass + GELU)
    captured in a HIP graph: the fused block kernel records no memset and
    allocates nothing, so every replay (with eager work and synchronisation
    between them) equals the eager step bit for bit, and the eager step
    matches the oracle."""
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    spec, fusable = INVERSE_BLOCK_CASES[name]
    g = geometry(*spec)
    say(f"[graph block {name}] n_local={g.n_local} kmax={g.kmax} kt={g.kt} Cin={g.c_in} Cout={g.c_out}")
    plan = D.Plan(desc_of(g))
    assert plan.block_fused == fusable
    M = plan.n_modes
    x = dev(torch, rand_real((g.batch, g.c_in) + g.n_local, 150))
    W = dev(torch, rand_cplx((M, g.c_in, g.c_out), 151, var=1.0 / (g.c_in * g.c_out)))
    wb = dev(torch, (rand_real((g.c_out, g.c_in), 152) / np.sqrt(g.c_in)).astype(np.float32))
    xhat = torch.empty(plan.spectral_shape(g.c_in), dtype=torch.complex64, device="cuda")
    yhat = torch.empty(plan.spectral_shape(g.c_out), dtype=torch.complex64, device="cuda")
    y = torch.empty(plan.spatial_shape(g.c_out), dtype=torch.float32, device="cuda")

    def step():
        plan.forward(x, xhat)
        plan.mix(xhat, W, yhat, 0, M, op=0)
        plan.inverse_block(yhat, x, wb, y)

    step()
    torch.cuda.synchronize()
    eager = np_of(y).copy()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    for r in range(3):
        y.fill_(-3.0)
        xhat.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(np_of(y), eager), f"replay {r} differs from the eager step"
    yh = O.mix(O.forward(np_of(x), g), np_of(W), 0, M).reshape(plan.spectral_shape(g.c_out))
    check(eager, O.block_epilogue(np_of(x), np_of(wb), O.inverse(yh, g)), "eager block vs oracle")
    plan.close()
