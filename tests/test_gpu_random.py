"""Parity on seeded random geometries: extents, shards, mode counts, k_t,
batch and channel counts drawn at random (odd and even extents, folded and
unfolded dimensions, ragged tiles, sharded t), so that the kernels' shape
logic is exercised in combinations the named cases do not list.  Every
geometry is regenerated from its seed; the ones the library does not cover
(its kernel limits) are left out when the list is built."""

import numpy as np
import pytest

import oracle as O
from gpu_common import Guarded, check, desc_of, dev, geometry, np_of, rand_cplx, rand_real, say, torch_gpu

pytestmark = pytest.mark.gpu

N_SMALL = 48   # extents up to 16 x 24 x 48
N_LARGE = 16   # y up to 80 and z up to 96: several fused slot groups and z tiles
_T_EXTENTS = (3, 4, 5, 6, 8, 10, 12, 16, 21, 24, 32)


def _draw(seed, large):
    rng = np.random.default_rng(seed)
    if large:
        ng = [int(rng.integers(2, 9)), int(rng.integers(16, 81)), int(rng.integers(16, 97)),
              int(rng.choice((8, 12, 16, 24, 32)))]
    else:
        ng = [int(rng.integers(2, 17)), int(rng.integers(2, 25)), int(rng.integers(2, 49)),
              int(rng.choice(_T_EXTENTS))]
    split_prob = (0.5, 0.3, 0.2, 0.15)
    nl, off = [], []
    for d in range(4):
        if rng.random() < split_prob[d]:
            n = int(rng.integers(1, ng[d] + 1))
            nl.append(n)
            off.append(int(rng.integers(0, ng[d] - n + 1)))
        else:
            nl.append(ng[d])
            off.append(0)
    kmax = [int(rng.integers(1, ng[d] // 2 + 1)) for d in range(3)]
    kt = int(rng.integers(1, min(16, ng[3] // 2 + 1) + 1))
    if large:
        return (tuple(ng), tuple(nl), tuple(off), tuple(kmax), kt, 1, int(rng.integers(1, 4)),
                int(rng.integers(1, 4)))
    return (tuple(ng), tuple(nl), tuple(off), tuple(kmax), kt, int(rng.integers(1, 3)),
            int(rng.integers(1, 6)), int(rng.integers(1, 6)))


def _family(first_seed, count, large, D):
    out, seed = [], first_seed
    while len(out) < count and seed < first_seed + 40 * count:
        args = _draw(seed, large)
        seed += 1
        g = geometry(*args)
        try:
            g.validate()
            D.dtst_desc_validate(desc_of(g))
        except Exception:
            continue
        out.append((seed - 1, args))
    return out


def _cases():
    try:
        import paper_2607_14394_amd as D
    except Exception:  # library not built: the module is skipped below
        return []
    return _family(7000, N_SMALL, False, D) + _family(9000, N_LARGE, True, D)


CASES = _cases()
if not CASES:
    pytestmark = [pytest.mark.gpu, pytest.mark.skip(reason="libdtst.so not built")]


def _setup(seed, args, split):
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    g = geometry(*args)
    say(f"[random seed {seed}{' split' if split else ''}] n_global={g.n_global} n_local={g.n_local} "
        f"offset={g.offset} kmax={g.kmax} kt={g.kt} B={g.batch} Cin={g.c_in} Cout={g.c_out}")
    return torch, D, g, D.Plan(desc_of(g), flags=D.PLAN_SPLIT_SCHEDULE if split else 0)


@pytest.mark.parametrize("idx", range(len(CASES)))
def test_random_geometry(idx):
    seed, args = CASES[idx]
    # every fourth geometry also forces the separate t+z / y launches
    torch, D, g, plan = _setup(seed, args, idx % 4 == 3)
    M = plan.n_modes

    x = rand_real((g.batch, g.c_in) + g.n_local, seed)
    ref = O.forward(x, g)
    out = Guarded(torch, plan.spectral_shape(g.c_in), torch.complex64)
    plan.forward(dev(torch, x), out.t)
    plan.forward(dev(torch, x), out.t, accumulate=True)
    torch.cuda.synchronize()
    check(np_of(out.t), 2 * ref, "forward twice, accumulated")
    assert out.guards_intact()

    yh = rand_cplx((g.batch, g.c_out) + g.K, seed + 1)
    outy = Guarded(torch, plan.spatial_shape(g.c_out), torch.float32)
    plan.inverse(dev(torch, yh), outy.t)
    torch.cuda.synchronize()
    check(np_of(outy.t), O.inverse(yh, g), "inverse")
    assert outy.guards_intact()

    G = rand_cplx((g.batch, g.c_in) + g.K, seed + 2)
    ga = Guarded(torch, plan.spatial_shape(g.c_in), torch.float32)
    plan.forward_adj(dev(torch, G), ga.t)
    gy = rand_real((g.batch, g.c_out) + g.n_local, seed + 3)
    gb = Guarded(torch, plan.spectral_shape(g.c_out), torch.complex64)
    plan.inverse_adj(dev(torch, gy), gb.t)
    torch.cuda.synchronize()
    check(np_of(ga.t), O.forward_adj(G, g), "forward_adj")
    check(np_of(gb.t), O.inverse_adj(gy, g), "inverse_adj")
    assert ga.guards_intact() and gb.guards_intact()

    # mix, data gradient and weight gradient on a random mode range
    rng = np.random.default_rng(seed + 4)
    m0 = int(rng.integers(0, M))
    m1 = int(rng.integers(m0 + 1, M + 1))
    X = rand_cplx((g.batch, g.c_in) + g.K, seed + 5)
    W = rand_cplx((m1 - m0, g.c_in, g.c_out), seed + 6, var=1.0 / (g.c_in * g.c_out))
    base = rand_cplx((g.batch, g.c_out) + g.K, seed + 7)
    Y = Guarded(torch, plan.spectral_shape(g.c_out), torch.complex64, fill=dev(torch, base))
    plan.mix(dev(torch, X), dev(torch, W), Y.t, m0, m1, op=0)
    GY = rand_cplx((g.batch, g.c_out) + g.K, seed + 8)
    GX = Guarded(torch, plan.spectral_shape(g.c_in), torch.complex64, fill=dev(torch, rand_cplx((g.batch, g.c_in) + g.K, seed + 9)))
    plan.mix(dev(torch, GY), dev(torch, W), GX.t, m0, m1, op=1)
    GW = Guarded(torch, (m1 - m0, g.c_in, g.c_out), torch.complex64)
    plan.wgrad(dev(torch, X), dev(torch, GY), GW.t, m0, m1)
    torch.cuda.synchronize()
    got = np_of(Y.t).reshape(g.batch, g.c_out, M)
    ref = O.mix(X, W, m0, m1, yhat_in=base)
    check(got[:, :, m0:m1], ref[:, :, m0:m1], "mix range")
    assert np.array_equal(got[:, :, :m0], base.reshape(g.batch, g.c_out, M)[:, :, :m0])
    assert np.array_equal(got[:, :, m1:], base.reshape(g.batch, g.c_out, M)[:, :, m1:])
    gx = np_of(GX.t).reshape(g.batch, g.c_in, M)
    check(gx[:, :, m0:m1], O.mix_data_grad(GY, W, m0, m1)[:, :, m0:m1], "mix data grad range")
    check(np_of(GW.t), O.mix_wgrad(X, GY, m0, m1), "wgrad range")
    assert Y.guards_intact() and GX.guards_intact() and GW.guards_intact()
