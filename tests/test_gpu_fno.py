"""GPU parity of the FNO forward (lift, four Fourier layers of Algorithm 1,
projection) run through the library on the shards of a decomposition, one
after another, against the fp64 oracle's FNO forward on the whole domain
(the result does not depend on the decomposition).  Also the point-wise
layer (lift / projection) against the oracle on its own."""

import numpy as np
import pytest

import oracle as O
import synth
from gpu_common import check, dev, np_of, say, torch_gpu

pytestmark = pytest.mark.gpu

# name: (n_global, kmax, kt, batch, d_v, C_in, C_out, shard grid (x, y))
CASES = {
    "one_shard": ((12, 10, 8, 8), (3, 2, 2), 3, 2, 4, 3, 2, (1, 1)),
    "x_slabs": ((12, 10, 8, 8), (3, 2, 2), 3, 2, 4, 3, 2, (2, 1)),
    "pencils": ((12, 10, 8, 8), (3, 2, 2), 3, 1, 4, 3, 2, (2, 2)),
    # k_t = 16 of N_t = 32, as the paper's modes (8, 8, 8, 16): the separate t+z and y launches
    "kt16_slabs": ((8, 8, 16, 32), (2, 2, 4), 16, 1, 5, 2, 3, (2, 1)),
    # the paper's width d_v = 20 (Sec. VI-A) with five fields in and out, on a small grid
    "dv20_small": ((8, 8, 16, 32), (2, 2, 4), 16, 1, 20, 5, 5, (2, 1)),
    # the paper's model shape (Sec. VI-A): d_v = 20, modes (8, 8, 8, 16) -- K = 16 of each
    # spatial dimension and k_t = 16 -- on a 32^3 x 32 grid in 4 x-slabs of 8 (P = 4)
    "paper_model_32cubed": ((32, 32, 32, 32), (8, 8, 8), 16, 1, 20, 5, 5, (4, 1)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_fno_forward_matches_oracle(name):
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    from paper_2607_14394_amd.fno import FNO
    ng, kmax, kt, B, dv, cin, cout, (gx, gy) = CASES[name]
    say(f"[fno {name}] n_global={ng} kmax={kmax} kt={kt} B={B} d_v={dv} C_in={cin} C_out={cout} grid={gx}x{gy}")
    g = O.Geometry(ng, ng, (0, 0, 0, 0), kmax, kt, B, dv, dv)
    M = O.n_modes(g)
    lift, layers, proj = synth.fno_params_np(M, dv, cin, cout, 4, 7100)
    x = synth.np_normal((B, cin) + ng, 7000)
    ref = O.fno_forward(x, g, lift, layers, proj)

    lx, ly = ng[0] // gx, ng[1] // gy
    descs, xs = [], []
    for p in range(gx * gy):
        ox, oy = (p // gy) * lx, (p % gy) * ly
        descs.append(D.make_desc(ng, (lx, ly, ng[2], ng[3]), (ox, oy, 0, 0), kmax, kt, B, dv, dv))
        xs.append(dev(torch, x[:, :, ox:ox + lx, oy:oy + ly]))
    t = lambda a: dev(torch, a)
    fno = FNO(descs, (t(lift[0]), t(lift[1])), [(t(r), t(w)) for r, w in layers], (t(proj[0]), t(proj[1])))
    outs = [torch.empty(fno.output_shape(p), dtype=torch.float32, device="cuda") for p in range(len(descs))]
    fno.forward(xs, outs)
    torch.cuda.synchronize()
    got = np.empty_like(ref)
    for p, o in enumerate(outs):
        ox, oy = (p // gy) * lx, (p % gy) * ly
        got[:, :, ox:ox + lx, oy:oy + ly] = np_of(o)
    fno.close()
    check(got, ref, "fno forward")


@pytest.mark.parametrize("act", [0, 1])
@pytest.mark.parametrize("points", [4096, 1001])
def test_pointwise_matches_oracle(act, points):
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    B, ci, co = 2, 5, 20
    x = synth.np_normal((B, ci, points), 7200)
    w = synth.np_normal((co, ci), 7201)
    b = synth.np_normal((co,), 7202)
    y = torch.full((B, co, points), -7.25, dtype=torch.float32, device="cuda")
    D.dtst_pointwise(dev(torch, x), dev(torch, w), dev(torch, b), y, act=act)
    torch.cuda.synchronize()
    check(np_of(y), O.pointwise(x, w, b, act=bool(act)), f"pointwise act={act}")
    y2 = torch.empty((B, co, points), dtype=torch.float32, device="cuda")
    D.dtst_pointwise(dev(torch, x), dev(torch, w), None, y2, act=act)
    torch.cuda.synchronize()
    check(np_of(y2), O.pointwise(x, w, None, act=bool(act)), f"pointwise act={act} no bias")


def test_pointwise_rejects_bad_arguments():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    x = torch.zeros((1, 4, 64), dtype=torch.float32, device="cuda")
    w = torch.zeros((8, 4), dtype=torch.float32, device="cuda")
    y = torch.zeros((1, 8, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(D.DtstError) as e:       # act must be 0 or 1
        D._check(D.lib.dtst_pointwise(D._ptr(x), D._ptr(w), None, D._ptr(y), 1, 4, 8, 64, 2, None))
    assert e.value.status == 1
    with pytest.raises(D.DtstError) as e:       # in place is not allowed
        D._check(D.lib.dtst_pointwise(D._ptr(x), D._ptr(w), None, D._ptr(x), 1, 4, 4, 64, 0, None))
    assert e.value.status == 1 and "overlap" in str(e.value)
    with pytest.raises(D.DtstError) as e:       # weights beyond the LDS limit
        D._check(D.lib.dtst_pointwise(D._ptr(x), D._ptr(w), None, D._ptr(y), 1, 400, 400, 64, 0, None))
    assert e.value.status == 2
