"""dtst_forward_noalloc, the forward for callers that cannot allocate: its
workspace is the library's per-device scratch array.  Called through the C
ABI and checked against dtst_forward (the existing entry point, same
kernels) and the fp64 oracle, on two calls in a row, the second with a
smaller input; plans whose workspace exceeds the array are rejected."""

import ctypes

import numpy as np
import pytest

import oracle as O
from gpu_common import check, desc_of, dev, geometry, np_of, rand_real, say, torch_gpu

pytestmark = pytest.mark.gpu

# (n_global, n_local, offset, kmax, kt, B, C_in, C_out): a slab of the fused
# schedule with several slot groups, then a smaller shard on the split schedule
# (odd extents, t not a multiple of 4)
FIRST = ((64, 64, 64, 32), (16, 64, 64, 32), (32, 0, 0, 0), (16, 16, 16), 8, 1, 3, 2)
SECOND = ((9, 7, 5, 6), (3, 7, 5, 6), (6, 0, 0, 0), (2, 3, 1), 4, 1, 2, 1)


def _noalloc(D, plan, x, xhat, accumulate):
    st = D.lib.dtst_forward_noalloc(plan.handle, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(xhat.data_ptr()),
                                    int(accumulate), ctypes.c_void_p(D.torch_stream()))
    D._check(st)


def _run(torch, D, args, seed):
    g = geometry(*args)
    plan = D.Plan(desc_of(g))
    say(f"[noalloc] n_global={g.n_global} n_local={g.n_local} workspace={plan.ws_bytes} B")
    assert 0 < plan.ws_bytes <= D.SCRATCH_BYTES
    x = rand_real((g.batch, g.c_in) + g.n_local, seed)
    xd = dev(torch, x)
    ref_dev = torch.empty(plan.spectral_shape(g.c_in), dtype=torch.complex64, device="cuda")
    plan.forward(xd, ref_dev)
    got = torch.full(plan.spectral_shape(g.c_in), complex(-7.25, 3.5), dtype=torch.complex64, device="cuda")
    _noalloc(D, plan, xd, got, 0)
    torch.cuda.synchronize()
    # the same kernels on the same input: identical to dtst_forward, and to the oracle within tolerance
    assert np.array_equal(np_of(got), np_of(ref_dev))
    ref = O.forward(x, g)
    check(np_of(got), ref, "forward_noalloc")
    _noalloc(D, plan, xd, got, 1)
    torch.cuda.synchronize()
    check(np_of(got), 2 * ref, "forward_noalloc accumulate")
    plan.close()


def test_noalloc_matches_forward_twice_then_smaller():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    _run(torch, D, FIRST, 301)
    _run(torch, D, SECOND, 302)


def test_noalloc_rejects_a_workspace_above_the_scratch_array():
    torch = torch_gpu()
    import paper_2607_14394_amd as D
    # (.., N_x, K_y, K_z, K_t) complex intermediate: 64 x 32 x 32 x 8 x 17 channels x 8 B > 64 MiB
    g = geometry((128, 128, 128, 32), (64, 128, 128, 32), (0, 0, 0, 0), (16, 16, 16), 8, 1, 17, 17)
    plan = D.Plan(desc_of(g))
    assert plan.ws_bytes > D.SCRATCH_BYTES
    x = torch.zeros(64, dtype=torch.float32, device="cuda")     # never read: the call is rejected first
    out = torch.full((64,), complex(5.0, 0.0), dtype=torch.complex64, device="cuda")
    with pytest.raises(D.DtstError) as e:
        _noalloc(D, plan, x, out, 0)
    assert e.value.status == 2 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 5.0).all().item())
    plan.close()
