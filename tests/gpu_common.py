"""Helpers shared by the GPU parity tests (not a test module)."""

import math
import sys

import numpy as np
import pytest

import oracle as O
import synth

# Tolerances fixed for the fp32 path against the fp64 oracle: relative L2
# error of the whole output tensor, and the largest absolute error relative
# to the RMS of the oracle's output.
REL_L2 = 1e-5
MAXABS_RMS = 1e-4


def torch_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def errors(got, ref):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = (got.astype(np.complex128) - ref.astype(np.complex128)).ravel()
    nref = np.linalg.norm(ref.ravel())
    rms = nref / math.sqrt(max(ref.size, 1))
    rel = np.linalg.norm(d) / max(nref, 1e-300)
    mx = np.abs(d).max() / max(rms, 1e-300) if d.size else 0.0
    return rel, mx


def check(got, ref, name, rel_l2=REL_L2, maxabs_rms=MAXABS_RMS):
    rel, mx = errors(got, ref)
    say(f"  {name}: rel_l2={rel:.2e} maxabs/rms={mx:.2e}")
    assert rel <= rel_l2 and mx <= maxabs_rms, f"{name}: rel_l2={rel:.3e} maxabs/rms={mx:.3e}"


def geometry(ng, nl, off, k, kt, b, ci, co):
    return O.Geometry(tuple(ng), tuple(nl), tuple(off), tuple(k), kt, b, ci, co)


def desc_of(g):
    import paper_2607_14394_amd as D
    return D.make_desc(g.n_global, g.n_local, g.offset, g.kmax, g.kt, g.batch, g.c_in, g.c_out)


class Guarded:
    """A device tensor surrounded by guard bands filled with a sentinel, to
    catch writes outside the output."""

    PAD = 64

    def __init__(self, torch, shape, dtype, fill=None):
        n = int(np.prod(shape))
        self.torch = torch
        self.buf = torch.empty(n + 2 * self.PAD, dtype=dtype, device="cuda")
        if dtype == torch.complex64:
            self.buf.copy_(torch.full((n + 2 * self.PAD,), complex(-7.25, 3.5), dtype=dtype))
        else:
            self.buf.fill_(-7.25)
        self.t = self.buf[self.PAD:self.PAD + n].view(shape)
        if fill is not None:
            self.t.copy_(fill)
        self.n = n

    def guards_intact(self):
        torch = self.torch
        lo = self.buf[:self.PAD]
        hi = self.buf[self.PAD + self.n:]
        if self.buf.dtype == torch.complex64:
            want = complex(-7.25, 3.5)
            return bool((lo == want).all().item() and (hi == want).all().item())
        return bool((lo == -7.25).all().item() and (hi == -7.25).all().item())


def np_of(t):
    return t.detach().cpu().numpy()


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def rand_real(shape, seed):
    return synth.np_normal(shape, seed, dtype=np.float32)


def rand_cplx(shape, seed, var=1.0):
    return synth.np_complex_normal(shape, seed, var=var)
