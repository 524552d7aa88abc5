"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function declared in include/dtst.h, validates descriptors, sizes its
workspace, and builds fp32 basis tables that agree with the fp64 oracle's
basis rounded to fp32."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
D = pytest.importorskip("paper_2607_14394_amd", reason="libdtst.so not built")


def header_functions():
    src = open(os.path.join(ROOT, "include", "dtst.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dtst_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = header_functions()
    assert "dtst_forward" in names and "dtst_mix_wgrad" in names and "dtst_inverse_adj" in names
    lib = ctypes.CDLL(D.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def desc(**kw):
    base = dict(n_global=(12, 10, 8, 8), n_local=(4, 10, 8, 8), offset=(4, 0, 0, 0), kmax=(3, 2, 2), kt=3,
                batch=1, c_in=2, c_out=3)
    base.update(kw)
    return D.make_desc(**base)


def test_valid_descriptor():
    D.dtst_desc_validate(desc())
    D.dtst_desc_validate(desc(batch=0))
    D.dtst_desc_validate(desc(c_out=512))
    D.dtst_desc_validate(desc(n_global=(12, 10, 128, 64), n_local=(4, 10, 128, 64), kmax=(3, 2, 64), kt=16))


@pytest.mark.parametrize("kw,status", [
    (dict(kmax=(7, 2, 2)), 1),                       # 2k > N
    (dict(kmax=(0, 2, 2)), 1),                       # k = 0
    (dict(kt=6), 1),                                 # kt > N_t/2 + 1
    (dict(kt=0), 1),
    (dict(offset=(10, 0, 0, 0)), 1),                 # offset + local > global
    (dict(offset=(-1, 0, 0, 0)), 1),
    (dict(n_local=(0, 10, 8, 8)), 1),
    (dict(n_global=(12, 10, 8, 0), n_local=(4, 10, 8, 0)), 1),
    (dict(batch=-1), 1),
    (dict(c_in=0), 1),
    (dict(c_out=0), 1),
    (dict(n_global=(12, 10, 8, 80), n_local=(4, 10, 8, 80), kt=20), 2),   # kt > 16: not covered
    (dict(n_global=(12, 10, 8, 80), n_local=(4, 10, 8, 80), kt=4), 2),    # N_t local > 64
    (dict(c_out=513), 2),                                                   # mix kernels take C_out <= 512
    (dict(n_global=(12, 10, 260, 8), n_local=(4, 10, 260, 8), kmax=(3, 2, 65)), 2),  # > 64 z modes per class
])
def test_invalid_descriptors(kw, status):
    with pytest.raises(D.DtstError) as e:
        D.dtst_desc_validate(desc(**kw))
    assert e.value.status == status
    assert str(e.value)


def test_workspace_bytes():
    d = desc(batch=2, c_in=2, c_out=3)
    # complex intermediates of the largest channel count: (.., Nx, Ky, Kz, Kt) between the y and x
    # steps, and (.., Nx, Ny, Kz, Kt) between the t+z and y steps when those are separate launches
    w1 = 2 * 3 * 4 * 10 * 4 * 3 * 8
    w2 = 2 * 3 * 4 * 4 * 4 * 3 * 8
    r = lambda v: (v + 255) // 256 * 256
    assert D.dtst_desc_workspace_bytes(d) == r(w2)          # y fused into the stream kernels
    assert D.dtst_desc_workspace_bytes(desc(batch=0)) == 0
    # N_t = 6 (not a multiple of 4) keeps the separate launches
    d6 = desc(batch=2, c_in=2, c_out=3, n_global=(12, 10, 8, 6), n_local=(4, 10, 8, 6))
    assert D.dtst_desc_workspace_bytes(d6) == r(2 * 3 * 4 * 10 * 4 * 3 * 8) + r(w2)
    assert D.dtst_desc_workspace_bytes(d, D.PLAN_SPLIT_SCHEDULE) == r(w1) + r(w2)
    # the library reads no environment: the schedule is a plan option only
    os.environ["DTST_SCHEDULE"] = "split"
    try:
        assert D.dtst_desc_workspace_bytes(d) == r(w2)
    finally:
        del os.environ["DTST_SCHEDULE"]


def test_unknown_plan_flag_rejected():
    n = ctypes.c_size_t(0)
    st = D.lib.dtst_desc_workspace_bytes_ex(ctypes.byref(desc()), 4, ctypes.byref(n))
    assert st == 1 and b"flag" in D.lib.dtst_last_error()
    # the two documented flags, alone and together, are accepted
    for flags in (D.PLAN_SPLIT_SCHEDULE, D.PLAN_UNFUSED_BLOCK, D.PLAN_SPLIT_SCHEDULE | D.PLAN_UNFUSED_BLOCK):
        assert D.lib.dtst_desc_workspace_bytes_ex(ctypes.byref(desc()), flags, ctypes.byref(n)) == 0
    h = ctypes.c_void_p()
    st = D.lib.dtst_plan_ex(ctypes.byref(desc()), 1 << 31, ctypes.byref(h))
    assert st == 1 and h.value is None


@pytest.mark.parametrize("g", [
    ((12, 10, 8, 8), (4, 10, 8, 8), (4, 0, 0, 0), (3, 2, 2), 3),
    ((512, 512, 512, 32), (32, 512, 512, 32), (480, 0, 0, 0), (16, 16, 16), 8),
    ((9, 7, 5, 6), (3, 7, 5, 6), (6, 0, 0, 0), (2, 3, 1), 4),
])
def test_basis_tables_match_oracle(g):
    ng, nl, off, k, kt = g
    d = D.make_desc(ng, nl, off, k, kt, 1, 1, 1)
    idx = [O.retained_indices(ng[i], k[i]) for i in range(3)] + [O.retained_t(kt)]
    for dim in range(4):
        ref = O.basis(ng[dim], off[dim], nl[dim], idx[dim])
        got = D.dtst_basis_host(d, dim, 0)
        assert got.shape == ref.shape
        assert np.abs(got - ref).max() <= 1.2e-7       # one fp32 ulp at |v| <= 1
        got_c = D.dtst_basis_host(d, dim, 1)
        assert np.abs(got_c - np.conj(ref)).max() <= 1.2e-7


def test_basis_rejects_bad_request():
    d = desc()
    with pytest.raises(D.DtstError):
        D.dtst_basis_host(d, 4, 0)
    buf = (ctypes.c_float * 8)()
    st = D.lib.dtst_basis_host(ctypes.byref(d), 0, 0, buf, 8)
    assert st == 1 and b"count" in D.lib.dtst_last_error()


def test_status_strings():
    for s, name in D.STATUS_NAMES.items():
        assert D.lib.dtst_status_string(s).decode() == name


def test_destroyed_or_null_plan_rejected_without_gpu():
    st = D.lib.dtst_plan_destroy(None)
    assert st == 1
    st = D.lib.dtst_plan_info(ctypes.c_void_p(12345), None, None)
    assert st == 1
    st = D.lib.dtst_forward(None, None, None, 0, None, 0, None)
    assert st == 1
