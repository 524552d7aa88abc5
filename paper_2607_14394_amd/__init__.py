"""Python binding of the DTST spectral-layer library (libdtst.so).

Argument marshalling only: every function here forwards to the C ABI of the
same name declared in ``include/dtst.h``.  Device arrays are torch tensors
(PyTorch provides device memory and streams); their data pointers and the
current HIP stream are passed straight through.  The library must be built
(``python paper_2607_14394_amd/build.py``); importing this module fails
loudly when it is missing -- there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os

__all__ = [
    "DtstError", "Desc", "lib", "make_desc", "dtst_desc_validate", "dtst_desc_workspace_bytes",
    "dtst_basis_host", "dtst_plan", "dtst_plan_destroy", "dtst_plan_info", "dtst_forward", "dtst_mix",
    "dtst_inverse", "dtst_forward_adj", "dtst_inverse_adj", "dtst_mix_wgrad", "dtst_block_epilogue",
    "dtst_inverse_block", "dtst_pointwise", "dtst_forward_noalloc", "dtst_profile_enable",
    "dtst_profile_collect", "dtst_plan_block_info", "Plan", "LIB_PATH", "PLAN_SPLIT_SCHEDULE",
    "PLAN_UNFUSED_BLOCK", "SCRATCH_BYTES", "torch_stream",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdtst.so")

DTST_OK = 0
PLAN_SPLIT_SCHEDULE = 1      # DTST_PLAN_SPLIT_SCHEDULE of include/dtst.h
PLAN_UNFUSED_BLOCK = 2       # DTST_PLAN_UNFUSED_BLOCK of include/dtst.h
SCRATCH_BYTES = 64 << 20     # DTST_SCRATCH_BYTES of include/dtst.h
STATUS_NAMES = {0: "DTST_OK", 1: "DTST_ERR_INVALID_ARG", 2: "DTST_ERR_UNSUPPORTED",
                3: "DTST_ERR_OUT_OF_MEMORY", 4: "DTST_ERR_DEVICE"}


class DtstError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 40), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


class Desc(ctypes.Structure):
    _fields_ = [
        ("n_global", ctypes.c_int64 * 4),
        ("n_local", ctypes.c_int64 * 4),
        ("offset", ctypes.c_int64 * 4),
        ("kmax", ctypes.c_int32 * 3),
        ("kt", ctypes.c_int32),
        ("batch", ctypes.c_int64),
        ("c_in", ctypes.c_int64),
        ("c_out", ctypes.c_int64),
    ]


def _load():
    # torch ships its own HIP runtime under the same soname (libamdhip64.so.7).
    # Loading torch first makes libdtst.so bind to that one copy; loading
    # libdtst.so first would bring a second HIP/HSA runtime into the process,
    # and one of the two then finds no device.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libdtst.so not found at {LIB_PATH}; build it with "
                          "`python paper_2607_14394_amd/build.py` (no fallback path exists)")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, SZ, I, VP = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p
    sig = {
        "dtst_desc_validate": [ctypes.POINTER(Desc)],
        "dtst_desc_workspace_bytes": [ctypes.POINTER(Desc), ctypes.POINTER(SZ)],
        "dtst_desc_workspace_bytes_ex": [ctypes.POINTER(Desc), ctypes.c_uint32, ctypes.POINTER(SZ)],
        "dtst_basis_host": [ctypes.POINTER(Desc), I, I, ctypes.POINTER(ctypes.c_float), SZ],
        "dtst_plan": [ctypes.POINTER(Desc), ctypes.POINTER(P)],
        "dtst_plan_ex": [ctypes.POINTER(Desc), ctypes.c_uint32, ctypes.POINTER(P)],
        "dtst_plan_destroy": [P],
        "dtst_plan_info": [P, ctypes.POINTER(I64), ctypes.POINTER(SZ)],
        "dtst_plan_block_info": [P, ctypes.POINTER(SZ), ctypes.POINTER(I)],
        "dtst_forward": [P, VP, VP, I, VP, SZ, VP],
        "dtst_mix": [P, VP, VP, VP, I64, I64, I, VP],
        "dtst_inverse": [P, VP, VP, VP, SZ, VP],
        "dtst_forward_adj": [P, VP, VP, VP, SZ, VP],
        "dtst_inverse_adj": [P, VP, VP, I, VP, SZ, VP],
        "dtst_mix_wgrad": [P, VP, VP, VP, I64, I64, I, VP],
        "dtst_block_epilogue": [P, VP, VP, VP, VP],
        "dtst_inverse_block": [P, VP, VP, VP, VP, VP, SZ, VP],
        "dtst_pointwise": [VP, VP, VP, VP, I64, I64, I64, I64, I, VP],
        "dtst_forward_noalloc": [P, VP, VP, I, VP],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.dtst_profile_enable.argtypes = [I]
    L.dtst_profile_enable.restype = ctypes.c_int
    L.dtst_profile_collect.argtypes = [ctypes.POINTER(KernelTime), I, ctypes.POINTER(I)]
    L.dtst_profile_collect.restype = ctypes.c_int
    L.dtst_status_string.argtypes = [ctypes.c_int]
    L.dtst_status_string.restype = ctypes.c_char_p
    L.dtst_last_error.argtypes = []
    L.dtst_last_error.restype = ctypes.c_char_p
    return L


lib = _load()


def _check(status):
    if status != DTST_OK:
        raise DtstError(status, lib.dtst_last_error().decode())


def make_desc(n_global, n_local, offset, kmax, kt, batch, c_in, c_out) -> Desc:
    d = Desc()
    for i in range(4):
        d.n_global[i] = int(n_global[i])
        d.n_local[i] = int(n_local[i])
        d.offset[i] = int(offset[i])
    for i in range(3):
        d.kmax[i] = int(kmax[i])
    d.kt = int(kt)
    d.batch, d.c_in, d.c_out = int(batch), int(c_in), int(c_out)
    return d


def _desc(d):
    if isinstance(d, Desc):
        return d
    return make_desc(d["n_global"], d["n_local"], d["offset"], d["kmax"], d["kt"], d["batch"], d["c_in"], d["c_out"])


# ---- host-only helpers -----------------------------------------------------
def dtst_desc_validate(desc):
    _check(lib.dtst_desc_validate(ctypes.byref(_desc(desc))))


def dtst_desc_workspace_bytes(desc, flags=0) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.dtst_desc_workspace_bytes_ex(ctypes.byref(_desc(desc)), int(flags), ctypes.byref(n)))
    return n.value


def dtst_basis_host(desc, dim, kind):
    """fp32 basis of one dimension as a complex64 numpy array (K, N_loc)."""
    import numpy as np
    d = _desc(desc)
    if 0 <= dim <= 3:
        k = 2 * d.kmax[dim] if dim < 3 else d.kt
        n = d.n_local[dim]
    else:
        k = n = 1  # the library rejects the request
    buf = np.zeros(max(2 * k * n, 2), dtype=np.float32)
    _check(lib.dtst_basis_host(ctypes.byref(d), int(dim), int(kind),
                               buf.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), buf.size))
    return buf.view(np.complex64).reshape(k, n)


# ---- plans and execute calls (device tensors) ------------------------------
def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def torch_stream():
    """The current torch stream as the integer value of its hipStream_t."""
    import torch
    return torch.cuda.current_stream().cuda_stream


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    return ctypes.c_void_p(torch_stream())


def dtst_plan(desc, flags=0):
    """dtst_plan_ex; flags 0 or a combination of PLAN_SPLIT_SCHEDULE and
    PLAN_UNFUSED_BLOCK."""
    h = ctypes.c_void_p()
    _check(lib.dtst_plan_ex(ctypes.byref(_desc(desc)), int(flags), ctypes.byref(h)))
    return h


def dtst_plan_destroy(plan):
    _check(lib.dtst_plan_destroy(plan))


def dtst_plan_info(plan):
    m = ctypes.c_int64(0)
    ws = ctypes.c_size_t(0)
    _check(lib.dtst_plan_info(plan, ctypes.byref(m), ctypes.byref(ws)))
    return m.value, ws.value


def dtst_plan_block_info(plan):
    """(workspace bytes of dtst_inverse_block, 1 if it runs the fused kernel)."""
    ws = ctypes.c_size_t(0)
    fused = ctypes.c_int(0)
    _check(lib.dtst_plan_block_info(plan, ctypes.byref(ws), ctypes.byref(fused)))
    return ws.value, fused.value


def _wsargs(ws):
    if ws is None:
        return None, 0
    return _ptr(ws), ws.numel() * ws.element_size()


def dtst_forward(plan, x, xhat, accumulate, ws, stream=None):
    p, n = _wsargs(ws)
    _check(lib.dtst_forward(plan, _ptr(x), _ptr(xhat), int(accumulate), p, n, _stream(stream)))


def dtst_forward_noalloc(plan, x, xhat, accumulate, stream=None):
    _check(lib.dtst_forward_noalloc(plan, _ptr(x), _ptr(xhat), int(accumulate), _stream(stream)))


def dtst_mix(plan, xhat, w_shard, yhat, m0, m1, op=0, stream=None):
    _check(lib.dtst_mix(plan, _ptr(xhat), _ptr(w_shard), _ptr(yhat), int(m0), int(m1), int(op), _stream(stream)))


def dtst_inverse(plan, yhat, y, ws, stream=None):
    p, n = _wsargs(ws)
    _check(lib.dtst_inverse(plan, _ptr(yhat), _ptr(y), p, n, _stream(stream)))


def dtst_forward_adj(plan, g_xhat, g_x, ws, stream=None):
    p, n = _wsargs(ws)
    _check(lib.dtst_forward_adj(plan, _ptr(g_xhat), _ptr(g_x), p, n, _stream(stream)))


def dtst_inverse_adj(plan, g_y, g_yhat, accumulate, ws, stream=None):
    p, n = _wsargs(ws)
    _check(lib.dtst_inverse_adj(plan, _ptr(g_y), _ptr(g_yhat), int(accumulate), p, n, _stream(stream)))


def dtst_block_epilogue(plan, x, w_bypass, y, stream=None):
    _check(lib.dtst_block_epilogue(plan, _ptr(x), _ptr(w_bypass), _ptr(y), _stream(stream)))


def dtst_inverse_block(plan, yhat, x, w_bypass, y, ws, stream=None):
    _check(lib.dtst_inverse_block(plan, _ptr(yhat), _ptr(x), _ptr(w_bypass), _ptr(y), *_wsargs(ws),
                                  _stream(stream)))


def dtst_pointwise(x, w, bias, y, act=0, stream=None):
    """y = act(w x + bias) over the points of x (batch, c_in, ...) into y
    (batch, c_out, ...); bias may be None.  Shape checks here, arithmetic in
    the library."""
    import torch
    if x.dim() < 2 or y.dim() != x.dim() or x.shape[0] != y.shape[0] or x.shape[2:] != y.shape[2:]:
        raise ValueError(f"x {tuple(x.shape)} and y {tuple(y.shape)} must be (batch, channels, points...)")
    for t, name in ((x, "x"), (w, "w"), (y, "y")) + (((bias, "bias"),) if bias is not None else ()):
        if t.device.type != "cuda" or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 device tensor")
    B, ci, co = x.shape[0], x.shape[1], y.shape[1]
    if tuple(w.shape) != (co, ci) or (bias is not None and tuple(bias.shape) != (co,)):
        raise ValueError(f"w must be ({co}, {ci}) and bias ({co},)")
    points = x[0, 0].numel()
    _check(lib.dtst_pointwise(_ptr(x), _ptr(w), _ptr(bias), _ptr(y), int(B), int(ci), int(co), int(points), int(act),
                              _stream(stream)))


def dtst_mix_wgrad(plan, xhat, g_yhat, g_w_shard, m0, m1, accumulate, stream=None):
    _check(lib.dtst_mix_wgrad(plan, _ptr(xhat), _ptr(g_yhat), _ptr(g_w_shard), int(m0), int(m1), int(accumulate),
                              _stream(stream)))


def dtst_profile_enable(on=True):
    _check(lib.dtst_profile_enable(1 if on else 0))


def dtst_profile_collect():
    """{kernel role: (launches, total_ms)} since the last collect."""
    cap = 32
    arr = (KernelTime * cap)()
    n = ctypes.c_int(0)
    _check(lib.dtst_profile_collect(arr, cap, ctypes.byref(n)))
    return {arr[i].name.decode(): (arr[i].launches, arr[i].total_ms) for i in range(n.value)}


class Plan:
    """Owns one library plan and a torch-allocated workspace; shape and dtype
    checks on the tensors happen here, the arithmetic in the library."""

    def __init__(self, desc, device="cuda", flags=0):
        import torch
        self.desc = _desc(desc)
        self.handle = dtst_plan(self.desc, flags)
        self.n_modes, self.ws_bytes = dtst_plan_info(self.handle)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=device)
        self.block_ws_bytes, self.block_fused = dtst_plan_block_info(self.handle)
        self.ws_block = None   # allocated by the first inverse_block when larger than ws
        self.device = device
        d = self.desc
        self.K = (2 * d.kmax[0], 2 * d.kmax[1], 2 * d.kmax[2], d.kt)
        self.n_local = tuple(d.n_local)

    def close(self):
        if self.handle is not None:
            dtst_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- shape helpers --
    def spatial_shape(self, channels):
        return (self.desc.batch, channels) + self.n_local

    def spectral_shape(self, channels):
        return (self.desc.batch, channels) + self.K

    def _need(self, t, shape, dtype, name):
        import torch
        if t.device.type != "cuda":
            raise ValueError(f"{name} must be a device tensor")
        if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous():
            raise ValueError(f"{name}: need contiguous {dtype} of shape {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")
        return torch

    def forward(self, x, xhat, accumulate=False, stream=None):
        import torch
        self._need(x, self.spatial_shape(self.desc.c_in), torch.float32, "x")
        self._need(xhat, self.spectral_shape(self.desc.c_in), torch.complex64, "xhat")
        dtst_forward(self.handle, x, xhat, accumulate, self.ws, stream)

    def inverse(self, yhat, y, stream=None):
        import torch
        self._need(yhat, self.spectral_shape(self.desc.c_out), torch.complex64, "yhat")
        self._need(y, self.spatial_shape(self.desc.c_out), torch.float32, "y")
        dtst_inverse(self.handle, yhat, y, self.ws, stream)

    def forward_adj(self, g_xhat, g_x, stream=None):
        import torch
        self._need(g_xhat, self.spectral_shape(self.desc.c_in), torch.complex64, "g_xhat")
        self._need(g_x, self.spatial_shape(self.desc.c_in), torch.float32, "g_x")
        dtst_forward_adj(self.handle, g_xhat, g_x, self.ws, stream)

    def inverse_adj(self, g_y, g_yhat, accumulate=False, stream=None):
        import torch
        self._need(g_y, self.spatial_shape(self.desc.c_out), torch.float32, "g_y")
        self._need(g_yhat, self.spectral_shape(self.desc.c_out), torch.complex64, "g_yhat")
        dtst_inverse_adj(self.handle, g_y, g_yhat, accumulate, self.ws, stream)

    def mix(self, xhat, w, yhat, m0=0, m1=None, op=0, stream=None):
        import torch
        m1 = self.n_modes if m1 is None else m1
        cin, cout = (self.desc.c_in, self.desc.c_out) if op == 0 else (self.desc.c_out, self.desc.c_in)
        self._need(xhat, self.spectral_shape(cin), torch.complex64, "xhat")
        self._need(yhat, self.spectral_shape(cout), torch.complex64, "yhat")
        self._need(w, (m1 - m0, self.desc.c_in, self.desc.c_out), torch.complex64, "w")
        dtst_mix(self.handle, xhat, w, yhat, m0, m1, op, stream)

    def wgrad(self, xhat, g_yhat, g_w, m0=0, m1=None, accumulate=False, stream=None):
        import torch
        m1 = self.n_modes if m1 is None else m1
        self._need(xhat, self.spectral_shape(self.desc.c_in), torch.complex64, "xhat")
        self._need(g_yhat, self.spectral_shape(self.desc.c_out), torch.complex64, "g_yhat")
        self._need(g_w, (m1 - m0, self.desc.c_in, self.desc.c_out), torch.complex64, "g_w")
        dtst_mix_wgrad(self.handle, xhat, g_yhat, g_w, m0, m1, accumulate, stream)

    def inverse_block(self, yhat, x, w_bypass, y, stream=None):
        """y = GELU(w_bypass x + inverse(yhat)) (the block's last step)."""
        import torch
        self._need(yhat, self.spectral_shape(self.desc.c_out), torch.complex64, "yhat")
        self._need(x, self.spatial_shape(self.desc.c_in), torch.float32, "x")
        self._need(w_bypass, (self.desc.c_out, self.desc.c_in), torch.float32, "w_bypass")
        self._need(y, self.spatial_shape(self.desc.c_out), torch.float32, "y")
        ws = self.ws
        if self.block_ws_bytes > self.ws_bytes:
            if self.ws_block is None:
                self.ws_block = torch.empty(self.block_ws_bytes, dtype=torch.uint8, device=self.device)
            ws = self.ws_block
        dtst_inverse_block(self.handle, yhat, x, w_bypass, y, ws, stream)

    def block_epilogue(self, x, w_bypass, y, stream=None):
        """y <- GELU(w_bypass x + y) in place (the block's bypass and activation)."""
        import torch
        self._need(x, self.spatial_shape(self.desc.c_in), torch.float32, "x")
        self._need(w_bypass, (self.desc.c_out, self.desc.c_in), torch.float32, "w_bypass")
        self._need(y, self.spatial_shape(self.desc.c_out), torch.float32, "y")
        dtst_block_epilogue(self.handle, x, w_bypass, y, stream)
