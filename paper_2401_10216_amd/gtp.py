"""Thin ctypes binding of libgtp.so (the C ABI in include/gtp.h).

Only argument marshalling happens here: every step of the Gaunt tensor
product runs in the library's HIP kernels.  Tensors are torch CUDA (HIP)
tensors; the current torch stream is passed to the library.  If the library
is not built the import of any entry point raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libgtp.so")

GTP_OK, GTP_ERR_INVALID_ARG, GTP_ERR_UNSUPPORTED, GTP_ERR_NO_DEVICE, GTP_ERR_HIP, GTP_ERR_ALLOC = range(6)
GTP_F32, GTP_BF16 = 0, 1
GTP_CONV_AUTO, GTP_CONV_DIRECT, GTP_CONV_FFT, GTP_CONV_DFT = 0, 1, 2, 3
GTP_PLAN_HOST_ONLY = 16
GTP_FORCE_GENERIC = 32  # internal: use the workgroup-per-product kernel
GTP_SELF_STEPWISE, GTP_SELF_FUSED = 0, 1

_lib = None
_lock = threading.Lock()


class GTPError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


_STATUS = {0: "GTP_OK", 1: "GTP_ERR_INVALID_ARG", 2: "GTP_ERR_UNSUPPORTED", 3: "GTP_ERR_NO_DEVICE",
           4: "GTP_ERR_HIP", 5: "GTP_ERR_ALLOC"}

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int
_U = ctypes.c_uint
_DP = ctypes.POINTER(ctypes.c_double)

_SIGS = {
    "gtp_plan_create": (_I, [ctypes.POINTER(_P), _I, _I, _I, _U]),
    "gtp_plan_destroy": (_I, [_P]),
    "gtp_full": (_I, [_P, _P, _P, _I, _I64, _I64, _P, _P]),
    "gtp_full_backward": (_I, [_P, _P, _P, _I, _P, _I64, _I64, _P, _P, _P]),
    "gtp_full_weighted": (_I, [_P, _P, _P, _I, _P, _P, _P, _I, _I64, _I64, _P, _P]),
    "gtp_full_weighted_backward": (_I, [_P, _P, _P, _I, _P, _P, _P, _I, _P, _I64, _I64, _P, _P, _P, _P, _P, _P]),
    "gtp_conv_escn": (_I, [_P, _P, _I, _P, _P, _I64, _I64, _P, _P]),
    "gtp_conv_escn_noalloc": (_I, [_P, _P, _I, _P, _P, _I64, _I64, _P, _P]),
    "gtp_channel_mix": (_I, [_P, _P, _P, _I, _P, _I64, _I64, _I64, _I64, _P, _P]),
    "gtp_sh2fourier": (_I, [_P, _I, _P, _I, _I64, _P, _P]),
    "gtp_fourier_conv": (_I, [_P, _P, _P, _I64, _P, _P]),
    "gtp_fourier2sh": (_I, [_P, _P, _I64, _P, _P]),
    "gtp_selfproduct": (_I, [_I, _I, _I, _U, _P, _I, _I64, _I64, _P, _P]),
    "gtp_sh_filter": (_I, [_I, _P, _P, _I64, _I64, _P, _P]),
    "gtp_stream_probe": (_I, [_I, _P, _P, _I64, _P]),
    "gtp_compute_probe": (_I, [_I, _I64, _P, _DP, _P]),
    "gtp_grid_floats": (_I64, [_P, _I]),
    "gtp_plan_info": (_I, [_P, ctypes.POINTER(_I64)]),
    "gtp_plan_table": (_I, [_P, _I, _DP, ctypes.POINTER(_I64)]),
    "gtp_debug_host_pipeline": (_I, [_P, _DP, _DP, _I64, _DP]),
    "gtp_status_str": (ctypes.c_char_p, [_I]),
    "gtp_last_error": (ctypes.c_char_p, []),
}


def _load(path: str):
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2401_10216_amd.build`")
    L = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


def lib():
    """Load libgtp.so once (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            _lib = _load(LIB_PATH)
    return _lib


class use_library:
    """Context in which the entry points (and the plans created there) use
    another build of the library, e.g. the poisoned-LDS debug build
    (libgtp_poison.so).  A plan keeps the library it was created with."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        with _lock:
            self.saved = _lib
            _lib = _load(self.path)
        return _lib

    def __exit__(self, *exc):
        global _lib
        with _lock:
            _lib = self.saved
        return False


def _check(status: int, L=None):
    if status != GTP_OK:
        raise GTPError(status, (L or lib()).gtp_last_error().decode())


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return GTP_F32
    if t.dtype == torch.bfloat16:
        return GTP_BF16
    raise TypeError(f"unsupported input dtype {t.dtype} (float32 or bfloat16)")


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _want(t, name, shape, dtypes, device=None):
    """Validate a caller-supplied tensor before anything reaches the library:
    exact shape, one of the allowed dtypes, contiguous, on the device of the
    other operands.  Raises TypeError (dtype) or ValueError (everything else)
    and returns the tensor's device pointer."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}; expected " + " or ".join(str(d) for d in dtypes))
    if tuple(t.shape) != tuple(int(v) for v in shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}; expected {tuple(int(v) for v in shape)}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}; the other operands are on {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _on_gpu(t, name):
    """Last check before a call: the operands (all on t's device) are device tensors."""
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")


def _f32():
    import torch
    return (torch.float32,)


def _inputs():
    import torch
    return (torch.float32, torch.bfloat16)


def nsh(L: int) -> int:
    return (L + 1) * (L + 1)


class Plan:
    """gtp_plan_create / gtp_plan_destroy."""

    def __init__(self, L1: int, L2: int, Lout: int, flags: int = 0):
        self.L1, self.L2, self.Lout, self.flags = L1, L2, Lout, flags
        h = _P()
        self.lib = lib()
        _check(self.lib.gtp_plan_create(ctypes.byref(h), L1, L2, Lout, flags), self.lib)
        self.handle = h

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            self.lib.gtp_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> dict:
        out = (_I64 * 8)()
        _check(self.lib.gtp_plan_info(self.handle, out), self.lib)
        keys = ["L1", "L2", "Lout", "U", "Le", "NT", "NP", "conv"]
        return dict(zip(keys, [int(v) for v in out]))

    def table(self, which: int):
        import numpy as np
        cnt = _I64(0)
        _check(self.lib.gtp_plan_table(self.handle, which, None, ctypes.byref(cnt)), self.lib)
        buf = np.zeros(cnt.value, dtype=np.float64)
        _check(self.lib.gtp_plan_table(self.handle, which, buf.ctypes.data_as(_DP), ctypes.byref(cnt)), self.lib)
        return buf

    def grid_floats(self, which: int) -> int:
        return int(self.lib.gtp_grid_floats(self.handle, which))


def gtp_full(plan: Plan, x1, x2, y=None, stream=None):
    """y[B,C,(Lout+1)^2] = Gaunt tensor product of x1[B,C,(L1+1)^2] and x2[B,C,(L2+1)^2]."""
    import torch
    if x1.dtype != x2.dtype:
        raise TypeError("x1 and x2 must have the same dtype")
    if x1.dim() != 3 or x2.dim() != 3 or x1.shape[:2] != x2.shape[:2]:
        raise ValueError("x1, x2 must be [B, C, K] with equal B, C")
    if x1.shape[2] != nsh(plan.L1) or x2.shape[2] != nsh(plan.L2):
        raise ValueError("coefficient dimension does not match the plan")
    B, C = int(x1.shape[0]), int(x1.shape[1])
    code = _dtype_code(x1)
    p1 = _want(x1, "x1", x1.shape, _inputs())
    p2 = _want(x2, "x2", x2.shape, _inputs(), x1.device)
    if y is None:
        y = torch.empty((B, C, nsh(plan.Lout)), dtype=torch.float32, device=x1.device)
    py = _want(y, "y", (B, C, nsh(plan.Lout)), _f32(), x1.device)
    _on_gpu(x1, "x1")
    _check(plan.lib.gtp_full(plan.handle, p1, p2, code, B, C, py, _stream(stream)), plan.lib)
    return y


def gtp_channel_mix(plan: Plan, x1, x2, W, y=None, stream=None):
    """y[B,Co,(Lout+1)^2] = sum_{c1,c2} W[co,c1,c2] GTP(x1[:,c1], x2[:,c2]); W float32 [Co, C1, C2]."""
    import torch
    if x1.dtype != x2.dtype:
        raise TypeError("x1 and x2 must have the same dtype")
    if x1.dim() != 3 or x2.dim() != 3 or x1.shape[0] != x2.shape[0]:
        raise ValueError("x1 [B, C1, K1] and x2 [B, C2, K2] with equal B")
    if x1.shape[2] != nsh(plan.L1) or x2.shape[2] != nsh(plan.L2):
        raise ValueError("coefficient dimension does not match the plan")
    B, C1, C2 = int(x1.shape[0]), int(x1.shape[1]), int(x2.shape[1])
    if W.dim() != 3 or tuple(W.shape[1:]) != (C1, C2) or W.dtype != torch.float32:
        raise ValueError("W must be float32 [Co, C1, C2]")
    Co = int(W.shape[0])
    code = _dtype_code(x1)
    p1 = _want(x1, "x1", x1.shape, _inputs())
    p2 = _want(x2, "x2", x2.shape, _inputs(), x1.device)
    pw = _want(W, "W", (Co, C1, C2), _f32(), x1.device)
    if y is None:
        y = torch.empty((B, Co, nsh(plan.Lout)), dtype=torch.float32, device=x1.device)
    py = _want(y, "y", (B, Co, nsh(plan.Lout)), _f32(), x1.device)
    _on_gpu(x1, "x1")
    _check(plan.lib.gtp_channel_mix(plan.handle, p1, p2, code, pw, B, C1, C2, Co, py, _stream(stream)), plan.lib)
    return y


def gtp_conv_escn(plan: Plan, x, r, h, y=None, stream=None, noalloc: bool = False):
    """y[B,C,(Lout+1)^2] = GTP(x, h[b,c,l] Y_l(r_b / |r_b|)) in the edge's rotated frame; r [B, 3], h [B, C, L2+1] fp32.
    noalloc=True calls gtp_conv_escn_noalloc (static device scratch, no allocation by the library; y must then be
    given for no allocation to happen at all)."""
    import torch
    if x.dim() != 3 or x.shape[2] != nsh(plan.L1):
        raise ValueError("x must be [B, C, (L1+1)^2]")
    B, C = int(x.shape[0]), int(x.shape[1])
    if tuple(r.shape) != (B, 3) or r.dtype != torch.float32:
        raise ValueError("r must be float32 [B, 3]")
    if tuple(h.shape) != (B, C, plan.L2 + 1) or h.dtype != torch.float32:
        raise ValueError("h must be float32 [B, C, L2+1]")
    code = _dtype_code(x)
    px = _want(x, "x", x.shape, _inputs())
    pr = _want(r, "r", (B, 3), _f32(), x.device)
    ph = _want(h, "h", (B, C, plan.L2 + 1), _f32(), x.device)
    if y is None:
        y = torch.empty((B, C, nsh(plan.Lout)), dtype=torch.float32, device=x.device)
    py = _want(y, "y", (B, C, nsh(plan.Lout)), _f32(), x.device)
    _on_gpu(x, "x")
    fn = plan.lib.gtp_conv_escn_noalloc if noalloc else plan.lib.gtp_conv_escn
    _check(fn(plan.handle, px, code, pr, ph, B, C, py, _stream(stream)), plan.lib)
    return y


def gtp_full_weighted(plan: Plan, x1, x2, w1=None, w2=None, wout=None, per_channel: bool = False, y=None,
                      stream=None):
    """y = wout * GTP(w1 * x1, w2 * x2) with per-degree weights w1[R, L1+1], w2[R, L2+1], wout[R, Lout+1]
    (fp32 device tensors or None = ones; R = C if per_channel else 1)."""
    import torch
    if x1.dtype != x2.dtype:
        raise TypeError("x1 and x2 must have the same dtype")
    if x1.dim() != 3 or x2.dim() != 3 or x1.shape[:2] != x2.shape[:2]:
        raise ValueError("x1, x2 must be [B, C, K] with equal B, C")
    if x1.shape[2] != nsh(plan.L1) or x2.shape[2] != nsh(plan.L2):
        raise ValueError("coefficient dimension does not match the plan")
    B, C = int(x1.shape[0]), int(x1.shape[1])
    R = C if per_channel else 1
    ptrs = []
    for w, L, name in ((w1, plan.L1, "w1"), (w2, plan.L2, "w2"), (wout, plan.Lout, "wout")):
        if w is None:
            ptrs.append(ctypes.c_void_p(None))
            continue
        ptrs.append(_want(w, name, (R, L + 1), _f32(), x1.device))
    code = _dtype_code(x1)
    p1 = _want(x1, "x1", x1.shape, _inputs())
    p2 = _want(x2, "x2", x2.shape, _inputs(), x1.device)
    if y is None:
        y = torch.empty((B, C, nsh(plan.Lout)), dtype=torch.float32, device=x1.device)
    py = _want(y, "y", (B, C, nsh(plan.Lout)), _f32(), x1.device)
    _on_gpu(x1, "x1")
    _check(plan.lib.gtp_full_weighted(plan.handle, p1, p2, code, *ptrs, 1 if per_channel else 0, B, C, py,
                                      _stream(stream)), plan.lib)
    return y


def gtp_full_weighted_backward(plan: Plan, x1, x2, dy, w1=None, w2=None, wout=None, per_channel: bool = False,
                               need=("dx1", "dx2", "dw1", "dw2", "dwout"), stream=None):
    """Gradients of <dy, gtp_full_weighted(x1, x2, w1, w2, wout)>: a dict with the requested keys among dx1, dx2
    ([B, C, K] fp32) and dw1, dw2, dwout ([R, L+1] fp32, R = C if per_channel else 1)."""
    import torch
    if x1.dtype != x2.dtype:
        raise TypeError("x1 and x2 must have the same dtype")
    if x1.dim() != 3 or x2.dim() != 3 or x1.shape[:2] != x2.shape[:2]:
        raise ValueError("x1, x2 must be [B, C, K] with equal B, C")
    if x1.shape[2] != nsh(plan.L1) or x2.shape[2] != nsh(plan.L2):
        raise ValueError("coefficient dimension does not match the plan")
    unknown = set(need) - {"dx1", "dx2", "dw1", "dw2", "dwout"}
    if unknown:
        raise ValueError(f"unknown gradients {sorted(unknown)}")
    B, C = int(x1.shape[0]), int(x1.shape[1])
    R = C if per_channel else 1
    code = _dtype_code(x1)
    px1 = _want(x1, "x1", x1.shape, _inputs())
    px2 = _want(x2, "x2", x2.shape, _inputs(), x1.device)
    pdy = _want(dy, "dy", (B, C, nsh(plan.Lout)), _f32(), x1.device)
    ws = []
    for w, L, name in ((w1, plan.L1, "w1"), (w2, plan.L2, "w2"), (wout, plan.Lout, "wout")):
        ws.append(ctypes.c_void_p(None) if w is None else _want(w, name, (R, L + 1), _f32(), x1.device))
    shapes = {"dx1": (B, C, nsh(plan.L1)), "dx2": (B, C, nsh(plan.L2)), "dw1": (R, plan.L1 + 1),
              "dw2": (R, plan.L2 + 1), "dwout": (R, plan.Lout + 1)}
    out = {k: torch.empty(shapes[k], dtype=torch.float32, device=x1.device) for k in need}
    ptr = {k: (ctypes.c_void_p(out[k].data_ptr()) if k in out else ctypes.c_void_p(None)) for k in shapes}
    _on_gpu(x1, "x1")
    _check(plan.lib.gtp_full_weighted_backward(plan.handle, px1, px2, code, *ws, 1 if per_channel else 0, pdy, B, C,
                                               ptr["dx1"], ptr["dx2"], ptr["dw1"], ptr["dw2"], ptr["dwout"],
                                               _stream(stream)), plan.lib)
    return out


def gtp_full_backward(plan: Plan, x1, x2, dy, need_dx1: bool = True, need_dx2: bool = True, dx1=None, dx2=None,
                      stream=None):
    """(dx1, dx2): gradients of <dy, gtp_full(x1, x2)> in x1 and x2 (fp32; None when not requested)."""
    import torch
    if x1.dtype != x2.dtype:
        raise TypeError("x1 and x2 must have the same dtype")
    if x1.dim() != 3 or x2.dim() != 3 or dy.dim() != 3 or x1.shape[:2] != x2.shape[:2] or dy.shape[:2] != x1.shape[:2]:
        raise ValueError("x1, x2, dy must be [B, C, K] with equal B, C")
    if x1.shape[2] != nsh(plan.L1) or x2.shape[2] != nsh(plan.L2) or dy.shape[2] != nsh(plan.Lout):
        raise ValueError("coefficient dimension does not match the plan")
    if dy.dtype != torch.float32:
        raise TypeError("dy must be float32")
    B, C = int(x1.shape[0]), int(x1.shape[1])
    code = _dtype_code(x1)
    px1 = _want(x1, "x1", x1.shape, _inputs())
    px2 = _want(x2, "x2", x2.shape, _inputs(), x1.device)
    pdy = _want(dy, "dy", (B, C, nsh(plan.Lout)), _f32(), x1.device)
    if need_dx1 and dx1 is None:
        dx1 = torch.empty((B, C, nsh(plan.L1)), dtype=torch.float32, device=x1.device)
    if need_dx2 and dx2 is None:
        dx2 = torch.empty((B, C, nsh(plan.L2)), dtype=torch.float32, device=x1.device)
    p1 = _want(dx1, "dx1", (B, C, nsh(plan.L1)), _f32(), x1.device) if need_dx1 else ctypes.c_void_p(None)
    p2 = _want(dx2, "dx2", (B, C, nsh(plan.L2)), _f32(), x1.device) if need_dx2 else ctypes.c_void_p(None)
    _on_gpu(x1, "x1")
    _check(plan.lib.gtp_full_backward(plan.handle, px1, px2, code, pdy, B, C, p1, p2, _stream(stream)), plan.lib)
    return (dx1 if need_dx1 else None), (dx2 if need_dx2 else None)


def gtp_sh2fourier(plan: Plan, which: int, x, grid=None, stream=None):
    """Complex grids [n, 2L+1, 2L+1] (as torch.complex64) of x[n, (L+1)^2]."""
    import torch
    if which not in (1, 2):
        raise ValueError("which must be 1 or 2")
    L = plan.L1 if which == 1 else plan.L2
    if x.dim() != 2:
        raise ValueError("x must be [n, (L+1)^2]")
    n = int(x.shape[0])
    code = _dtype_code(x)
    px = _want(x, "x", (n, nsh(L)), _inputs())
    if grid is None:
        grid = torch.empty((n, 2 * L + 1, 2 * L + 1), dtype=torch.complex64, device=x.device)
    pg = _want(grid, "grid", (n, 2 * L + 1, 2 * L + 1), (torch.complex64,), x.device)
    _on_gpu(x, "x")
    _check(plan.lib.gtp_sh2fourier(plan.handle, which, px, code, n, pg, _stream(stream)), plan.lib)
    return grid


def gtp_fourier_conv(plan: Plan, g1, g2, g3=None, stream=None):
    import torch
    if g1.dim() != 3:
        raise ValueError("g1 must be [n, 2 L1 + 1, 2 L1 + 1]")
    n = int(g1.shape[0])
    D1, D2, D3 = 2 * plan.L1 + 1, 2 * plan.L2 + 1, 2 * (plan.L1 + plan.L2) + 1
    c64 = (torch.complex64,)
    p1 = _want(g1, "g1", (n, D1, D1), c64)
    p2 = _want(g2, "g2", (n, D2, D2), c64, g1.device)
    if g3 is None:
        g3 = torch.empty((n, D3, D3), dtype=torch.complex64, device=g1.device)
    p3 = _want(g3, "g3", (n, D3, D3), c64, g1.device)
    _on_gpu(g1, "g1")
    _check(plan.lib.gtp_fourier_conv(plan.handle, p1, p2, n, p3, _stream(stream)), plan.lib)
    return g3


def gtp_fourier2sh(plan: Plan, g3, y=None, stream=None):
    import torch
    if g3.dim() != 3:
        raise ValueError("g3 must be [n, 2U + 1, 2U + 1]")
    n = int(g3.shape[0])
    D3 = 2 * (plan.L1 + plan.L2) + 1
    p3 = _want(g3, "g3", (n, D3, D3), (torch.complex64,))
    if y is None:
        y = torch.empty((n, nsh(plan.Lout)), dtype=torch.float32, device=g3.device)
    py = _want(y, "y", (n, nsh(plan.Lout)), _f32(), g3.device)
    _on_gpu(g3, "g3")
    _check(plan.lib.gtp_fourier2sh(plan.handle, p3, n, py, _stream(stream)), plan.lib)
    return y


def gtp_selfproduct(x, L: int, nu: int, Lout: int, mode: int = GTP_SELF_STEPWISE, y=None, stream=None):
    import torch
    if x.dim() != 3 or x.shape[2] != nsh(L):
        raise ValueError("x must be [B, C, (L+1)^2]")
    B, C = int(x.shape[0]), int(x.shape[1])
    code = _dtype_code(x)
    px = _want(x, "x", x.shape, _inputs())
    if y is None:
        y = torch.empty((B, C, nsh(Lout)), dtype=torch.float32, device=x.device)
    py = _want(y, "y", (B, C, nsh(Lout)), _f32(), x.device)
    _on_gpu(x, "x")
    _check(lib().gtp_selfproduct(L, nu, Lout, mode, px, code, B, C, py, _stream(stream)))
    return y


def gtp_sh_filter(L: int, r, h=None, out=None, stream=None):
    """out[B,C,(L+1)^2] = h[B,C,L+1] * Y(r_b); h=None gives Y(r) with C = 1."""
    import torch
    if r.dim() != 2:
        raise ValueError("r must be [B, 3]")
    B = int(r.shape[0])
    pr = _want(r, "r", (B, 3), _f32())
    if h is not None and h.dim() != 3:
        raise ValueError("h must be [B, C, L+1]")
    C = 1 if h is None else int(h.shape[1])
    hp = ctypes.c_void_p(None) if h is None else _want(h, "h", (B, C, L + 1), _f32(), r.device)
    if out is None:
        out = torch.empty((B, C, nsh(L)), dtype=torch.float32, device=r.device)
    po = _want(out, "out", (B, C, nsh(L)), _f32(), r.device)
    _on_gpu(r, "r")
    _check(lib().gtp_sh_filter(L, pr, hp, B, C, po, _stream(stream)))
    return out


def gtp_stream_probe(mode: int, src, dst, stream=None):
    """HBM streaming probe: mode 0 reads src (dst: >= 1 float), 1 writes dst, 2 copies src to dst,
    3 writes the sum of src's two halves to dst (>= half of src)."""
    nbytes = (dst if mode == 1 else src).numel() * (dst if mode == 1 else src).element_size()
    if mode == 2 and dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst smaller than src")
    if mode == 3 and dst.numel() * dst.element_size() < nbytes // 2:
        raise ValueError("dst smaller than half of src")
    sp = ctypes.c_void_p(None) if mode == 1 else ctypes.c_void_p(src.data_ptr())
    _check(lib().gtp_stream_probe(mode, sp, ctypes.c_void_p(dst.data_ptr()), nbytes, _stream(stream)))


def gtp_compute_probe(mode: int, iters: int, sink, stream=None) -> float:
    """fp32 compute probe: mode 0 VALU FMA chains, 1 MFMA chains; returns the flops launched."""
    ps = _want(sink, "sink", (1,), _f32())
    fl = ctypes.c_double(0.0)
    _check(lib().gtp_compute_probe(mode, iters, ps, ctypes.byref(fl), _stream(stream)))
    return fl.value


def gtp_debug_host_pipeline(plan: Plan, x1, x2):
    """fp64 host evaluation of the plan's sampled pipeline (table check only)."""
    import numpy as np
    a = np.ascontiguousarray(x1, dtype=np.float64).reshape(-1, nsh(plan.L1))
    b = np.ascontiguousarray(x2, dtype=np.float64).reshape(-1, nsh(plan.L2))
    y = np.zeros((a.shape[0], nsh(plan.Lout)), dtype=np.float64)
    _check(plan.lib.gtp_debug_host_pipeline(plan.handle, a.ctypes.data_as(_DP), b.ctypes.data_as(_DP), a.shape[0],
                                            y.ctypes.data_as(_DP)), plan.lib)
    return y
