"""ctypes binding of libmiconv.so (include/miconv.h).

Argument marshalling only: every pass runs in the library's HIP kernels.
Tensors are torch tensors used as device memory (float32, contiguous, on the
current HIP device); kernels are enqueued on torch's current stream.  If the
library is not built, every call raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(PKG, "libmiconv.so")

OK = 0
STATUS = {
    0: "MICONV_OK", -1: "MICONV_ERR_SHAPE", -2: "MICONV_ERR_NULL",
    -3: "MICONV_ERR_WORKSPACE", -4: "MICONV_ERR_ALIAS", -5: "MICONV_ERR_ALIGN",
    -6: "MICONV_ERR_DEVICE", -7: "MICONV_ERR_LAUNCH", -8: "MICONV_ERR_PASS",
    -9: "MICONV_ERR_PLAN", -10: "MICONV_ERR_MODE", -11: "MICONV_ERR_SCRATCH",
}
POOL_MODES = {"max": 0, "avg": 1}
PASS_FWD, PASS_BWD_DATA, PASS_BWD_WEIGHT = 0, 1, 2

_lib = None
_I = ctypes.c_int
_P = ctypes.c_void_p
_Z = ctypes.c_size_t


class MiconvError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        msg = lib().conv_error_string(status).decode()
        super().__init__(f"{what}: {STATUS.get(status, status)} ({msg})")


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise RuntimeError(f"{LIBRARY} is not built; run paper_1903_06934_amd.build.build()")
    # torch first: its HIP runtime (soname libamdhip64.so.7) then also serves
    # the library's dependency.  Loaded the other way round, torch would load
    # a second runtime of its own next to it.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIBRARY)
    geo = [_I] * 10
    L.conv_output_size.argtypes = [_I] * 6 + [ctypes.POINTER(_I), ctypes.POINTER(_I)]
    L.conv_output_size.restype = _I
    L.conv_workspace_size.argtypes = [_I] + geo
    L.conv_workspace_size.restype = _Z
    L.conv_fwd.argtypes = geo + [_P, _P, _P, _P, _P, _Z, _P]
    L.conv_fwd.restype = _I
    L.conv_bwd_data.argtypes = geo + [_P, _P, _P, _P, _Z, _P]
    L.conv_bwd_data.restype = _I
    L.conv_bwd_weight.argtypes = geo + [_P, _P, _P, _P, _P, _Z, _P]
    L.conv_bwd_weight.restype = _I
    L.conv_bwd_weight_noalloc.argtypes = geo + [_P, _P, _P, _P, _P]
    L.conv_bwd_weight_noalloc.restype = _I
    L.conv_set_timing_events.argtypes = [_P, _P]
    L.conv_set_timing_events.restype = _I
    L.conv_error_string.argtypes = [_I]
    L.conv_error_string.restype = ctypes.c_char_p
    L.conv_plan_count.argtypes = [_I] + geo
    L.conv_plan_count.restype = _I
    L.conv_plan_get.argtypes = [_I] + geo
    L.conv_plan_get.restype = _I
    L.conv_plan_set.argtypes = [_I] + geo + [_I]
    L.conv_plan_set.restype = _I
    L.conv_plan_clear.argtypes = []
    L.conv_plan_clear.restype = _I
    L.conv_plan_name.argtypes = [_I] + geo + [_I, ctypes.c_char_p, _Z]
    L.conv_plan_name.restype = _I
    L.conv_plan_workspace_size.argtypes = [_I] + geo + [_I]
    L.conv_plan_workspace_size.restype = _Z
    L.conv_tune.argtypes = [_I] + geo + [_P, _P, _P, _P, _P, _P, _Z, _I, _P,
                                         ctypes.POINTER(_I)]
    L.conv_tune.restype = _I
    L.pool_output_size.argtypes = [_I] * 6 + [ctypes.POINTER(_I), ctypes.POINTER(_I)]
    L.pool_output_size.restype = _I
    L.pool_fwd.argtypes = [_I] * 9 + [_P, _P, _P, _P]
    L.pool_fwd.restype = _I
    L.pool_bwd.argtypes = [_I] * 9 + [_P, _P, _P, _P]
    L.pool_bwd.restype = _I
    _lib = L
    return L


def output_size(H, W, R, S, stride, pad):
    P, Q = _I(), _I()
    st = lib().conv_output_size(H, W, R, S, stride, pad, ctypes.byref(P), ctypes.byref(Q))
    if st != OK:
        raise MiconvError(st, "conv_output_size")
    return P.value, Q.value


def workspace_size(pass_id, shape):
    return int(lib().conv_workspace_size(pass_id, *[int(v) for v in shape]))


def _ptr(t):
    return None if t is None else t.data_ptr()


def _check(t, name):
    import torch
    if t.dtype != torch.float32 or not t.is_contiguous() or t.device.type != "cuda":
        raise ValueError(f"{name} must be a contiguous float32 device tensor")


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def _workspace(nbytes, device):
    import torch
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _call(fn, name, *args):
    st = fn(*args)
    if st != OK:
        raise MiconvError(st, name)


def conv_fwd(x, w, b=None, stride=1, pad=0, group=1, y=None, ws=None):
    """y[N,K,P,Q] = b + w (*) x.  x [N,C,H,W], w [K,C/G,R,S], b [K] or None."""
    import torch
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    shape = (N, C, H, W, K, R, S, stride, pad, group)
    P, Q = output_size(H, W, R, S, stride, pad)
    for t, n in ((x, "x"), (w, "w")):
        _check(t, n)
    if b is not None:
        _check(b, "b")
    if y is None:
        y = torch.empty((N, K, P, Q), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = _workspace(workspace_size(PASS_FWD, shape), x.device)
    _call(lib().conv_fwd, "conv_fwd", *shape, _ptr(x), _ptr(w), _ptr(b), _ptr(y), _ptr(ws),
          0 if ws is None else ws.numel() * ws.element_size(), _stream())
    return y


def conv_bwd_data(dy, w, input_hw, stride=1, pad=0, group=1, dx=None, ws=None):
    """dx[N,C,H,W] from dy [N,K,P,Q] and w [K,C/G,R,S]; input_hw = (H, W)."""
    import torch
    N, K, _, _ = dy.shape
    _, Cg, R, S = w.shape
    H, W = input_hw
    C = Cg * group
    shape = (N, C, H, W, K, R, S, stride, pad, group)
    for t, n in ((dy, "dy"), (w, "w")):
        _check(t, n)
    if dx is None:
        dx = torch.empty((N, C, H, W), dtype=torch.float32, device=dy.device)
    if ws is None:
        ws = _workspace(workspace_size(PASS_BWD_DATA, shape), dy.device)
    _call(lib().conv_bwd_data, "conv_bwd_data", *shape, _ptr(dy), _ptr(w), _ptr(dx), _ptr(ws),
          0 if ws is None else ws.numel() * ws.element_size(), _stream())
    return dx


def conv_bwd_weight(x, dy, filter_rs, stride=1, pad=0, group=1, with_bias=True,
                    dw=None, db=None, ws=None):
    """(dw [K,C/G,R,S], db [K] or None) from x [N,C,H,W] and dy [N,K,P,Q]."""
    import torch
    N, C, H, W = x.shape
    K = dy.shape[1]
    R, S = filter_rs
    shape = (N, C, H, W, K, R, S, stride, pad, group)
    for t, n in ((x, "x"), (dy, "dy")):
        _check(t, n)
    if dw is None:
        dw = torch.empty((K, C // group, R, S), dtype=torch.float32, device=x.device)
    if with_bias and db is None:
        db = torch.empty((K,), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = _workspace(workspace_size(PASS_BWD_WEIGHT, shape), x.device)
    _call(lib().conv_bwd_weight, "conv_bwd_weight", *shape, _ptr(x), _ptr(dy), _ptr(dw),
          _ptr(db), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _stream())
    return dw, db


# ---------------------------------------------------------------- plans
def _shape(shape):
    return [int(v) for v in shape]


def plan_count(pass_id, shape):
    n = lib().conv_plan_count(pass_id, *_shape(shape))
    if n < 0:
        raise MiconvError(n, "conv_plan_count")
    return n


def plan_get(pass_id, shape):
    i = lib().conv_plan_get(pass_id, *_shape(shape))
    if i < 0:
        raise MiconvError(i, "conv_plan_get")
    return i


def plan_set(pass_id, shape, index):
    _call(lib().conv_plan_set, "conv_plan_set", pass_id, *_shape(shape), int(index))


def plan_clear():
    _call(lib().conv_plan_clear, "conv_plan_clear")


def plan_name(pass_id, shape, index):
    buf = ctypes.create_string_buffer(256)
    _call(lib().conv_plan_name, "conv_plan_name", pass_id, *_shape(shape), int(index), buf,
          len(buf))
    return buf.value.decode()


def plan_workspace_size(pass_id, shape, index):
    return int(lib().conv_plan_workspace_size(pass_id, *_shape(shape), int(index)))


def conv_tune(pass_id, shape, in0, in1, in2, out0, out1, ws, reps=3):
    """Time the candidate plans of one pass on these tensors (see conv_tune in
    miconv.h for which tensor is which) and keep the fastest; returns its index."""
    chosen = _I(-1)
    _call(lib().conv_tune, "conv_tune", pass_id, *_shape(shape), _ptr(in0), _ptr(in1),
          _ptr(in2), _ptr(out0), _ptr(out1), _ptr(ws),
          0 if ws is None else ws.numel() * ws.element_size(), int(reps), _stream(),
          ctypes.byref(chosen))
    return chosen.value


# ---------------------------------------------------------------- pooling
def pool_output_size(H, W, R, S, stride, pad):
    P, Q = _I(), _I()
    st = lib().pool_output_size(H, W, R, S, stride, pad, ctypes.byref(P), ctypes.byref(Q))
    if st != OK:
        raise MiconvError(st, "pool_output_size")
    return P.value, Q.value


def pool_fwd(x, window, stride, pad=0, mode="max", y=None, mask=None):
    """(y [N,C,P,Q], mask [N,C,P,Q] int32 for max, else None) from x [N,C,H,W];
    window = (R, S)."""
    import torch
    N, C, H, W = x.shape
    R, S = window
    _check(x, "x")
    P, Q = pool_output_size(H, W, R, S, stride, pad)
    if y is None:
        y = torch.empty((N, C, P, Q), dtype=torch.float32, device=x.device)
    if mode == "max" and mask is None:
        mask = torch.empty((N, C, P, Q), dtype=torch.int32, device=x.device)
    _call(lib().pool_fwd, "pool_fwd", POOL_MODES[mode], N, C, H, W, R, S, stride, pad,
          _ptr(x), _ptr(y), _ptr(mask) if mode == "max" else None, _stream())
    return y, (mask if mode == "max" else None)


def pool_bwd(dy, input_hw, window, stride, pad=0, mode="max", mask=None, dx=None):
    """dx [N,C,H,W] from dy [N,C,P,Q] (and, for max, the forward's mask)."""
    import torch
    N, C, _, _ = dy.shape
    H, W = input_hw
    R, S = window
    _check(dy, "dy")
    if dx is None:
        dx = torch.empty((N, C, H, W), dtype=torch.float32, device=dy.device)
    _call(lib().pool_bwd, "pool_bwd", POOL_MODES[mode], N, C, H, W, R, S, stride, pad,
          _ptr(dy), _ptr(mask) if mode == "max" else None, _ptr(dx), _stream())
    return dx
