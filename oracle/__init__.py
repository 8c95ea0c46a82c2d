"""Plain CPU oracle for the three passes of a convolution layer, and for a
pooling layer's forward and backward passes.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The product library never imports,
links or runs anything here, and this package imports nothing from it.

The arithmetic lives in ``oracle.c`` (fp64 direct loop nests; its header
gives the definitions and the readings of the paper).  This module only
builds that file with gcc, loads it with ctypes and marshals numpy arrays.

Every function takes the canonical fp32 inputs, widens them to float64
(exact) and returns float64 ``(value, abs_sum)`` pairs, where ``abs_sum`` is
the sum of |product| over every product that entered the element (plus |b|
for the forward output).  The tolerance of a compared result is a multiple
of ``abs_sum``.

Shapes are passed as ``shape = (N, C, H, W, K, R, S, stride, pad, group)``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle.c")
LIBRARY = os.path.join(_HERE, "liboracle.so")

_D = ctypes.POINTER(ctypes.c_double)
_L = ctypes.POINTER(ctypes.c_int64)
_I = ctypes.c_int
_GEO = [_I] * 10


def build(src: str = SOURCE, out: str = LIBRARY, werror: bool = True) -> str:
    """Compile ``src`` into the shared library ``out`` (gcc -O2, strict fp)."""
    tmp = out + ".tmp"
    subprocess.check_call([
        "gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
        "-fPIC", "-shared", "-std=c99", "-Wall", "-Wextra",
    ] + (["-Werror"] if werror else []) + ["-o", tmp, src, "-lm"])
    os.replace(tmp, out)
    return out


def _f64(a):
    """Contiguous float64 copy (exact widening of the fp32 inputs)."""
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_D)


class Oracle:
    """ctypes view of one build of ``oracle.c``."""

    def __init__(self, path: str = LIBRARY):
        lib = ctypes.CDLL(path)
        lib.oracle_out_size.argtypes = [_I, _I, _I, _I]
        lib.oracle_out_size.restype = _I
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = _I
        sigs = {
            "oracle_conv_fwd": _GEO + [_D] * 5,
            "oracle_conv_bwd_data": _GEO + [_D] * 4,
            "oracle_conv_bwd_weight": _GEO + [_D] * 6,
            "oracle_conv_fwd_at": _GEO + [_D, _D, _D, _L, ctypes.c_int64, _D, _D],
            "oracle_conv_bwd_data_at": _GEO + [_D, _D, _L, ctypes.c_int64, _D, _D],
            "oracle_conv_bwd_weight_at": _GEO + [_D, _D, _L, ctypes.c_int64, _D, _D],
            "oracle_bias_grad": [_I, _I, _I, _I, _D, _D, _D],
            "oracle_pool_fwd": [_I] * 9 + [_D, _D, _D, _L],
            "oracle_pool_bwd": [_I] * 9 + [_D, _L, _D, _D],
        }
        for name, args in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = None
        lib.oracle_pool_out_size.argtypes = [_I, _I, _I, _I]
        lib.oracle_pool_out_size.restype = _I
        self.lib = lib

    def out_size(self, n_in: int, filt: int, stride: int, pad: int) -> int:
        return int(self.lib.oracle_out_size(n_in, filt, stride, pad))

    def num_threads(self) -> int:
        return int(self.lib.oracle_num_threads())

    def _geom(self, shape):
        g = tuple(int(v) for v in shape)
        N, C, H, W, K, R, S, stride, pad, group = g
        return g, self.out_size(H, R, stride, pad), self.out_size(W, S, stride, pad)

    def conv_fwd(self, shape, x, w, b=None):
        """y and its abs-sum, both [N,K,P,Q] float64."""
        g, P, Q = self._geom(shape)
        x, w = _f64(x), _f64(w)
        b = None if b is None else _f64(b)
        y = np.empty((g[0], g[4], P, Q))
        ay = np.empty_like(y)
        self.lib.oracle_conv_fwd(*g, _ptr(x), _ptr(w), _ptr(b), _ptr(y), _ptr(ay))
        return y, ay

    def conv_bwd_data(self, shape, dy, w):
        """dx and its abs-sum, both [N,C,H,W] float64 (scatter form)."""
        g, _, _ = self._geom(shape)
        dy, w = _f64(dy), _f64(w)
        dx = np.empty(g[:4])
        adx = np.empty_like(dx)
        self.lib.oracle_conv_bwd_data(*g, _ptr(dy), _ptr(w), _ptr(dx), _ptr(adx))
        return dx, adx

    def conv_bwd_weight(self, shape, x, dy):
        """(dw, adw, db, adb): dw [K,C/G,R,S], db [K] (scatter form)."""
        g, _, _ = self._geom(shape)
        N, C, H, W, K, R, S, stride, pad, group = g
        x, dy = _f64(x), _f64(dy)
        dw = np.empty((K, C // group, R, S))
        adw = np.empty_like(dw)
        db = np.empty(K)
        adb = np.empty(K)
        self.lib.oracle_conv_bwd_weight(*g, _ptr(x), _ptr(dy), _ptr(dw), _ptr(adw),
                                        _ptr(db), _ptr(adb))
        return dw, adw, db, adb

    def _at(self, fn, shape, ins, idx):
        g, _, _ = self._geom(shape)
        idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).ravel())
        val = np.empty(idx.shape[0])
        aval = np.empty_like(val)
        getattr(self.lib, fn)(*g, *[_ptr(a) for a in ins], idx.ctypes.data_as(_L),
                              ctypes.c_int64(idx.shape[0]), _ptr(val), _ptr(aval))
        return val, aval

    def conv_fwd_at(self, shape, x, w, b, idx):
        """y at flat indices into [N,K,P,Q] (gather form)."""
        return self._at("oracle_conv_fwd_at", shape,
                        [_f64(x), _f64(w), None if b is None else _f64(b)], idx)

    def conv_bwd_data_at(self, shape, dy, w, idx):
        """dx at flat indices into [N,C,H,W] (gather form)."""
        return self._at("oracle_conv_bwd_data_at", shape, [_f64(dy), _f64(w)], idx)

    def conv_bwd_weight_at(self, shape, x, dy, idx):
        """dw at flat indices into [K,C/G,R,S] (gather form)."""
        return self._at("oracle_conv_bwd_weight_at", shape, [_f64(x), _f64(dy)], idx)

    # Pooling (Sec. IV-D).  pshape = (N, C, H, W, R, S, stride, pad); mode
    # "max" or "avg".
    def pool_out_size(self, n_in: int, filt: int, stride: int, pad: int) -> int:
        return int(self.lib.oracle_pool_out_size(n_in, filt, stride, pad))

    def pool_fwd(self, mode, pshape, x):
        """(y, ay, mask): y [N,C,P,Q] float64, its abs-sum scale (|y| for max,
        sum|x| / area for avg), and for max the argmax h*W+w within the plane
        (int64; -1 for avg)."""
        N, C, H, W, R, S, st, pad = (int(v) for v in pshape)
        P, Q = self.pool_out_size(H, R, st, pad), self.pool_out_size(W, S, st, pad)
        if P < 1 or Q < 1:
            raise ValueError(f"no pooling for {pshape}: a window would cover no input element")
        x = _f64(x)
        y = np.empty((N, C, P, Q))
        ay = np.empty_like(y)
        mask = np.full((N, C, P, Q), -1, dtype=np.int64)
        self.lib.oracle_pool_fwd(_pool_mode(mode), N, C, H, W, R, S, st, pad, _ptr(x), _ptr(y),
                                 _ptr(ay), mask.ctypes.data_as(_L))
        return y, ay, mask

    def pool_bwd(self, mode, pshape, dy, mask=None):
        """(dx, adx) [N,C,H,W] float64 (scatter form); max needs the mask."""
        N, C, H, W, R, S, st, pad = (int(v) for v in pshape)
        dy = _f64(dy)
        m = None
        if _pool_mode(mode) == 0:
            m = np.ascontiguousarray(np.asarray(mask, dtype=np.int64))
            assert m.shape == dy.shape
            if m.size and (m.min() < 0 or m.max() >= H * W):
                raise ValueError("max-pooling mask entry outside the input plane")
        dx = np.empty((N, C, H, W))
        adx = np.empty_like(dx)
        self.lib.oracle_pool_bwd(_pool_mode(mode), N, C, H, W, R, S, st, pad, _ptr(dy),
                                 None if m is None else m.ctypes.data_as(_L), _ptr(dx),
                                 _ptr(adx))
        return dx, adx

    def bias_grad(self, dy):
        """db and its abs-sum from dy [N,K,P,Q]."""
        dy = _f64(dy)
        N, K, P, Q = dy.shape
        db = np.empty(K)
        adb = np.empty(K)
        self.lib.oracle_bias_grad(N, K, P, Q, _ptr(dy), _ptr(db), _ptr(adb))
        return db, adb


def _pool_mode(mode):
    return {"max": 0, "avg": 1}[mode]


_default = None


def default() -> Oracle:
    """The oracle built from ``oracle.c`` in this directory (built on first use)."""
    global _default
    if _default is None:
        if not os.path.exists(LIBRARY) or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE):
            build()
        _default = Oracle(LIBRARY)
    return _default


def out_size(n_in, filt, stride, pad):
    return default().out_size(n_in, filt, stride, pad)


def num_threads():
    return default().num_threads()


def conv_fwd(shape, x, w, b=None):
    return default().conv_fwd(shape, x, w, b)


def conv_bwd_data(shape, dy, w):
    return default().conv_bwd_data(shape, dy, w)


def conv_bwd_weight(shape, x, dy):
    return default().conv_bwd_weight(shape, x, dy)


def conv_fwd_at(shape, x, w, b, idx):
    return default().conv_fwd_at(shape, x, w, b, idx)


def conv_bwd_data_at(shape, dy, w, idx):
    return default().conv_bwd_data_at(shape, dy, w, idx)


def conv_bwd_weight_at(shape, x, dy, idx):
    return default().conv_bwd_weight_at(shape, x, dy, idx)


def bias_grad(dy):
    return default().bias_grad(dy)


def pool_out_size(n_in, filt, stride, pad):
    return default().pool_out_size(n_in, filt, stride, pad)


def pool_fwd(mode, pshape, x):
    return default().pool_fwd(mode, pshape, x)


def pool_bwd(mode, pshape, dy, mask=None):
    return default().pool_bwd(mode, pshape, dy, mask)
