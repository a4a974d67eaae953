"""fp64 CPU oracle for 2-D convolution (forward, backward-data, backward-weight).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg import this module.  It never imports the GPU
package and the GPU package never imports it.

The arithmetic lives in ``conv_oracle.c`` (plain C loops in double precision,
written from the textbook definition of convolution: the paper states the
operation only as an API call in Sec. 3.2, Listings 4-5, trained by
back-propagation, Sec. 2.1, with the loss scaling of Sec. 3.3, Listing 6).
This module compiles that file with gcc and marshals numpy arrays to it.

Array conventions (the paper's "base axis 1": batch first, channels second):
    x  : float64 [N, C, H, W]
    w  : float64 [K, C/g, R, S]
    y  : float64 [N, K, P, Q]
Channel-last data is compared by transposing numpy arrays (pure data
movement) before or after calling in here.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "conv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libconv_oracle.so")
_lock = threading.Lock()
_lib = None

_I64 = ctypes.c_int64
_DP = ctypes.POINTER(ctypes.c_double)
_IP = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = True, src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (IEEE semantics: no -ffast-math)."""
    if not force and os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(src):
        return out
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _declare(lib):
    shape = [_I64] * 14
    lib.oracle_output_dims.argtypes = shape + [_IP, _IP]
    lib.oracle_conv_fwd.argtypes = shape + [_DP, _DP, ctypes.c_double, _DP]
    lib.oracle_conv_dgrad.argtypes = shape + [_DP, _DP, ctypes.c_double, _DP]
    lib.oracle_conv_dgrad_scatter.argtypes = shape + [_DP, _DP, ctypes.c_double, _DP]
    lib.oracle_conv_wgrad.argtypes = shape + [_DP, _DP, ctypes.c_double, ctypes.c_int, _DP]
    lib.oracle_conv_fwd_points.argtypes = shape + [_DP, _DP, ctypes.c_double, _I64, _IP, _DP]
    lib.oracle_conv_dgrad_points.argtypes = shape + [_DP, _DP, ctypes.c_double, _I64, _IP, _DP]
    lib.oracle_conv_wgrad_points.argtypes = shape + [_DP, _DP, _I64, _IP, _DP]
    lib.oracle_any_nonfinite.argtypes = [_DP, _I64]
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    for f in ("oracle_output_dims", "oracle_conv_fwd", "oracle_conv_dgrad",
              "oracle_conv_dgrad_scatter", "oracle_conv_wgrad",
              "oracle_conv_fwd_points", "oracle_conv_dgrad_points",
              "oracle_conv_wgrad_points", "oracle_any_nonfinite",
              "oracle_get_threads"):
        getattr(lib, f).restype = ctypes.c_int
    lib.oracle_set_threads.restype = None
    return lib


def load(path: str | None = None):
    """Load (building first if needed) the oracle shared library.

    With ``path`` given, load that build instead of the default one (the
    planted-mistake tests compile modified copies)."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
                build()
            _lib = _declare(ctypes.CDLL(_LIB_PATH))
    return _lib


def _p(a):
    return a.ctypes.data_as(_DP)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


class Conv:
    """One convolution geometry, evaluated by the oracle library ``lib``."""

    def __init__(self, n, c, h, w, k, r, s, stride=(1, 1), pad=(0, 0),
                 dil=(1, 1), groups=1, lib=None):
        self.lib = lib if lib is not None else load()
        self.args = tuple(int(v) for v in (n, c, h, w, k, r, s, stride[0], stride[1],
                                           pad[0], pad[1], dil[0], dil[1], groups))
        p = ctypes.c_int64()
        q = ctypes.c_int64()
        if not self.lib.oracle_output_dims(*self.args, ctypes.byref(p), ctypes.byref(q)):
            raise ValueError("invalid convolution shape %r" % (self.args,))
        self.n, self.c, self.h, self.w, self.k, self.r, self.s = self.args[:7]
        self.groups = groups
        self.p, self.q = p.value, q.value

    @property
    def x_shape(self):
        return (self.n, self.c, self.h, self.w)

    @property
    def w_shape(self):
        return (self.k, self.c // self.groups, self.r, self.s)

    @property
    def y_shape(self):
        return (self.n, self.k, self.p, self.q)

    def _check(self, a, shape, name):
        if tuple(a.shape) != tuple(shape):
            raise ValueError("%s has shape %r, expected %r" % (name, a.shape, shape))

    def fwd(self, x, w, alpha=1.0):
        x, w = _f64(x), _f64(w)
        self._check(x, self.x_shape, "x")
        self._check(w, self.w_shape, "w")
        y = np.empty(self.y_shape, np.float64)
        assert self.lib.oracle_conv_fwd(*self.args, _p(x), _p(w), float(alpha), _p(y))
        return y

    def dgrad(self, dy, w, alpha=1.0):
        dy, w = _f64(dy), _f64(w)
        self._check(dy, self.y_shape, "dy")
        self._check(w, self.w_shape, "w")
        dx = np.empty(self.x_shape, np.float64)
        assert self.lib.oracle_conv_dgrad(*self.args, _p(dy), _p(w), float(alpha), _p(dx))
        return dx

    def dgrad_scatter(self, dy, w, alpha=1.0):
        dy, w = _f64(dy), _f64(w)
        self._check(dy, self.y_shape, "dy")
        self._check(w, self.w_shape, "w")
        dx = np.empty(self.x_shape, np.float64)
        assert self.lib.oracle_conv_dgrad_scatter(*self.args, _p(dy), _p(w), float(alpha), _p(dx))
        return dx

    def wgrad(self, x, dy, inv_loss_scale=1.0, beta=0, dw_old=None):
        x, dy = _f64(x), _f64(dy)
        self._check(x, self.x_shape, "x")
        self._check(dy, self.y_shape, "dy")
        if beta:
            if dw_old is None:
                raise ValueError("beta=1 needs dw_old")
            dw = _f64(dw_old).copy()
            self._check(dw, self.w_shape, "dw_old")
        else:
            dw = np.zeros(self.w_shape, np.float64)
        assert self.lib.oracle_conv_wgrad(*self.args, _p(x), _p(dy), float(inv_loss_scale),
                                          1 if beta else 0, _p(dw))
        return dw

    def fwd_points(self, x, w, idx, alpha=1.0):
        x, w = _f64(x), _f64(w)
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        out = np.empty(idx.shape, np.float64)
        assert self.lib.oracle_conv_fwd_points(*self.args, _p(x), _p(w), float(alpha),
                                               idx.size, idx.ctypes.data_as(_IP), _p(out))
        return out

    def dgrad_points(self, dy, w, idx, alpha=1.0):
        dy, w = _f64(dy), _f64(w)
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        out = np.empty(idx.shape, np.float64)
        assert self.lib.oracle_conv_dgrad_points(*self.args, _p(dy), _p(w), float(alpha),
                                                 idx.size, idx.ctypes.data_as(_IP), _p(out))
        return out

    def wgrad_points(self, x, dy, idx):
        """Raw weight-gradient sums (before the loss-scale step) at KCRS flat indices."""
        x, dy = _f64(x), _f64(dy)
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        out = np.empty(idx.shape, np.float64)
        assert self.lib.oracle_conv_wgrad_points(*self.args, _p(x), _p(dy), idx.size,
                                                 idx.ctypes.data_as(_IP), _p(out))
        return out


def any_nonfinite(a, lib=None) -> bool:
    lib = lib if lib is not None else load()
    a = _f64(a).ravel()
    return bool(lib.oracle_any_nonfinite(_p(a), a.size))


def set_threads(n: int, lib=None) -> None:
    (lib if lib is not None else load()).oracle_set_threads(int(n))


def get_threads(lib=None) -> int:
    return int((lib if lib is not None else load()).oracle_get_threads())


def rel_err(got, ref) -> float:
    """max|got - ref| / max|ref| (the parity measure); exact match required
    when the reference is identically zero."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    m = float(np.max(np.abs(ref))) if ref.size else 0.0
    d = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    if m == 0.0:
        return 0.0 if d == 0.0 else float("inf")
    return d / m
