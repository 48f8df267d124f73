"""ctypes front end of the C oracle (test infrastructure only).

The arithmetic lives in conv2d_oracle.c; this file marshals numpy arrays and
computes the normalised error readings from the oracle's y and A outputs.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle status {code}")
        self.code = code


class _Params(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int64) for f in (
        "n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
        "dil_h", "dil_w", "groups", "has_bias")]


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER(_Params)
        vp = ctypes.c_void_p
        lib.oracle_output_dims.argtypes = [P, ctypes.POINTER(ctypes.c_int64),
                                           ctypes.POINTER(ctypes.c_int64)]
        lib.oracle_conv2d.argtypes = [P, vp, vp, vp, vp, vp, ctypes.c_int]
        lib.oracle_conv2d_points.argtypes = [P, vp, vp, vp, ctypes.c_int64, vp, vp, vp,
                                             ctypes.c_int]
        lib.oracle_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _params(x_shape, w_shape, stride, pad, dil, groups, has_bias):
    n, c, h, w = x_shape
    k, cg, r, s = w_shape
    return _Params(n, c, h, w, k, r, s, stride[0], stride[1], pad[0], pad[1], dil[0], dil[1],
                   groups, 1 if has_bias else 0)


def output_dims(x_shape, w_shape, stride=(1, 1), pad=(0, 0), dil=(1, 1), groups=1):
    lib = load()
    p = _params(x_shape, w_shape, stride, pad, dil, groups, False)
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    st = lib.oracle_output_dims(ctypes.byref(p), ctypes.byref(ho), ctypes.byref(wo))
    if st:
        raise OracleError(st)
    return ho.value, wo.value


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _check_w(x, w, groups):
    if x.ndim != 4 or w.ndim != 4:
        raise ValueError("x and w must be 4-D (NCHW and K x C/g x R x S)")
    if groups < 1 or x.shape[1] % groups or w.shape[1] * groups != x.shape[1]:
        raise ValueError("w.shape[1] * groups must equal C")


def conv2d(x, w, b=None, stride=(1, 1), pad=(0, 0), dil=(1, 1), groups=1, nthreads=0,
           want_abs=True):
    """Full fp64 evaluation.  x NCHW fp32, w K x C/g x R x S fp32, b fp32 or None.
    Returns (y, A) as float64 N x K x Ho x Wo arrays (A is None if not wanted)."""
    lib = load()
    x, w = _f32(x), _f32(w)
    _check_w(x, w, groups)
    bb = None if b is None else _f32(b)
    p = _params(x.shape, w.shape, stride, pad, dil, groups, b is not None)
    ho, wo = output_dims(x.shape, w.shape, stride, pad, dil, groups)
    y = np.empty((x.shape[0], w.shape[0], ho, wo), dtype=np.float64)
    a = np.empty_like(y) if want_abs else None
    st = lib.oracle_conv2d(ctypes.byref(p), x.ctypes.data, w.ctypes.data,
                           None if bb is None else bb.ctypes.data, y.ctypes.data,
                           None if a is None else a.ctypes.data, int(nthreads))
    if st:
        raise OracleError(st)
    return y, a


def conv2d_points(x, w, b, idx, stride=(1, 1), pad=(0, 0), dil=(1, 1), groups=1, nthreads=0):
    """Evaluate only at the rows of idx (int64 [npts, 4] of n, k, ho, wo).
    Returns (y, A) float64 vectors."""
    lib = load()
    x, w = _f32(x), _f32(w)
    _check_w(x, w, groups)
    bb = None if b is None else _f32(b)
    idx = np.ascontiguousarray(idx, dtype=np.int64).reshape(-1, 4)
    p = _params(x.shape, w.shape, stride, pad, dil, groups, b is not None)
    y = np.empty(idx.shape[0], dtype=np.float64)
    a = np.empty(idx.shape[0], dtype=np.float64)
    st = lib.oracle_conv2d_points(ctypes.byref(p), x.ctypes.data, w.ctypes.data,
                                  None if bb is None else bb.ctypes.data, idx.shape[0],
                                  idx.ctypes.data, y.ctypes.data, a.ctypes.data, int(nthreads))
    if st:
        raise OracleError(st)
    return y, a


def max_threads() -> int:
    return int(load().oracle_max_threads())


def normalised_errors(y, y_ref, a_ref):
    """The two error readings of a result against the oracle.

    literal   = max_o |y - y_ref| / max_o A
    per_point = max over outputs with A > 0 of |y - y_ref| / A; outputs with
                A == 0 must match exactly, else the reading is +inf.
    """
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    a_ref = np.asarray(a_ref, dtype=np.float64)
    if y.shape != y_ref.shape or y.shape != a_ref.shape:
        raise ValueError(f"shape mismatch {y.shape} {y_ref.shape} {a_ref.shape}")
    if y.size == 0:
        return 0.0, 0.0
    if not np.all(np.isfinite(y)):
        return float("inf"), float("inf")
    e = np.abs(y - y_ref)
    amax = float(a_ref.max())
    literal = float(e.max() / amax) if amax > 0 else (0.0 if e.max() == 0 else float("inf"))
    pos = a_ref > 0
    per_point = float((e[pos] / a_ref[pos]).max()) if pos.any() else 0.0
    if np.any(e[~pos] != 0):
        per_point = float("inf")
    return literal, per_point
