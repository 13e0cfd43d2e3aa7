"""numpy front-end to the oracle's float64 C layer definitions (``oracle.c``).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Every function takes and returns float64 numpy arrays (inputs of other float
types are widened first) and follows one textbook layer definition:

* ``conv2d``      zero-padded cross-correlation plus bias, floor-mode output size
* ``batchnorm``   inference batch normalisation, eps 1e-5
* ``maxpool2d``   window maximum, padding counted as -infinity
* ``avgpool2d``, ``avgpool_global``   window / global mean
* ``linear``      x W^T + b
* ``layernorm``   per-row normalisation with affine, biased variance
* ``gelu``        exact-erf GELU
* ``attention``   multi-head softmax(Q K^T / sqrt(d_head)) V
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np

from . import build as _build

_lib = None
_lock = threading.Lock()
_dp = ctypes.POINTER(ctypes.c_double)


def _load():
    global _lib
    with _lock:
        if _lib is None:
            path = _build.build(force=False)
            lib = ctypes.CDLL(path)
            i32, i64, dbl = ctypes.c_int, ctypes.c_int64, ctypes.c_double
            lib.oracle_conv2d.argtypes = [_dp, i32, i32, i32, i32, _dp, i32, i32, i32,
                                          i32, i32, _dp, _dp]
            lib.oracle_batchnorm.argtypes = [_dp, i32, i32, i64, _dp, _dp, _dp, _dp, dbl]
            lib.oracle_relu.argtypes = [_dp, i64]
            lib.oracle_add.argtypes = [_dp, _dp, i64]
            lib.oracle_maxpool2d.argtypes = [_dp, i32, i32, i32, i32, i32, i32, i32, _dp]
            lib.oracle_avgpool2d.argtypes = [_dp, i32, i32, i32, i32, i32, i32, _dp]
            lib.oracle_avgpool_global.argtypes = [_dp, i32, i32, i64, _dp]
            lib.oracle_linear.argtypes = [_dp, i64, i32, _dp, i32, _dp, _dp]
            lib.oracle_layernorm.argtypes = [_dp, i64, i32, _dp, _dp, dbl, _dp]
            lib.oracle_gelu.argtypes = [_dp, i64]
            lib.oracle_attention.argtypes = [_dp, i32, i32, i32, i32, _dp]
            lib.oracle_max_tokens.restype = i32
            _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    return None if a is None else a.ctypes.data_as(_dp)


def set_threads(n: int) -> None:
    """Set the OpenMP thread count used by later oracle calls (0 = leave default)."""
    if n > 0:
        os.environ["OMP_NUM_THREADS"] = str(n)
        try:
            ctypes.CDLL("libgomp.so.1").omp_set_num_threads(ctypes.c_int(n))
        except OSError:
            pass


def conv2d(x, w, bias=None, stride: int = 1, pad: int = 0) -> np.ndarray:
    """x [N, C, H, W], w [O, C, kh, kw], bias [O] or None -> [N, O, Ho, Wo]."""
    lib = _load()
    x, w = _f64(x), _f64(w)
    N, C, H, W = x.shape
    O, Cw, kh, kw = w.shape
    if Cw != C:
        raise ValueError(f"conv2d: input has {C} channels, weight expects {Cw}")
    Ho = (H + 2 * pad - kh) // stride + 1
    Wo = (W + 2 * pad - kw) // stride + 1
    if Ho <= 0 or Wo <= 0:
        raise ValueError("conv2d: empty output")
    b = None if bias is None else _f64(bias)
    y = np.empty((N, O, Ho, Wo), np.float64)
    lib.oracle_conv2d(_p(x), N, C, H, W, _p(w), O, kh, kw, stride, pad, _p(b), _p(y))
    return y


def batchnorm(x, gamma, beta, mean, var, eps: float = 1e-5) -> np.ndarray:
    lib = _load()
    y = _f64(x).copy()
    N, C = y.shape[0], y.shape[1]
    hw = int(np.prod(y.shape[2:])) if y.ndim > 2 else 1
    lib.oracle_batchnorm(_p(y), N, C, hw, _p(_f64(gamma)), _p(_f64(beta)),
                         _p(_f64(mean)), _p(_f64(var)), float(eps))
    return y


def relu(x) -> np.ndarray:
    lib = _load()
    y = _f64(x).copy()
    lib.oracle_relu(_p(y), y.size)
    return y


def add(a, b) -> np.ndarray:
    lib = _load()
    y = _f64(a).copy()
    b = _f64(b)
    if b.shape != y.shape:
        raise ValueError("add: shape mismatch")
    lib.oracle_add(_p(y), _p(b), y.size)
    return y


def maxpool2d(x, k: int, stride: int, pad: int = 0) -> np.ndarray:
    lib = _load()
    x = _f64(x)
    N, C, H, W = x.shape
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    y = np.empty((N, C, Ho, Wo), np.float64)
    lib.oracle_maxpool2d(_p(x), N, C, H, W, k, stride, pad, _p(y))
    return y


def avgpool2d(x, k: int, stride: int) -> np.ndarray:
    lib = _load()
    x = _f64(x)
    N, C, H, W = x.shape
    y = np.empty((N, C, (H - k) // stride + 1, (W - k) // stride + 1), np.float64)
    lib.oracle_avgpool2d(_p(x), N, C, H, W, k, stride, _p(y))
    return y


def avgpool_global(x) -> np.ndarray:
    """[N, C, H, W] -> [N, C, 1, 1]."""
    lib = _load()
    x = _f64(x)
    N, C = x.shape[0], x.shape[1]
    hw = int(np.prod(x.shape[2:]))
    y = np.empty((N, C, 1, 1), np.float64)
    lib.oracle_avgpool_global(_p(x), N, C, hw, _p(y))
    return y


def linear(x, w, bias=None) -> np.ndarray:
    """x [..., K], w [O, K] -> [..., O]."""
    lib = _load()
    x, w = _f64(x), _f64(w)
    lead = x.shape[:-1]
    K = x.shape[-1]
    O = w.shape[0]
    if w.shape[1] != K:
        raise ValueError("linear: inner dimension mismatch")
    M = int(np.prod(lead)) if lead else 1
    y = np.empty(lead + (O,), np.float64)
    b = None if bias is None else _f64(bias)
    lib.oracle_linear(_p(x), M, K, _p(w), O, _p(b), _p(y))
    return y


def layernorm(x, gamma, beta, eps: float = 1e-6) -> np.ndarray:
    lib = _load()
    x = _f64(x)
    D = x.shape[-1]
    M = x.size // D
    y = np.empty_like(x)
    lib.oracle_layernorm(_p(x), M, D, _p(_f64(gamma)), _p(_f64(beta)), float(eps), _p(y))
    return y


def gelu(x) -> np.ndarray:
    lib = _load()
    y = _f64(x).copy()
    lib.oracle_gelu(_p(y), y.size)
    return y


def attention(qkv, heads: int) -> np.ndarray:
    """qkv [N, T, 3D] -> [N, T, D] (per-head softmax attention, heads concatenated)."""
    lib = _load()
    qkv = _f64(qkv)
    N, T, D3 = qkv.shape
    D = D3 // 3
    if D3 != 3 * D or D % heads:
        raise ValueError("attention: bad qkv width / head count")
    if T > lib.oracle_max_tokens():
        raise ValueError("attention: sequence too long for the oracle")
    y = np.empty((N, T, D), np.float64)
    lib.oracle_attention(_p(qkv), N, T, D, heads, _p(y))
    return y
