"""Test infrastructure: ctypes access to the oracle's C primitives (``prim.c``), fp64 numpy in/out.

Builds ``_prim.so`` with gcc on first use (or when the source is newer).  Only tests, the smoke
check and the benchmark's CPU-baseline leg may use the oracle.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_DIR = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_DIR, "prim.c")
_LIB = os.path.join(_DIR, "_prim.so")
_lib = None


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        D = ctypes.POINTER(ctypes.c_double)
        i = ctypes.c_int
        for name in ("pnn_oracle_conv_fwd", "pnn_oracle_conv_bwd_data", "pnn_oracle_conv_bwd_weight"):
            getattr(_lib, name).argtypes = [D, i, i, i, i, D, i, i, i, i, D, i, i]
        _lib.pnn_oracle_maxpool_fwd.argtypes = [D, i, i, i, i, i, i, i, D, i, i]
        _lib.pnn_oracle_maxpool_bwd.argtypes = [D, i, i, i, i, i, i, i, D, D, i, i]
        _lib.pnn_oracle_bn_stats.argtypes = [D, ctypes.c_long, i, D, D]
        _lib.pnn_oracle_colsum2.argtypes = [D, D, ctypes.c_long, i, D, D]
        _lib.pnn_oracle_round_bf16.argtypes = [D, ctypes.c_size_t]
        _lib.pnn_oracle_threads.restype = i
        L_ = ctypes.POINTER(ctypes.c_long)
        for name in ("pnn_oracle_conv_fwd_at", "pnn_oracle_conv_bwd_data_at", "pnn_oracle_conv_bwd_weight_at"):
            getattr(_lib, name).argtypes = [D, i, i, i, i, D, i, i, i, i, i, i, L_, ctypes.c_long, D]
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _c(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def threads() -> int:
    return lib().pnn_oracle_threads()


def out_hw(H, W, k, st, pad):
    return (H + 2 * pad - k) // st + 1, (W + 2 * pad - k) // st + 1


def conv_fwd(x, w, st, pad):
    x, w = _c(x), _c(w)
    B, H, W, C = x.shape
    K, k, _, Cw = w.shape
    assert Cw == C
    Ho, Wo = out_hw(H, W, k, st, pad)
    y = np.empty((B, Ho, Wo, K))
    lib().pnn_oracle_conv_fwd(_p(x), B, H, W, C, _p(w), K, k, st, pad, _p(y), Ho, Wo)
    return y


def conv_bwd_data(gy, w, x_shape, st, pad):
    gy, w = _c(gy), _c(w)
    B, H, W, C = x_shape
    K, k, _, _ = w.shape
    Ho, Wo = gy.shape[1], gy.shape[2]
    gx = np.empty((B, H, W, C))
    lib().pnn_oracle_conv_bwd_data(_p(gy), B, H, W, C, _p(w), K, k, st, pad, _p(gx), Ho, Wo)
    return gx


def conv_bwd_weight(x, gy, k, st, pad):
    x, gy = _c(x), _c(gy)
    B, H, W, C = x.shape
    K = gy.shape[3]
    Ho, Wo = gy.shape[1], gy.shape[2]
    gw = np.empty((K, k, k, C))
    lib().pnn_oracle_conv_bwd_weight(_p(x), B, H, W, C, _p(gy), K, k, st, pad, _p(gw), Ho, Wo)
    return gw


def maxpool_fwd(x, k, st, pad):
    x = _c(x)
    B, H, W, C = x.shape
    Ho, Wo = out_hw(H, W, k, st, pad)
    y = np.empty((B, Ho, Wo, C))
    lib().pnn_oracle_maxpool_fwd(_p(x), B, H, W, C, k, st, pad, _p(y), Ho, Wo)
    return y


def maxpool_bwd(x, gy, k, st, pad):
    x, gy = _c(x), _c(gy)
    B, H, W, C = x.shape
    gx = np.zeros_like(x)
    lib().pnn_oracle_maxpool_bwd(_p(x), B, H, W, C, k, st, pad, _p(gy), _p(gx), gy.shape[1], gy.shape[2])
    return gx


def bn_stats(x2d):
    x2d = _c(x2d)
    M, C = x2d.shape
    mean, var = np.empty(C), np.empty(C)
    lib().pnn_oracle_bn_stats(_p(x2d), M, C, _p(mean), _p(var))
    return mean, var


def colsum2(a2d, b2d):
    a2d, b2d = _c(a2d), _c(b2d)
    M, C = a2d.shape
    sa, sab = np.empty(C), np.empty(C)
    lib().pnn_oracle_colsum2(_p(a2d), _p(b2d), M, C, _p(sa), _p(sab))
    return sa, sab


def round_bf16(x):
    y = np.array(x, dtype=np.float64, copy=True, order="C")
    lib().pnn_oracle_round_bf16(_p(y), y.size)
    return y


def _idx(idx):
    a = np.ascontiguousarray(idx, dtype=np.int64)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_long))


def conv_fwd_at(x, w, st, pad, idx):
    """conv_fwd(x, w, st, pad).ravel()[idx]"""
    x, w = _c(x), _c(w)
    B, H, W, C = x.shape
    K, k, _, _ = w.shape
    Ho, Wo = out_hw(H, W, k, st, pad)
    a, ap = _idx(idx)
    out = np.empty(len(a))
    lib().pnn_oracle_conv_fwd_at(_p(x), B, H, W, C, _p(w), K, k, st, pad, Ho, Wo, ap, len(a), _p(out))
    return out


def conv_bwd_data_at(gy, w, x_shape, st, pad, idx):
    """conv_bwd_data(gy, w, x_shape, st, pad).ravel()[idx]"""
    gy, w = _c(gy), _c(w)
    B, H, W, C = x_shape
    K, k, _, _ = w.shape
    a, ap = _idx(idx)
    out = np.empty(len(a))
    lib().pnn_oracle_conv_bwd_data_at(_p(gy), B, H, W, C, _p(w), K, k, st, pad, gy.shape[1], gy.shape[2],
                                      ap, len(a), _p(out))
    return out


def conv_bwd_weight_at(x, gy, k, st, pad, idx):
    """conv_bwd_weight(x, gy, k, st, pad).ravel()[idx]"""
    x, gy = _c(x), _c(gy)
    B, H, W, C = x.shape
    K = gy.shape[3]
    a, ap = _idx(idx)
    out = np.empty(len(a))
    lib().pnn_oracle_conv_bwd_weight_at(_p(x), B, H, W, C, _p(gy), K, k, st, pad, gy.shape[1], gy.shape[2],
                                        ap, len(a), _p(out))
    return out
