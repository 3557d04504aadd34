"""Python bindings of the oracle operators in ``oracle.c``.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Every function takes and returns float64 NumPy arrays in NHWC layout; convolution
weights are [K][R][S][C] and FC weights [out][in].  The arithmetic lives in
``oracle.c`` (textbook definitions, double accumulation); this module only
checks shapes and marshals pointers.  Element-wise operators that need no loop
(ReLU, residual add, global average pool) are written directly in NumPy here.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (plain gcc, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or (
                os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
            build(force=True)
        _lib = ctypes.CDLL(_LIB_PATH)
        _lib.oc_softmax_ce.restype = ctypes.c_double
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i(v):
    return ctypes.c_int(int(v))


def out_size(H: int, R: int, st: int, pad: int) -> int:
    return (H + 2 * pad - R) // st + 1


# ------------------------------------------------------------------ conv

def conv_fwd(x, w, b, stride: int, pad: int) -> np.ndarray:
    x = _f64(x); w = _f64(w)
    N, H, W, C = x.shape
    K, R, S, C2 = w.shape
    assert C == C2
    P, Q = out_size(H, R, stride, pad), out_size(W, S, stride, pad)
    y = np.empty((N, P, Q, K), np.float64)
    bb = _f64(b) if b is not None else None
    lib().oc_conv_fwd(_p(x), _i(N), _i(H), _i(W), _i(C), _p(w),
                      _p(bb) if bb is not None else None,
                      _i(K), _i(R), _i(S), _i(stride), _i(pad), _i(P), _i(Q), _p(y))
    return y


def conv_fwd_at(x, w, b, stride, pad, idx) -> np.ndarray:
    """Conv forward evaluated only at the flat NHWC output indices ``idx``."""
    x = _f64(x); w = _f64(w)
    N, H, W, C = x.shape
    K, R, S, _ = w.shape
    P, Q = out_size(H, R, stride, pad), out_size(W, S, stride, pad)
    idx = np.ascontiguousarray(idx, np.int64)
    out = np.empty(idx.size, np.float64)
    bb = _f64(b) if b is not None else None
    lib().oc_conv_fwd_at(_p(x), _i(N), _i(H), _i(W), _i(C), _p(w),
                         _p(bb) if bb is not None else None,
                         _i(K), _i(R), _i(S), _i(stride), _i(pad), _i(P), _i(Q),
                         _p(idx), ctypes.c_long(idx.size), _p(out))
    return out


def conv_dgrad(dy, w, stride: int, pad: int, H: int, W: int) -> np.ndarray:
    dy = _f64(dy); w = _f64(w)
    N, P, Q, K = dy.shape
    K2, R, S, C = w.shape
    assert K == K2
    dx = np.empty((N, H, W, C), np.float64)
    lib().oc_conv_dgrad(_p(dy), _i(N), _i(P), _i(Q), _i(K), _p(w), _i(R), _i(S), _i(C),
                        _i(stride), _i(pad), _i(H), _i(W), _p(dx))
    return dx


def conv_dgrad_at(dy, w, stride, pad, H, W, idx) -> np.ndarray:
    dy = _f64(dy); w = _f64(w)
    N, P, Q, K = dy.shape
    _, R, S, C = w.shape
    idx = np.ascontiguousarray(idx, np.int64)
    out = np.empty(idx.size, np.float64)
    lib().oc_conv_dgrad_at(_p(dy), _i(N), _i(P), _i(Q), _i(K), _p(w), _i(R), _i(S), _i(C),
                           _i(stride), _i(pad), _i(H), _i(W), _p(idx),
                           ctypes.c_long(idx.size), _p(out))
    return out


def conv_wgrad(x, dy, R: int, S: int, stride: int, pad: int, bias: bool):
    x = _f64(x); dy = _f64(dy)
    N, H, W, C = x.shape
    N2, P, Q, K = dy.shape
    assert N == N2
    dw = np.empty((K, R, S, C), np.float64)
    db = np.empty(K, np.float64) if bias else None
    lib().oc_conv_wgrad(_p(x), _i(N), _i(H), _i(W), _i(C), _p(dy), _i(P), _i(Q), _i(K),
                        _i(R), _i(S), _i(stride), _i(pad), _p(dw),
                        _p(db) if db is not None else None)
    return dw, db


def conv_wgrad_at(x, dy, R, S, stride, pad, idx) -> np.ndarray:
    x = _f64(x); dy = _f64(dy)
    N, H, W, C = x.shape
    _, P, Q, K = dy.shape
    idx = np.ascontiguousarray(idx, np.int64)
    out = np.empty(idx.size, np.float64)
    lib().oc_conv_wgrad_at(_p(x), _i(N), _i(H), _i(W), _i(C), _p(dy), _i(P), _i(Q), _i(K),
                           _i(R), _i(S), _i(stride), _i(pad), _p(idx),
                           ctypes.c_long(idx.size), _p(out))
    return out


# -------------------------------------------------------------------- FC

def fc_fwd(x, w, b) -> np.ndarray:
    x = _f64(x).reshape(x.shape[0], -1); w = _f64(w)
    B, IN = x.shape
    OUT, IN2 = w.shape
    assert IN == IN2
    y = np.empty((B, OUT), np.float64)
    bb = _f64(b) if b is not None else None
    lib().oc_fc_fwd(_p(x), _i(B), _i(IN), _p(w), _p(bb) if bb is not None else None,
                    _i(OUT), _p(y))
    return y


def fc_dgrad(dy, w) -> np.ndarray:
    dy = _f64(dy); w = _f64(w)
    B, OUT = dy.shape
    _, IN = w.shape
    dx = np.empty((B, IN), np.float64)
    lib().oc_fc_dgrad(_p(dy), _i(B), _i(OUT), _p(w), _i(IN), _p(dx))
    return dx


def fc_wgrad(x, dy, bias: bool):
    x = _f64(x).reshape(x.shape[0], -1); dy = _f64(dy)
    B, IN = x.shape
    _, OUT = dy.shape
    dw = np.empty((OUT, IN), np.float64)
    db = np.empty(OUT, np.float64) if bias else None
    lib().oc_fc_wgrad(_p(x), _i(B), _i(IN), _p(dy), _i(OUT), _p(dw),
                      _p(db) if db is not None else None)
    return dw, db


# -------------------------------------------------------------- max-pool

def maxpool_fwd(x, R: int, stride: int, pad: int) -> np.ndarray:
    x = _f64(x)
    N, H, W, C = x.shape
    P, Q = out_size(H, R, stride, pad), out_size(W, R, stride, pad)
    y = np.empty((N, P, Q, C), np.float64)
    lib().oc_maxpool_fwd(_p(x), _i(N), _i(H), _i(W), _i(C), _i(R), _i(R), _i(stride),
                         _i(pad), _i(P), _i(Q), _p(y))
    return y


def maxpool_bwd(x, dy, R: int, stride: int, pad: int) -> np.ndarray:
    x = _f64(x); dy = _f64(dy)
    N, H, W, C = x.shape
    _, P, Q, _ = dy.shape
    dx = np.empty_like(x)
    lib().oc_maxpool_bwd(_p(x), _i(N), _i(H), _i(W), _i(C), _i(R), _i(R), _i(stride),
                         _i(pad), _i(P), _i(Q), _p(dy), _p(dx))
    return dx


# ------------------------------------------------------------ batch-norm

def bn_fwd(x, gamma, beta, eps: float):
    """Training-mode batch-norm; returns (y, mean, invstd)."""
    x = _f64(x)
    C = x.shape[-1]
    M = x.size // C
    y = np.empty_like(x)
    mean = np.empty(C, np.float64)
    invstd = np.empty(C, np.float64)
    g = _f64(gamma); bt = _f64(beta)
    lib().oc_bn_fwd(_p(x), ctypes.c_long(M), _i(C), _p(g), _p(bt), ctypes.c_double(eps),
                    _p(y), _p(mean), _p(invstd))
    return y, mean, invstd


def bn_bwd(x, dy, gamma, mean, invstd):
    """Returns (dx, dgamma, dbeta)."""
    x = _f64(x); dy = _f64(dy)
    C = x.shape[-1]
    M = x.size // C
    dx = np.empty_like(x)
    dg = np.empty(C, np.float64)
    dbt = np.empty(C, np.float64)
    g = _f64(gamma); mu = _f64(mean); iv = _f64(invstd)
    lib().oc_bn_bwd(_p(x), _p(dy), ctypes.c_long(M), _i(C), _p(g), _p(mu), _p(iv),
                    _p(dx), _p(dg), _p(dbt))
    return dx, dg, dbt


# ------------------------------------------------ element-wise operators

def relu_fwd(x) -> np.ndarray:
    """y = max(x, 0)."""
    return np.maximum(_f64(x), 0.0)


def relu_bwd(x, dy) -> np.ndarray:
    """dx = dy where x > 0, else 0 (the derivative at 0 is taken as 0)."""
    return np.where(_f64(x) > 0.0, _f64(dy), 0.0)


def gap_fwd(x) -> np.ndarray:
    """Global average pool: y[n,c] = mean over (h,w) of x[n,h,w,c]."""
    x = _f64(x)
    N, H, W, C = x.shape
    return x.reshape(N, H * W, C).sum(axis=1) / float(H * W)


def gap_bwd(dy, H: int, W: int) -> np.ndarray:
    """dx[n,h,w,c] = dy[n,c] / (H W)."""
    dy = _f64(dy)
    N, C = dy.shape
    return np.broadcast_to((dy / float(H * W))[:, None, None, :], (N, H, W, C)).copy()


# ------------------------------------------------- softmax cross-entropy

def softmax_ce(z, labels):
    """Returns (mean loss, dz)."""
    z = _f64(z)
    B, K = z.shape
    lab = np.ascontiguousarray(labels, np.int32)
    assert lab.shape == (B,)
    dz = np.empty_like(z)
    loss = lib().oc_softmax_ce(_p(z), _i(B), _i(K), lab.ctypes.data_as(ctypes.c_void_p),
                               _p(dz))
    return float(loss), dz
