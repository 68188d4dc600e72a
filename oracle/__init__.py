"""Reference oracle (TEST INFRASTRUCTURE ONLY).

A plain, slow CPU implementation of the DML-style conv2d layer and the ops
around it, written from the paper's definitions ("Deep Learning with Apache
SystemML", Sections 2 and 3).  It exists to check the GPU library, never to
stand in for it: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with the
HIP library.

The arithmetic lives in ``oracle.c`` (fp64, nested loops, fixed summation
order).  This module builds it with gcc and wraps it for numpy arrays.  Every
array argument is converted to a C-contiguous float64 array; fp32-mode callers
pass fp32-rounded data, which converts exactly.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_CFLAGS = ["-O2", "-fopenmp", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
           "-std=c99", "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (plain C99 + OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *_CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None

_d = ctypes.POINTER(ctypes.c_double)
_i32 = ctypes.POINTER(ctypes.c_int32)
_int = ctypes.c_int


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    sig = {
        "oracle_set_threads": (None, [_int]),
        "oracle_get_threads": (_int, []),
        "oracle_conv2d_out_dim": (_int, [_int] * 4),
        "oracle_conv2d_forward_pre_elem": (ctypes.c_double, [_d, _d, _d] + [_int] * 11),
        "oracle_conv2d_forward": (None, [_d, _d, _d, _d] + [_int] * 10),
        "oracle_conv2d_backward_filter_elem": (ctypes.c_double, [_d, _d, _d] + [_int] * 13),
        "oracle_conv2d_backward_bias_elem": (ctypes.c_double, [_d, _d] + [_int] * 5),
        "oracle_conv2d_backward_filter": (None, [_d, _d, _d, _d, _d] + [_int] * 9),
        "oracle_conv2d_backward_data_elem": (ctypes.c_double, [_d, _d, _d] + [_int] * 12),
        "oracle_conv2d_backward_data": (None, [_d, _d, _d, _d] + [_int] * 9),
        "oracle_bias_add_relu": (None, [_d, _d, _d] + [_int] * 4),
        "oracle_max_pool2d_fwd": (None, [_d, _d, _i32] + [_int] * 8),
        "oracle_max_pool2d_bwd": (None, [_d, _i32, _d] + [_int] * 8),
        "oracle_affine_fwd": (None, [_d, _d, _d, _d] + [_int] * 4),
        "oracle_affine_bwd": (None, [_d, _d, _d, _d, _d, _d, _d] + [_int] * 3),
        "oracle_softmax_xent": (ctypes.c_double, [_d, _d, _d, _d, _int, _int]),
        "oracle_softmax_forward": (None, [_d, _d, _int, _int]),
        "oracle_xent_forward": (ctypes.c_double, [_d, _d, _int, _int]),
        "oracle_xent_backward": (None, [_d, _d, _d, _int, _int]),
        "oracle_softmax_backward": (None, [_d, _d, _d, _int, _int]),
        "oracle_sgd_update": (None, [_d, _d, ctypes.c_double, ctypes.c_longlong]),
        "oracle_sgd_nesterov_update": (None, [_d, _d, _d, ctypes.c_double, ctypes.c_double,
                                              ctypes.c_longlong]),
        "oracle_adagrad_update": (None, [_d, _d, _d, ctypes.c_double, ctypes.c_double,
                                         ctypes.c_longlong]),
        "oracle_rmsprop_update": (None, [_d, _d, _d] + [ctypes.c_double] * 3
                                  + [ctypes.c_longlong]),
        "oracle_adam_update": (None, [_d, _d, _d, _d] + [ctypes.c_double] * 4
                               + [ctypes.c_longlong, ctypes.c_longlong]),
        "oracle_sgd_momentum_update": (None, [_d, _d, _d, ctypes.c_double, ctypes.c_double,
                                              ctypes.c_longlong]),
        "oracle_count_nonzero": (ctypes.c_longlong, [_d, ctypes.c_longlong]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    if a is None:
        return None
    return a.ctypes.data_as(_d)


def _pi(a):
    return a.ctypes.data_as(_i32)


def set_threads(n: int) -> None:
    _load().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(_load().oracle_get_threads())


def out_dim(Hin, Hf, stride, pad) -> int:
    return int(_load().oracle_conv2d_out_dim(Hin, Hf, stride, pad))


# --------------------------------------------------------------------------- conv2d
def conv2d_forward(X, W, b, C, Hin, Win, Hf, Wf, stride, pad, relu=True):
    """Paper Section 3 (builtin conv2d): out = relu(conv(X, W) + b), N x (F*Hout*Wout)."""
    X, W = _f64(X), _f64(W)
    b = None if b is None else _f64(b)
    N, F = X.shape[0], W.shape[0]
    Hout, Wout = out_dim(Hin, Hf, stride, pad), out_dim(Win, Wf, stride, pad)
    out = np.empty((N, F * Hout * Wout), dtype=np.float64)
    _load().oracle_conv2d_forward(_p(X), _p(W), _p(b), _p(out), N, C, Hin, Win, F, Hf, Wf,
                                  stride, pad, int(bool(relu)))
    return out, Hout, Wout


def conv2d_forward_pre_elem(X, W, b, C, Hin, Win, Hf, Wf, stride, pad, n, f, oh, ow):
    """One pre-activation value; X, W, b must already be float64 contiguous."""
    return _load().oracle_conv2d_forward_pre_elem(_p(X), _p(W), _p(b), C, Hin, Win, Hf, Wf,
                                                  stride, pad, n, f, oh, ow)


def conv2d_backward_filter(X, dout, out_fwd, C, Hin, Win, Hf, Wf, stride, pad, F):
    """Returns (dW F x C*Hf*Wf, db F); out_fwd None means no relu mask."""
    X, dout = _f64(X), _f64(dout)
    out_fwd = None if out_fwd is None else _f64(out_fwd)
    N = X.shape[0]
    dW = np.empty((F, C * Hf * Wf), dtype=np.float64)
    db = np.empty((F,), dtype=np.float64)
    _load().oracle_conv2d_backward_filter(_p(X), _p(dout), _p(out_fwd), _p(dW), _p(db),
                                          N, C, Hin, Win, F, Hf, Wf, stride, pad)
    return dW, db


def conv2d_backward_filter_elem(X, dout, out_fwd, N, C, Hin, Win, F, Hf, Wf, stride, pad,
                                f, c, i, j):
    return _load().oracle_conv2d_backward_filter_elem(_p(X), _p(dout), _p(out_fwd), N, C, Hin,
                                                      Win, F, Hf, Wf, stride, pad, f, c, i, j)


def conv2d_backward_bias_elem(dout, out_fwd, N, F, Hout, Wout, f):
    return _load().oracle_conv2d_backward_bias_elem(_p(dout), _p(out_fwd), N, F, Hout, Wout, f)


def conv2d_backward_data(W, dout, out_fwd, C, Hin, Win, Hf, Wf, stride, pad):
    """Returns dX, N x (C*Hin*Win)."""
    W, dout = _f64(W), _f64(dout)
    out_fwd = None if out_fwd is None else _f64(out_fwd)
    N, F = dout.shape[0], W.shape[0]
    dX = np.empty((N, C * Hin * Win), dtype=np.float64)
    _load().oracle_conv2d_backward_data(_p(W), _p(dout), _p(out_fwd), _p(dX), N, C, Hin, Win,
                                        F, Hf, Wf, stride, pad)
    return dX


def conv2d_backward_data_elem(W, dout, out_fwd, C, Hin, Win, F, Hf, Wf, stride, pad,
                              n, c, h, w):
    return _load().oracle_conv2d_backward_data_elem(_p(W), _p(dout), _p(out_fwd), C, Hin, Win,
                                                    F, Hf, Wf, stride, pad, n, c, h, w)


# --------------------------------------------------------------------------- others
def bias_add_relu(X, b, C, HW, relu=True):
    X = _f64(X)
    b = None if b is None else _f64(b)
    out = np.empty_like(X)
    _load().oracle_bias_add_relu(_p(X), _p(b), _p(out), X.shape[0], C, HW, int(bool(relu)))
    return out


def max_pool2d_fwd(X, C, Hin, Win, Hf, Wf, stride, pad):
    """Returns (out, argmax int32 in-row index, Hout, Wout)."""
    X = _f64(X)
    N = X.shape[0]
    Hout, Wout = out_dim(Hin, Hf, stride, pad), out_dim(Win, Wf, stride, pad)
    out = np.empty((N, C * Hout * Wout), dtype=np.float64)
    idx = np.empty((N, C * Hout * Wout), dtype=np.int32)
    _load().oracle_max_pool2d_fwd(_p(X), _p(out), _pi(idx), N, C, Hin, Win, Hf, Wf, stride, pad)
    return out, idx, Hout, Wout


def max_pool2d_bwd(dout, argmax, C, Hin, Win, Hf, Wf, stride, pad):
    dout = _f64(dout)
    argmax = np.ascontiguousarray(argmax, dtype=np.int32)
    N = dout.shape[0]
    dX = np.empty((N, C * Hin * Win), dtype=np.float64)
    _load().oracle_max_pool2d_bwd(_p(dout), _pi(argmax), _p(dX), N, C, Hin, Win, Hf, Wf,
                                  stride, pad)
    return dX


def affine_fwd(X, W, b, relu=False):
    X, W = _f64(X), _f64(W)
    b = None if b is None else _f64(b)
    N, D = X.shape
    M = W.shape[1]
    out = np.empty((N, M), dtype=np.float64)
    _load().oracle_affine_fwd(_p(X), _p(W), _p(b), _p(out), N, D, M, int(bool(relu)))
    return out


def affine_bwd(dout, X, W, out_fwd=None, want_dX=True):
    """Returns [dX, dW, db] (dX None when want_dX is False)."""
    dout, X, W = _f64(dout), _f64(X), _f64(W)
    out_fwd = None if out_fwd is None else _f64(out_fwd)
    N, D = X.shape
    M = W.shape[1]
    dX = np.empty((N, D), dtype=np.float64) if want_dX else None
    dW = np.empty((D, M), dtype=np.float64)
    db = np.empty((M,), dtype=np.float64)
    _load().oracle_affine_bwd(_p(dout), _p(X), _p(W), _p(out_fwd), _p(dX), _p(dW), _p(db),
                              N, D, M)
    return dX, dW, db


def softmax_xent(S, Y, want_probs=True):
    """Fused closed form. Returns (loss, dS, probs-or-None)."""
    S, Y = _f64(S), _f64(Y)
    N, K = S.shape
    dS = np.empty_like(S)
    P = np.empty_like(S) if want_probs else None
    loss = _load().oracle_softmax_xent(_p(S), _p(Y), _p(P), _p(dS), N, K)
    return float(loss), dS, P


def softmax_forward(S):
    S = _f64(S)
    P = np.empty_like(S)
    _load().oracle_softmax_forward(_p(S), _p(P), S.shape[0], S.shape[1])
    return P


def xent_forward(P, Y):
    P, Y = _f64(P), _f64(Y)
    return float(_load().oracle_xent_forward(_p(P), _p(Y), P.shape[0], P.shape[1]))


def xent_backward(P, Y):
    P, Y = _f64(P), _f64(Y)
    dP = np.empty_like(P)
    _load().oracle_xent_backward(_p(P), _p(Y), _p(dP), P.shape[0], P.shape[1])
    return dP


def softmax_backward(dP, P):
    dP, P = _f64(dP), _f64(P)
    dS = np.empty_like(P)
    _load().oracle_softmax_backward(_p(dP), _p(P), _p(dS), P.shape[0], P.shape[1])
    return dS


def sgd_momentum_update(theta, grad, v, lr, mu):
    """In-place on copies: returns (theta_new, v_new)."""
    theta = _f64(theta).copy()
    v = _f64(v).copy()
    grad = _f64(grad)
    _load().oracle_sgd_momentum_update(_p(theta), _p(grad), _p(v), float(lr), float(mu),
                                       theta.size)
    return theta, v


def sgd_update(theta, grad, lr):
    """Returns theta - lr*grad (inputs untouched)."""
    theta = _f64(theta).copy()
    grad = _f64(grad)
    _load().oracle_sgd_update(_p(theta), _p(grad), float(lr), theta.size)
    return theta


def sgd_nesterov_update(theta, grad, v, lr, mu):
    """Returns (theta_new, v_new)."""
    theta, v, grad = _f64(theta).copy(), _f64(v).copy(), _f64(grad)
    _load().oracle_sgd_nesterov_update(_p(theta), _p(grad), _p(v), float(lr), float(mu),
                                       theta.size)
    return theta, v


def adagrad_update(theta, grad, cache, lr, eps):
    """Returns (theta_new, cache_new)."""
    theta, cache, grad = _f64(theta).copy(), _f64(cache).copy(), _f64(grad)
    _load().oracle_adagrad_update(_p(theta), _p(grad), _p(cache), float(lr), float(eps),
                                  theta.size)
    return theta, cache


def rmsprop_update(theta, grad, cache, lr, decay, eps):
    """Returns (theta_new, cache_new)."""
    theta, cache, grad = _f64(theta).copy(), _f64(cache).copy(), _f64(grad)
    _load().oracle_rmsprop_update(_p(theta), _p(grad), _p(cache), float(lr), float(decay),
                                  float(eps), theta.size)
    return theta, cache


def adam_update(theta, grad, m, v, lr, beta1, beta2, eps, t):
    """Returns (theta_new, m_new, v_new) after step t (t >= 1)."""
    theta, m, v, grad = _f64(theta).copy(), _f64(m).copy(), _f64(v).copy(), _f64(grad)
    _load().oracle_adam_update(_p(theta), _p(grad), _p(m), _p(v), float(lr), float(beta1),
                               float(beta2), float(eps), int(t), theta.size)
    return theta, m, v


def count_nonzero(X):
    X = _f64(X)
    return int(_load().oracle_count_nonzero(_p(X), X.size))
