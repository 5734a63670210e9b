"""CPU oracle: plain fp64 loop nests for the convnet SGD step (test infrastructure).

Only the tests, the smoke check and the bench's CPU-baseline leg use this
package.  It is the checker, never a fallback: nothing in the HIP library or
its Python binding imports it.

The arithmetic lives in ``oracle.c`` (compiled with gcc, OpenMP over
independent output elements only).  This module marshals float64 numpy arrays
into it and computes output shapes with its own formula.

Parity status of each function (pins are in tests/test_oracle_pins.py):

* conv2d_fwd        pinned: library conv (torch float64 CPU), 1x1 conv = matmul,
                    delta / shifted-delta kernels, all-ones closed form.
* conv2d_bwd_input  pinned: finite differences, adjoint identity, delta kernel.
* conv2d_bwd_input  also pinned against torch autograd (float64 CPU).
* conv2d_bwd_filter pinned: finite differences, adjoint identity, full-window
                    VALID conv = outer-product matmul, torch autograd.
* conv2d_bwd_filter_at  pinned: torch autograd at the selected entries.
* bias_relu_fwd/bwd pinned: finite differences off the kink, numpy column sums.
* maxpool_fwd       pinned: reshape-max for non-overlapping windows, brute-force
                    numpy argmax (first maximum) for any window, planted ties.
* maxpool_bwd       pinned: mass conservation, finite differences at tie-free
                    points, support only on argmax positions.
* apply_sgd         pinned: closed form and a surrogate-loss decrease.
* apply_momentum    pinned: constant-gradient closed forms (classical and nesterov),
                    momentum 0 = SGD, the velocity as a geometric sum of past gradients.
* apply_adam        pinned: constant-gradient closed form, first-step form, the moments
                    as bias-weighted sums of past gradients, beta = 0 forms.
* softmax_xent      pinned: library cross-entropy and its autograd gradient, uniform-logit
                    closed form, invariance to a per-row shift of 1000 (overflow),
                    zero gradient row sums, NaN rows for out-of-range labels.
* sampled_softmax   pinned: with every class sampled (the true one removed as an accidental
                    hit) it is the full softmax cross-entropy of the logits minus log q;
                    a constant shift of log q changes nothing; finite differences in h,
                    W and b.
* step (net.py)     pinned: finite differences of the whole single-layer loss
                    and the exact first-order decrease of a piecewise-linear net.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)
_i = ctypes.c_int
_l = ctypes.c_int64


def build(force: bool = False, lib_path: str = _LIB, extra_flags=()) -> str:
    """Compile oracle.c into a shared library with gcc (-O2 -fopenmp)."""
    if force or not os.path.exists(lib_path) or os.path.getmtime(lib_path) < os.path.getmtime(_SRC):
        tmp = lib_path + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", *extra_flags,
               "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, lib_path)
    return lib_path


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        _declare(lib)
        _lib = lib
    return _lib


def _declare(lib):
    lib.orc_num_threads.restype = _i
    lib.orc_set_num_threads.argtypes = [_i]
    lib.orc_out_len.restype = _i
    lib.orc_out_len.argtypes = [_i] * 5
    lib.orc_conv2d_fwd.argtypes = [_dp, _i, _i, _i, _i, _dp, _i, _i, _i, _i, _i, _i, _i, _dp, _i, _i]
    lib.orc_conv2d_bwd_input.argtypes = [_dp, _i, _i, _i, _i, _dp, _i, _i, _i, _i, _i, _i,
                                         _dp, _i, _i, _i, _i]
    lib.orc_conv2d_bwd_filter.argtypes = [_dp, _i, _i, _i, _i, _dp, _i, _i, _i,
                                          _i, _i, _i, _i, _i, _i, _dp]
    lib.orc_conv2d_bwd_filter_at.argtypes = [_dp, _i, _i, _i, _i, _dp, _i, _i, _i, _i, _i, _i, _i, _i, _i,
                                             ctypes.POINTER(ctypes.c_int64), _l, _dp]
    lib.orc_bias_relu_fwd.argtypes = [_dp, _dp, _l, _i, _dp]
    lib.orc_bias_relu_bwd.argtypes = [_dp, _dp, _l, _i, _dp, _dp]
    lib.orc_maxpool_fwd.argtypes = [_dp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _dp, _ip, _i, _i]
    lib.orc_maxpool_bwd.argtypes = [_dp, _ip, _l, _dp, _l, _i]
    lib.orc_apply_sgd.argtypes = [_dp, _dp, _l, ctypes.c_double]
    lib.orc_apply_momentum.argtypes = [_dp, _dp, _dp, _l, ctypes.c_double, ctypes.c_double, ctypes.c_int]
    lib.orc_sampled_softmax.argtypes = [_dp, _dp, _dp, _ip, _ip, _dp, _dp, _l, _i, _i, _i, ctypes.c_double, _dp,
                                        _dp, _dp, _dp]
    lib.orc_softmax_xent.argtypes = [_dp, _dp, _ip, _l, _i, ctypes.c_double, _dp, _dp]
    lib.orc_apply_adam.argtypes = [_dp, _dp, _dp, _dp, _l, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                   ctypes.c_double, ctypes.c_int]


def use_library(path: str):
    """Load the oracle from another build of oracle.c (used by mutation tests)."""
    global _lib
    lib = ctypes.CDLL(path)
    _declare(lib)
    _lib = lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return a.ctypes.data_as(_dp)


def num_threads() -> int:
    return _load().orc_num_threads()


def set_num_threads(n: int):
    _load().orc_set_num_threads(int(n))


def out_len(n, k, s, p0, p1) -> int:
    return _load().orc_out_len(n, k, s, p0, p1)


def conv2d_fwd(x, w, stride, pads):
    """y = x (*) w, cross-correlation; x NHWC, w HWIO, pads = (top, bottom, left, right)."""
    lib = _load()
    x, w = _f64(x), _f64(w)
    N, H, W, C = x.shape
    KH, KW, Ci, K = w.shape
    assert Ci == C
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    pt, pb, pl, pr = pads
    OH, OW = out_len(H, KH, sh, pt, pb), out_len(W, KW, sw, pl, pr)
    assert OH >= 1 and OW >= 1
    y = np.empty((N, OH, OW, K))
    lib.orc_conv2d_fwd(_ptr(x), N, H, W, C, _ptr(w), KH, KW, K, sh, sw, pt, pl, _ptr(y), OH, OW)
    return y


def conv2d_bwd_input(dy, w, input_shape, stride, pads, dx=None, beta=0):
    """dx = conv2d_fwd^T(dy) for an input of ``input_shape`` (NHWC)."""
    lib = _load()
    dy, w = _f64(dy), _f64(w)
    N, OH, OW, K = dy.shape
    KH, KW, C, K2 = w.shape
    assert K2 == K
    Nx, H, W, Cx = input_shape
    assert Nx == N and Cx == C
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    pt, pb, pl, pr = pads
    assert OH == out_len(H, KH, sh, pt, pb) and OW == out_len(W, KW, sw, pl, pr)
    if beta:
        out = _f64(dx).copy()
    else:
        out = np.empty((N, H, W, C))
    lib.orc_conv2d_bwd_input(_ptr(dy), N, OH, OW, K, _ptr(w), KH, KW, sh, sw, pt, pl,
                             _ptr(out), H, W, C, 1 if beta else 0)
    return out


def conv2d_bwd_filter(x, dy, kernel_hw, stride, pads):
    """dW[kh,kw,ci,co] = sum_{n,oh,ow} X[...] * dy[n,oh,ow,co]."""
    lib = _load()
    x, dy = _f64(x), _f64(dy)
    N, H, W, C = x.shape
    N2, OH, OW, K = dy.shape
    assert N2 == N
    KH, KW = kernel_hw
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    pt, pb, pl, pr = pads
    assert OH == out_len(H, KH, sh, pt, pb) and OW == out_len(W, KW, sw, pl, pr)
    dw = np.empty((KH, KW, C, K))
    lib.orc_conv2d_bwd_filter(_ptr(x), N, H, W, C, _ptr(dy), OH, OW, K, KH, KW, sh, sw, pt, pl,
                              _ptr(dw))
    return dw


def conv2d_bwd_filter_at(x, dy, kernel_hw, stride, pads, flat_idx):
    """Selected entries dW.flat[flat_idx] of conv2d_bwd_filter (HWIO flat indices)."""
    lib = _load()
    x, dy = _f64(x), _f64(dy)
    N, H, W, C = x.shape
    N2, OH, OW, K = dy.shape
    assert N2 == N
    KH, KW = kernel_hw
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    pt, pb, pl, pr = pads
    assert OH == out_len(H, KH, sh, pt, pb) and OW == out_len(W, KW, sw, pl, pr)
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    assert idx.min() >= 0 and idx.max() < KH * KW * C * K
    out = np.empty(idx.size)
    lib.orc_conv2d_bwd_filter_at(_ptr(x), N, H, W, C, _ptr(dy), OH, OW, K, KH, KW, sh, sw, pt, pl,
                                 idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), idx.size, _ptr(out))
    return out


def bias_relu_fwd(pre, b):
    lib = _load()
    pre, b = _f64(pre), _f64(b)
    C = pre.shape[-1]
    assert b.shape == (C,)
    y = np.empty_like(pre)
    lib.orc_bias_relu_fwd(_ptr(pre), _ptr(b), pre.size // C, C, _ptr(y))
    return y


def bias_relu_bwd(y, dy):
    """Returns (dpre, db)."""
    lib = _load()
    y, dy = _f64(y), _f64(dy)
    assert y.shape == dy.shape
    C = y.shape[-1]
    dpre = np.empty_like(dy)
    db = np.empty(C)
    lib.orc_bias_relu_bwd(_ptr(y), _ptr(dy), y.size // C, C, _ptr(dpre), _ptr(db))
    return dpre, db


def maxpool_fwd(x, kernel_hw, stride, pads):
    """Returns (y, argmax int32 flat NHWC index into x)."""
    lib = _load()
    x = _f64(x)
    N, H, W, C = x.shape
    KH, KW = kernel_hw
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    pt, pb, pl, pr = pads
    OH, OW = out_len(H, KH, sh, pt, pb), out_len(W, KW, sw, pl, pr)
    y = np.empty((N, OH, OW, C))
    am = np.empty((N, OH, OW, C), dtype=np.int32)
    lib.orc_maxpool_fwd(_ptr(x), N, H, W, C, KH, KW, sh, sw, pt, pl, _ptr(y),
                        am.ctypes.data_as(_ip), OH, OW)
    return y, am


def maxpool_bwd(dy, argmax, x_shape, dx=None, beta=0):
    lib = _load()
    dy = _f64(dy)
    am = np.ascontiguousarray(argmax, dtype=np.int32)
    assert am.shape == dy.shape
    if beta:
        out = _f64(dx).copy()
    else:
        out = np.empty(tuple(x_shape))
    lib.orc_maxpool_bwd(_ptr(dy), am.ctypes.data_as(_ip), dy.size, _ptr(out), out.size,
                        1 if beta else 0)
    return out


def apply_sgd(var, grad, lr):
    """Returns var - lr * grad (fp64), leaving the inputs untouched."""
    lib = _load()
    out = _f64(var).copy()
    g = _f64(grad)
    assert out.shape == g.shape
    lib.orc_apply_sgd(_ptr(out), _ptr(g), out.size, float(lr))
    return out


def apply_momentum(var, accum, grad, lr, momentum, nesterov=False):
    """One Momentum update (fp64); returns (var', accum'), leaving the inputs untouched."""
    lib = _load()
    out, acc, g = _f64(var).copy(), _f64(accum).copy(), _f64(grad)
    assert out.shape == acc.shape == g.shape
    lib.orc_apply_momentum(_ptr(out), _ptr(acc), _ptr(g), out.size, float(lr), float(momentum), int(bool(nesterov)))
    return out, acc


def apply_adam(var, m, v, grad, lr, beta1, beta2, epsilon, t):
    """One Adam update at step t >= 1 (fp64); returns (var', m', v'), inputs untouched."""
    lib = _load()
    out, mm, vv, g = _f64(var).copy(), _f64(m).copy(), _f64(v).copy(), _f64(grad)
    assert out.shape == mm.shape == vv.shape == g.shape and t >= 1
    lib.orc_apply_adam(_ptr(out), _ptr(mm), _ptr(vv), _ptr(g), out.size, float(lr), float(beta1), float(beta2),
                       float(epsilon), int(t))
    return out, mm, vv


def softmax_xent(logits, labels, scale=1.0, bias=None):
    """Softmax cross-entropy of (n, c) logits (+ bias[c]) against int labels; returns
    (loss per row, scale * (softmax - onehot)) in fp64."""
    lib = _load()
    z = _f64(logits)
    assert z.ndim == 2
    n, c = z.shape
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    assert lab.shape == (n,)
    b = None if bias is None else _f64(bias)
    assert b is None or b.shape == (c,)
    loss = np.zeros(n)
    dz = np.zeros((n, c))
    lib.orc_softmax_xent(_ptr(z), None if b is None else _ptr(b), lab.ctypes.data_as(_ip), n, c, float(scale),
                         _ptr(loss), _ptr(dz))
    return loss, dz


def sampled_softmax(h, W, b, labels, sampled, lq_true, lq_sampled, scale=1.0):
    """Sampled softmax cross-entropy; returns (loss per row, dh, dW dense, db dense) in fp64."""
    lib = _load()
    h, W, b = _f64(h), _f64(W), _f64(b)
    n, d = h.shape
    v = W.shape[0]
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    smp = np.ascontiguousarray(sampled, dtype=np.int32)
    lqt, lqs = _f64(lq_true), _f64(lq_sampled)
    m = smp.size
    assert W.shape == (v, d) and b.shape == (v,) and lab.shape == (n,) and lqt.shape == (n,) and lqs.shape == (m,)
    assert np.all((lab >= 0) & (lab < v)) and np.all((smp >= 0) & (smp < v))
    loss, dh, dW, db = np.zeros(n), np.zeros((n, d)), np.zeros((v, d)), np.zeros(v)
    lib.orc_sampled_softmax(_ptr(h), _ptr(W), _ptr(b), lab.ctypes.data_as(_ip), smp.ctypes.data_as(_ip),
                            _ptr(lqt), _ptr(lqs), n, d, v, m, float(scale), _ptr(loss), _ptr(dh), _ptr(dW),
                            _ptr(db))
    return loss, dh, dW, db
