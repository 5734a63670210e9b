"""Python binding of the tfk_* C ABI over torch device tensors.

Argument marshalling only: every step runs in the HIP kernels of libtfk.so.
Tensors are NHWC torch tensors on the GPU; a 4-D tensor may be a channel
slice of a wider NHWC buffer (its pixel stride is passed to the library).
Filters are dense HWIO.  Every call is enqueued on ``stream`` (default: torch's
current stream) and raises TfkError on a non-OK status.  There is no CPU path.
"""
from __future__ import annotations

import ctypes
from typing import NamedTuple, Optional, Sequence, Tuple

import torch

from ._lib import Nhwc, TfkError, Window, TFK_BF16, TFK_F32, check, load

__all__ = ["conv2d_fwd", "conv2d_fwd_bias_relu", "conv2d_bwd_input", "conv2d_bwd_filter", "conv2d_workspace_bytes", "bias_relu_fwd",
           "bias_relu_bwd", "bias_relu_bwd_workspace_bytes", "maxpool_fwd", "maxpool_bwd", "maxpool_bwd_relu_bwd", "apply_sgd",
           "apply_sgd_multi", "apply_momentum", "apply_adam", "softmax_xent",
           "gather_rows_t", "sampled_softmax_xent", "scatter_apply_sgd", "stream_wait", "Program", "out_len", "nhwc",
           "window", "TfkError", "abi_version", "DeferredBias", "bias_grad_finish"]


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return TFK_F32
    if t.dtype == torch.bfloat16:
        return TFK_BF16
    raise TypeError("tfk supports float32 and bfloat16 tensors, got %s" % t.dtype)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> ctypes.c_void_p:
    return ctypes.c_void_p(t.data_ptr() if t is not None else 0)


def nhwc(t: torch.Tensor) -> Nhwc:
    """Describes a 4-D NHWC tensor (or a channel slice of one) for the library."""
    if t.dim() != 4:
        raise ValueError("expected a 4-D NHWC tensor, got shape %s" % (tuple(t.shape),))
    n, h, w, c = t.shape
    s0, s1, s2, s3 = t.stride()
    if n * h * w > 0:
        ps = s2 if w > 1 else (s1 if h > 1 else (s0 if n > 1 else c))
        if s3 != 1 or (w > 1 and s2 != ps) or (h > 1 and s1 != w * ps) or (n > 1 and s0 != h * w * ps):
            raise ValueError("tensor is not an NHWC view with unit channel stride: strides %s" % (t.stride(),))
    else:
        ps = c
    return Nhwc(n, h, w, c, ps)


def window(kh, kw, stride, pads) -> Window:
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    pt, pb, pl, pr = pads
    return Window(kh, kw, sh, sw, pt, pb, pl, pr)


def out_len(n, k, s, p0, p1) -> int:
    return (n + p0 + p1 - k) // s + 1


def abi_version() -> int:
    return load().tfk_abi_version()


def _empty(stream, *args, **kw) -> torch.Tensor:
    """torch.empty on the stream the op is enqueued on: the caching allocator then hands the
    memory, once freed, only to later work on that same stream (a temporary freed on return
    cannot be reused by another stream while the kernel still runs)."""
    if stream is None:
        return torch.empty(*args, **kw)
    with torch.cuda.stream(stream):
        return torch.empty(*args, **kw)


def _empty_like(stream, t: torch.Tensor) -> torch.Tensor:
    return _empty(stream, t.shape, dtype=t.dtype, device=t.device)


def _ws(nbytes: int, device, stream=None) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return None
    return _empty(stream, (nbytes + 15) // 16 * 16, dtype=torch.uint8, device=device)


# ----------------------------------------------------------------------------- convolution
def conv2d_workspace_bytes(op: int, x: torch.Tensor, cout: int, kh, kw, stride, pads) -> int:
    return load().tfk_conv2d_workspace_bytes(op, nhwc(x), cout, window(kh, kw, stride, pads), _dt(x))


def _conv_fwd(x, w, bias, stride, pads, y, ws, stream):
    lib = load()
    kh, kw, cin, cout = w.shape
    win = window(kh, kw, stride, pads)
    need = lib.tfk_conv2d_workspace_bytes(0, nhwc(x), cout, win, _dt(x))
    if need and (ws is None or ws.numel() < need):
        ws = _ws(need, x.device, stream)
    if y is None:
        n, h, ww, _ = x.shape
        y = _empty(stream, (n, out_len(h, kh, win.stride_h, pads[0], pads[1]),
                         out_len(ww, kw, win.stride_w, pads[2], pads[3]), cout), dtype=x.dtype, device=x.device)
    if w.dtype != x.dtype or y.dtype != x.dtype:
        raise TypeError("x, w and y must share one dtype")
    wsp = _ptr(ws) if need else None
    if bias is None:
        check(lib.tfk_conv2d_fwd(_ptr(x), nhwc(x), _ptr(w), cout, win, _dt(x), _ptr(y), nhwc(y), wsp, need,
                                 _stream(stream)))
    else:
        if bias.dtype != torch.float32 or bias.numel() != cout or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous float32 vector of cout values")
        check(lib.tfk_conv2d_fwd_bias_relu(_ptr(x), nhwc(x), _ptr(w), cout, _ptr(bias), win, _dt(x), _ptr(y),
                                           nhwc(y), wsp, need, _stream(stream)))
    return y


def conv2d_fwd(x, w, stride, pads, y=None, ws=None, stream=None):
    """y = x (*) w (cross-correlation).  x NHWC, w HWIO, pads (top, bottom, left, right)."""
    return _conv_fwd(x, w, None, stride, pads, y, ws, stream)


def conv2d_fwd_bias_relu(x, w, bias, stride, pads, y=None, ws=None, stream=None):
    """y = max(x (*) w + bias, 0) in one kernel (bias fp32, one value per output channel)."""
    return _conv_fwd(x, w, bias, stride, pads, y, ws, stream)


def conv2d_fwd_bias_relu_maxpool(x, w, bias, stride, pads, pool_hw, pool_stride, pool_pads=(0, 0, 0, 0), y=None,
                                 py=None, taps=None, ws=None, stream=None):
    """y = max(x (*) w + bias, 0) and its max-pool (py, uint8 window taps) in one call; one kernel
    where the convolution's row bands hold whole pool windows.  Returns (y, py, taps)."""
    lib = load()
    kh, kw, cin, cout = w.shape
    win = window(kh, kw, stride, pads)
    need = lib.tfk_conv2d_workspace_bytes(0, nhwc(x), cout, win, _dt(x))
    if need and (ws is None or ws.numel() < need):
        ws = _ws(need, x.device, stream)
    n, h, ww, _ = x.shape
    oh = out_len(h, kh, win.stride_h, pads[0], pads[1])
    ow = out_len(ww, kw, win.stride_w, pads[2], pads[3])
    if y is None:
        y = _empty(stream, (n, oh, ow, cout), dtype=x.dtype, device=x.device)
    pkh, pkw = pool_hw
    pwin = window(pkh, pkw, pool_stride, pool_pads)
    poh = out_len(oh, pkh, pwin.stride_h, pool_pads[0], pool_pads[1])
    pow_ = out_len(ow, pkw, pwin.stride_w, pool_pads[2], pool_pads[3])
    if py is None:
        py = _empty(stream, (n, poh, pow_, cout), dtype=x.dtype, device=x.device)
    if taps is None:
        taps = _empty(stream, (n, poh, pow_, cout), dtype=torch.uint8, device=x.device)
    if not (w.dtype == y.dtype == py.dtype == x.dtype):
        raise TypeError("x, w, y and py must share one dtype")
    if taps.dtype != torch.uint8 or not taps.is_contiguous():
        raise ValueError("taps must be a dense uint8 tensor")
    if bias.dtype != torch.float32 or bias.numel() != cout or not bias.is_contiguous():
        raise ValueError("bias must be a contiguous float32 vector of cout values")
    check(lib.tfk_conv2d_fwd_bias_relu_maxpool(_ptr(x), nhwc(x), _ptr(w), cout, _ptr(bias), win, _dt(x), _ptr(y),
                                               nhwc(y), pwin, _ptr(py), nhwc(py), _ptr(taps),
                                               _ptr(ws) if need else None, need, _stream(stream)))
    return y, py, taps


def conv2d_bwd_input(dy, w, dx, stride, pads, beta=0.0, ws=None, stream=None):
    """dx (= or +=) conv2d_fwd^T(dy).  dx gives the forward input's shape (it is written)."""
    lib = load()
    kh, kw, cin, cout = w.shape
    if not (w.dtype == dy.dtype == dx.dtype):
        raise TypeError("dy, w and dx must share one dtype")
    win = window(kh, kw, stride, pads)
    need = lib.tfk_conv2d_workspace_bytes(1, nhwc(dx), cout, win, _dt(dx))
    if need and (ws is None or ws.numel() < need):
        ws = _ws(need, dx.device, stream)
    check(lib.tfk_conv2d_bwd_input(_ptr(dy), nhwc(dy), _ptr(w), win, _dt(dy), _ptr(dx), nhwc(dx), float(beta),
                                   _ptr(ws) if need else None, need, _stream(stream)))
    return dx


def conv2d_bwd_input_relu_bwd(dy, w, y, dpre, stride, pads, dbias=None, ws=None, stream=None, defer=False,
                              beta=0.0):
    """dpre = (y > 0) * (beta * dpre + conv2d_fwd^T(dy)), dbias = column sums of dpre (fp32): the
    input gradient fused with the ReLU backward of the layers that produced the input (y, dpre: its
    view); beta = 1 adds it to the gradient the input's other readers stored in dpre.
    defer=True: returns (dpre, DeferredBias) instead, the partials left in ws (see bias_grad_finish)."""
    lib = load()
    kh, kw, cin, cout = w.shape
    if not (w.dtype == dy.dtype == y.dtype == dpre.dtype):
        raise TypeError("dy, w, y and dpre must share one dtype")
    d_y, d_p = nhwc(y), nhwc(dpre)
    if (d_y.n, d_y.h, d_y.w, d_y.c, d_y.pixel_stride) != (d_p.n, d_p.h, d_p.w, d_p.c, d_p.pixel_stride):
        raise ValueError("y and dpre must share one view (extents and pixel stride)")
    win = window(kh, kw, stride, pads)
    need = lib.tfk_conv2d_workspace_bytes(3, d_p, cout, win, _dt(y))
    if defer:
        _need_ws(ws, need)
        dbias = None
    elif dbias is None:
        dbias = _empty(stream, cin, dtype=torch.float32, device=y.device)
    if need and (ws is None or ws.numel() < need):
        ws = _ws(need, y.device, stream)
    check(lib.tfk_conv2d_bwd_input_relu_bwd(_ptr(dy), nhwc(dy), _ptr(w), win, _dt(dy), _ptr(y), _ptr(dpre), d_p,
                                            float(beta), _ptr(dbias), _ptr(ws) if need else None, need,
                                            _stream(stream)))
    return dpre, (_deferred(lib, cin) if defer else dbias)


def conv2d_bwd_filter(x, dy, kernel_hw, stride, pads, dw=None, ws=None, stream=None):
    """dW (fp32 HWIO) = sum over pixels of x-gather * dy."""
    lib = load()
    kh, kw = kernel_hw
    cout = dy.shape[3]
    if dw is None:
        dw = _empty(stream, (kh, kw, x.shape[3], cout), dtype=torch.float32, device=x.device)
    if dy.dtype != x.dtype or dw.dtype != torch.float32:
        raise TypeError("x and dy share one dtype; dw is float32")
    win = window(kh, kw, stride, pads)
    need = lib.tfk_conv2d_workspace_bytes(2, nhwc(x), cout, win, _dt(x))
    if ws is None or ws.numel() < need:
        ws = _ws(need, x.device, stream)
    check(lib.tfk_conv2d_bwd_filter(_ptr(x), nhwc(x), _ptr(dy), nhwc(dy), win, _dt(x), _ptr(dw), _ptr(ws),
                                    need, _stream(stream)))
    return dw


def conv2d_bwd_filter_noalloc(x, dy, kernel_hw, stride, pads, dw, stream=None):
    """conv2d_bwd_filter with the library's own device scratch in place of a workspace: the call
    allocates nothing (dw must be given).  Calls that overlap in time on one GPU race."""
    kh, kw = kernel_hw
    cout = dy.shape[3]
    if dy.dtype != x.dtype or dw.dtype != torch.float32:
        raise TypeError("x and dy share one dtype; dw is float32")
    if tuple(dw.shape) != (kh, kw, x.shape[3], cout) or not dw.is_contiguous():
        raise ValueError("dw must be a contiguous float32 HWIO tensor")
    check(load().tfk_conv2d_bwd_filter_noalloc(_ptr(x), nhwc(x), _ptr(dy), nhwc(dy), window(kh, kw, stride, pads),
                                               _dt(x), _ptr(dw), _stream(stream)))
    return dw


# ----------------------------------------------------------------------------- bias + relu
def bias_relu_fwd(y, bias, stream=None):
    """In place: y <- max(y + bias, 0)."""
    check(load().tfk_bias_relu_fwd(_ptr(y), nhwc(y), _ptr(bias), _dt(y), _stream(stream)))
    return y


def bias_relu_bwd_workspace_bytes(y) -> int:
    return load().tfk_bias_relu_bwd_workspace_bytes(nhwc(y), _dt(y))


def bias_relu_bwd(y, dy, dpre=None, dbias=None, ws=None, stream=None, defer=False):
    """dpre = dy * (y > 0) (dpre may be dy), dbias = column sums of dpre (fp32).  With y None
    (a bias-only layer) dpre = dy and dbias = column sums of dy.  defer=True: returns
    (dpre, DeferredBias) instead, the partials left in ws (see bias_grad_finish)."""
    lib = load()
    if dpre is None:
        dpre = _empty_like(stream, dy)
    view = y if y is not None else dy
    need = lib.tfk_bias_relu_bwd_workspace_bytes(nhwc(view), _dt(view))
    if defer:
        _need_ws(ws, need)
        dbias = None
    elif dbias is None:
        dbias = _empty(stream, dy.shape[3], dtype=torch.float32, device=dy.device)
    if ws is None or ws.numel() < need:
        ws = _ws(need, dy.device, stream)
    d_y, d_dy, d_dp = nhwc(view), nhwc(dy), nhwc(dpre)
    if (d_y.pixel_stride, d_y.c) != (d_dy.pixel_stride, d_dy.c) or (d_y.pixel_stride, d_y.c) != (d_dp.pixel_stride, d_dp.c):
        raise ValueError("y, dy and dpre must share one view (extents and pixel stride)")
    check(lib.tfk_bias_relu_bwd(_ptr(y), _ptr(dy), d_y, _ptr(dpre), _ptr(dbias), _dt(dy), _ptr(ws), need,
                                _stream(stream)))
    return dpre, (_deferred(lib, dy.shape[3]) if defer else dbias)


def softmax_xent(logits, labels, scale, bias=None, loss=None, dlogits=None, stream=None):
    """Softmax cross-entropy of contiguous logits (rows of the last dimension) + bias against int32
    labels: returns (per-row loss fp32, dlogits = scale * (softmax - onehot)); dlogits may be logits."""
    if not logits.is_contiguous():
        raise ValueError("logits must be contiguous")
    c = logits.shape[-1]
    n = logits.numel() // c if c else 0
    if labels.dtype != torch.int32 or labels.numel() != n:
        raise ValueError("labels must be int32, one per row")
    if bias is not None and (bias.dtype != torch.float32 or bias.numel() != c):
        raise ValueError("bias must be float32 [c]")
    if loss is None:
        loss = _empty(stream, n, dtype=torch.float32, device=logits.device)
    if dlogits is None:
        dlogits = _empty_like(stream, logits)
    if dlogits.dtype != logits.dtype or dlogits.numel() != logits.numel() or not dlogits.is_contiguous():
        raise ValueError("dlogits must be a contiguous tensor like logits")
    check(load().tfk_softmax_xent(_ptr(logits), _dt(logits), n, c, _ptr(bias), _ptr(labels), float(scale),
                                  _ptr(loss), _ptr(dlogits), _stream(stream)))
    return loss, dlogits


# ----------------------------------------------------------------------------- max-pool
def maxpool_fwd(x, kernel_hw, stride, pads, y=None, argmax=None, stream=None, taps=False):
    """Returns (y, argmax).  argmax is int32 dense NHWC indices into x, or with ``taps`` uint8
    window taps kh * KW + kw (a quarter of the bytes); the backward ops accept either."""
    lib = load()
    kh, kw = kernel_hw
    win = window(kh, kw, stride, pads)
    n, h, w, c = x.shape
    oh = out_len(h, kh, win.stride_h, pads[0], pads[1])
    ow = out_len(w, kw, win.stride_w, pads[2], pads[3])
    if y is None:
        y = _empty(stream, (n, oh, ow, c), dtype=x.dtype, device=x.device)
    if argmax is None:
        argmax = _empty(stream, (n, oh, ow, c), dtype=torch.uint8 if taps else torch.int32, device=x.device)
    fn = _argmax_fn(lib, "tfk_maxpool_fwd", argmax)
    check(fn(_ptr(x), nhwc(x), win, _dt(x), _ptr(y), nhwc(y), _ptr(argmax), _stream(stream)))
    return y, argmax


def _argmax_fn(lib, name, argmax):
    """The entry point for this argmax format: int32 dense indices, or uint8 taps (``_taps``)."""
    if not argmax.is_contiguous() or argmax.dtype not in (torch.int32, torch.uint8):
        raise ValueError("argmax must be a dense int32 (indices) or uint8 (taps) tensor")
    return getattr(lib, name + ("_taps" if argmax.dtype == torch.uint8 else ""))


def maxpool_bwd(dy, argmax, dx, kernel_hw, stride, pads, beta=0.0, stream=None):
    kh, kw = kernel_hw
    fn = _argmax_fn(load(), "tfk_maxpool_bwd", argmax)
    check(fn(_ptr(dy), _ptr(argmax), nhwc(dy), window(kh, kw, stride, pads), _dt(dy), _ptr(dx), nhwc(dx),
             float(beta), _stream(stream)))
    return dx


def maxpool_bwd_relu_bwd(dy, argmax, y, dpre, kernel_hw, stride, pads, beta=0.0, dbias=None, ws=None, stream=None,
                         py=None, defer=False):
    """dpre = (y > 0) * (beta * dpre + max-pool gradient of dy), dbias = column sums of dpre (fp32).

    y is the pool input (the ReLU output); dpre has its shape and view.  py (optional) is the
    pool's output: with beta = 0 the mask is taken from it per window and y is not read (y may
    then be None).  defer=True: returns (dpre, DeferredBias) instead, the partials left in ws
    (see bias_grad_finish).
    """
    lib = load()
    kh, kw = kernel_hw
    fn = _argmax_fn(lib, "tfk_maxpool_bwd_relu_bwd", argmax)
    d_p = nhwc(dpre)
    if y is not None:
        d_y = nhwc(y)
        if (d_y.n, d_y.h, d_y.w, d_y.c, d_y.pixel_stride) != (d_p.n, d_p.h, d_p.w, d_p.c, d_p.pixel_stride):
            raise ValueError("y and dpre must share one view (extents and pixel stride)")
    pys = 0
    if py is not None:
        if tuple(py.shape) != tuple(dy.shape) or py.dtype != dy.dtype:
            raise ValueError("py must have dy's shape and element type")
        pys = nhwc(py).pixel_stride
    need = lib.tfk_bias_relu_bwd_workspace_bytes(d_p, _dt(dpre))
    if defer:
        _need_ws(ws, need)
        dbias = None
    elif dbias is None:
        dbias = _empty(stream, dpre.shape[3], dtype=torch.float32, device=dpre.device)
    if ws is None or ws.numel() < need:
        ws = _ws(need, dpre.device, stream)
    check(fn(_ptr(dy), _ptr(argmax), nhwc(dy), window(kh, kw, stride, pads), _dt(dy),
             _ptr(y), _ptr(py), pys, _ptr(dpre), d_p,
             float(beta), _ptr(dbias), _ptr(ws), need, _stream(stream)))
    return dpre, (_deferred(lib, dpre.shape[3]) if defer else dbias)


# ----------------------------------------------------------------------------- deferred bias gradients
class DeferredBias(NamedTuple):
    """Where a call made with defer=True left its bias-gradient partials: inside the workspace it
    was given, which must stay untouched until bias_grad_finish has run."""
    part: int          # device address
    rows: int          # partials per channel
    channels: int


def _need_ws(ws, need):
    if ws is None or ws.numel() < need:
        raise ValueError("defer=True needs a caller workspace of at least %d bytes (the partials stay in it)" % need)


def _deferred(lib, channels) -> DeferredBias:
    part, rows = ctypes.c_void_p(), ctypes.c_int32()
    check(lib.tfk_last_bias_partials(ctypes.byref(part), ctypes.byref(rows)))
    return DeferredBias(part.value or 0, rows.value, int(channels))


def bias_grad_finish(jobs, stream=None):
    """For every (DeferredBias, dbias) in jobs: dbias = the fixed-order per-channel sums of the
    partials its deferred call left (the same bits as the call given dbias), in one launch."""
    lib = load()
    n = len(jobs)
    for d, db in jobs:
        if db.dtype != torch.float32 or not db.is_contiguous() or db.numel() != d.channels:
            raise ValueError("dbias must be contiguous float32 with one value per channel")
    parts = (ctypes.c_void_p * max(n, 1))(*[d.part for d, _ in jobs])
    rows = (ctypes.c_int32 * max(n, 1))(*[d.rows for d, _ in jobs])
    chans = (ctypes.c_int32 * max(n, 1))(*[d.channels for d, _ in jobs])
    dbs = (ctypes.c_void_p * max(n, 1))(*[db.data_ptr() for _, db in jobs])
    check(lib.tfk_bias_grad_finish(n, parts, rows, chans, dbs, _stream(stream)))


# ----------------------------------------------------------------------------- update
def apply_sgd(var, grad, lr, shadow=None, stream=None):
    """In place: var <- fma(-lr, grad, var); shadow (bf16) <- bf16(var) if given."""
    if var.dtype != torch.float32 or grad.dtype != torch.float32:
        raise TypeError("var and grad are float32")
    if not (var.is_contiguous() and grad.is_contiguous()) or var.numel() != grad.numel():
        raise ValueError("var and grad must be contiguous with the same size")
    if shadow is not None and (shadow.dtype != torch.bfloat16 or shadow.numel() != var.numel()
                               or not shadow.is_contiguous()):
        raise ValueError("shadow must be a contiguous bfloat16 tensor of var's size")
    check(load().tfk_apply_sgd(_ptr(var), _ptr(grad), var.numel(), float(lr), _ptr(shadow), _stream(stream)))
    return var


def _check_update(var, grad, slots, shadow):
    for t in (var, grad, *slots):
        if t.dtype != torch.float32:
            raise TypeError("var, grad and the optimizer slots are float32")
        if not t.is_contiguous() or t.numel() != var.numel():
            raise ValueError("var, grad and the optimizer slots must be contiguous with the same size")
    if shadow is not None and (shadow.dtype != torch.bfloat16 or shadow.numel() != var.numel()
                               or not shadow.is_contiguous()):
        raise ValueError("shadow must be a contiguous bfloat16 tensor of var's size")


def apply_momentum(var, accum, grad, lr, momentum, nesterov=False, shadow=None, stream=None):
    """In place: accum <- momentum * accum + grad; var <- var - lr * accum (or, look-ahead form,
    var <- var - lr * (grad + momentum * accum)); shadow (bf16) <- bf16(var) if given."""
    _check_update(var, grad, (accum,), shadow)
    check(load().tfk_apply_momentum(_ptr(var), _ptr(accum), _ptr(grad), var.numel(), float(lr), float(momentum),
                                    int(bool(nesterov)), _ptr(shadow), _stream(stream)))
    return var


def apply_adam(var, m, v, grad, lr, beta1, beta2, epsilon, t, shadow=None, stream=None):
    """In place, Adam step t >= 1: the moments m and v and var; shadow (bf16) <- bf16(var) if given."""
    _check_update(var, grad, (m, v), shadow)
    check(load().tfk_apply_adam(_ptr(var), _ptr(m), _ptr(v), _ptr(grad), var.numel(), float(lr), float(beta1),
                                float(beta2), float(epsilon), int(t), _ptr(shadow), _stream(stream)))
    return var


def apply_sgd_multi(vars_: Sequence[torch.Tensor], grads: Sequence[torch.Tensor], lr,
                    shadows: Optional[Sequence[Optional[torch.Tensor]]] = None, stream=None):
    count = len(vars_)
    VP = ctypes.c_void_p * max(count, 1)
    NS = ctypes.c_int64 * max(count, 1)
    v = VP(*[t.data_ptr() for t in vars_])
    g = VP(*[t.data_ptr() for t in grads])
    ns = NS(*[t.numel() for t in vars_])
    sh = None
    if shadows is not None:
        sh = VP(*[(t.data_ptr() if t is not None else 0) for t in shadows])
    check(load().tfk_apply_sgd_multi(count, v, g, ns, float(lr), sh, _stream(stream)))


# ----------------------------------------------------------------------------- sampled softmax
def gather_rows_t(table, idx, u_pad, out_t=None, stream=None):
    """out_t (d x u_pad) = table[idx]^T, zero past len(idx); table (rows x d) contiguous."""
    rows, d = table.shape
    u = idx.numel()
    if idx.dtype != torch.int32 or not table.is_contiguous():
        raise ValueError("idx must be int32 and table contiguous")
    if out_t is None:
        out_t = _empty(stream, d, u_pad, dtype=table.dtype, device=table.device)
    if out_t.dtype != table.dtype or out_t.numel() != d * u_pad or not out_t.is_contiguous():
        raise ValueError("out_t must be a contiguous d x u_pad tensor of table's type")
    check(load().tfk_gather_rows_t(_ptr(table), _dt(table), rows, d, _ptr(idx), u, u_pad, _ptr(out_t),
                                   _stream(stream)))
    return out_t


def sampled_softmax_xent(z, u, m, true_pos, lq_true, lq_sampled, scale, bias_c=None, loss=None, dz=None,
                         stream=None):
    """Cross-entropy over candidate logits z (n x u_pad): returns (loss per row, dz)."""
    n, u_pad = z.shape[0], z.shape[-1]
    if not z.is_contiguous() or z.numel() != n * u_pad:
        raise ValueError("z must be contiguous n x u_pad")
    if loss is None:
        loss = _empty(stream, n, dtype=torch.float32, device=z.device)
    if dz is None:
        dz = _empty_like(stream, z)
    check(load().tfk_sampled_softmax_xent(_ptr(z), _dt(z), n, u, u_pad, m, _ptr(bias_c), _ptr(true_pos),
                                          _ptr(lq_true), _ptr(lq_sampled), float(scale), _ptr(loss), _ptr(dz),
                                          _stream(stream)))
    return loss, dz


def scatter_apply_sgd(var, idx, grad_t, lr, shadow=None, stream=None):
    """var[idx[j]] -= lr * grad_t[:, j] (var rows x d fp32; grad_t d x ld fp32); shadow rewritten."""
    rows, d = var.shape if var.dim() == 2 else (var.shape[0], 1)
    ld = grad_t.shape[-1]
    if var.dtype != torch.float32 or grad_t.dtype != torch.float32 or idx.dtype != torch.int32:
        raise TypeError("var and grad_t are float32, idx int32")
    check(load().tfk_scatter_apply_sgd(_ptr(var), _ptr(shadow), rows, d, _ptr(idx), idx.numel(), _ptr(grad_t), ld,
                                       float(lr), _stream(stream)))
    return var


# ----------------------------------------------------------------------------- streams and programs
def stream_wait(waiter, producer):
    """Work enqueued on ``waiter`` afterwards waits for everything enqueued on ``producer`` so far
    (an event join inside the library; recorded into a program like the ops)."""
    check(load().tfk_stream_wait(ctypes.c_void_p(waiter.cuda_stream), ctypes.c_void_p(producer.cuda_stream)))


class Mark:
    """A point on one stream that other streams can wait for (``record`` then ``wait``): unlike
    ``stream_wait``, work the producer enqueues after ``record`` is not waited for.  Recorded
    into programs like the ops; a mark must outlive every program that uses it."""

    def __init__(self):
        self._lib = load()
        h = ctypes.c_void_p()
        check(self._lib.tfk_mark_create(ctypes.byref(h)))
        self._h = h

    def record(self, stream):
        check(self._lib.tfk_mark_record(self._h, ctypes.c_void_p(stream.cuda_stream)))

    def wait(self, waiter):
        """Work enqueued on ``waiter`` afterwards starts once the latest ``record`` is reached."""
        check(self._lib.tfk_stream_wait_mark(ctypes.c_void_p(waiter.cuda_stream), self._h))

    def close(self):
        if self._h is not None and self._h.value:
            self._lib.tfk_mark_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Program:
    """A recorded sequence of library calls, issued again from C++ by ``run()``.

    ``with prog.recording(): ...`` runs the calls made inside the block as usual and records
    each one that succeeds (same pointers, shapes, scalars and streams); ``run()`` enqueues them
    again in order.  Buffers the calls name must stay allocated while the program is used."""

    def __init__(self):
        self._lib = load()
        h = ctypes.c_void_p()
        check(self._lib.tfk_program_create(ctypes.byref(h)))
        self._h = h

    def recording(self):
        prog = self

        class _Rec:
            def __enter__(self):
                check(prog._lib.tfk_program_begin(prog._h))
                return prog

            def __exit__(self, *exc):
                check(prog._lib.tfk_program_end(prog._h))
                return False

        return _Rec()

    def __len__(self) -> int:
        return int(self._lib.tfk_program_length(self._h))

    def run(self):
        check(self._lib.tfk_program_run(self._h))

    def close(self):
        if self._h is not None and self._h.value:
            self._lib.tfk_program_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
