"""C ABI checks that need no GPU: the library loads, exports what include/tfk.h
declares, and rejects invalid arguments before launching anything.

Every call here fails validation (a GPU-free code path); pointers are fake
addresses that are never dereferenced.
"""
import ctypes
import os
import re
import subprocess
import tempfile

import pytest
import torch

from paper_1605_08695_amd import _lib, ops
from paper_1605_08695_amd._lib import Nhwc, Window

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tfk.h")

F32, BF16 = 0, 1
OK, NULL, SHAPE, DTYPE, ALIGN, OVERFLOW, ALIAS, WORKSPACE, HIP, ARG = range(10)
P = 0x10000000          # fake, 256-byte aligned device addresses (never dereferenced)


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def vp(a):
    return ctypes.c_void_p(a)


def test_header_symbols_exported(lib):
    decl = re.findall(r"TFK_API\s+[^;]*?\b(tfk_\w+)\s*\(", open(HEADER).read())
    assert sorted(set(decl)) == sorted(_lib.EXPORTS)
    out = subprocess.check_output(["nm", "-D", "--defined-only", _lib.LIB_PATH], text=True)
    exported = set(re.findall(r"\bT (tfk_\w+)", out))
    assert set(decl) == exported
    for name in decl:
        assert hasattr(lib, name)


def test_abi_version_and_status_strings(lib):
    assert lib.tfk_abi_version() == 16
    assert lib.tfk_status_string(0) == b"ok"
    assert lib.tfk_status_string(6) == b"illegal aliasing"
    assert lib.tfk_status_string(99) == b"unknown status"


def conv_fwd(lib, x=P, xd=(2, 8, 8, 16, 0), w=P + 0x100000, cout=32, win=(3, 3, 1, 1, 1, 1, 1, 1), dt=F32,
             y=P + 0x200000, yd=(2, 8, 8, 32, 0)):
    return lib.tfk_conv2d_fwd(vp(x), Nhwc(*xd), vp(w), cout, Window(*win), dt, vp(y), Nhwc(*yd), None, 0, None)


def test_conv_fwd_validation(lib):
    assert conv_fwd(lib, x=0) == NULL
    assert conv_fwd(lib, dt=7) == DTYPE
    assert conv_fwd(lib, yd=(2, 7, 8, 32, 0)) == SHAPE                 # wrong output extent
    assert conv_fwd(lib, yd=(2, 8, 8, 16, 0)) == SHAPE                 # wrong cout
    assert conv_fwd(lib, win=(3, 3, 1, 1, 3, 1, 1, 1)) == SHAPE        # pad == kernel extent
    assert conv_fwd(lib, win=(3, 3, 0, 1, 1, 1, 1, 1)) == SHAPE        # zero stride
    assert conv_fwd(lib, xd=(2, 8, 8, 16, 8)) == SHAPE                 # pixel stride < c
    assert conv_fwd(lib, x=P + 2) == ALIGN                             # fp32 needs 4-byte alignment
    assert conv_fwd(lib, y=P + 0x100) == ALIAS                         # y overlaps x
    assert conv_fwd(lib, xd=(2, 1, 1, 16, 0), yd=(2, 1, 1, 32, 0), win=(3, 3, 1, 1, 0, 0, 0, 0)) == SHAPE
    assert b"must be" in lib.tfk_last_error() or len(lib.tfk_last_error()) > 0


def test_conv_fwd_bias_relu_validation(lib):
    def fused(x=P, bias=P + 0x300000, y=P + 0x200000):
        return lib.tfk_conv2d_fwd_bias_relu(vp(x), Nhwc(2, 8, 8, 16, 0), vp(P + 0x100000), 32, vp(bias),
                                            Window(3, 3, 1, 1, 1, 1, 1, 1), F32, vp(y), Nhwc(2, 8, 8, 32, 0),
                                            None, 0, None)
    assert fused(bias=0) == NULL
    assert fused(bias=P + 0x300002) == ALIGN                            # fp32 bias, 4-byte aligned
    assert fused(bias=P + 0x200010) == ALIAS                            # bias inside y
    assert fused(x=0) == NULL                                           # the convolution's own checks
    assert fused(y=P + 0x100) == ALIAS


def test_conv_bwd_validation(lib):
    W = Window(3, 3, 1, 1, 1, 1, 1, 1)
    st = lib.tfk_conv2d_bwd_input(vp(P), Nhwc(2, 8, 8, 32, 0), vp(P + 0x100000), W, F32, vp(P + 0x200000),
                                  Nhwc(2, 8, 8, 16, 0), ctypes.c_float(0.5), None, 0, None)
    assert st == ARG                                                   # beta must be 0 or 1
    st = lib.tfk_conv2d_bwd_input(vp(P), Nhwc(2, 8, 8, 32, 0), vp(P + 0x100000), W, F32, vp(P + 0x100),
                                  Nhwc(2, 8, 8, 16, 0), ctypes.c_float(0.0), None, 0, None)
    assert st == ALIAS                                                 # dx overlaps dy
    # bwd-filter with splits needs a workspace
    xd = Nhwc(64, 56, 56, 64, 0)
    need = lib.tfk_conv2d_workspace_bytes(2, xd, 64, W, BF16)
    assert need > 0
    st = lib.tfk_conv2d_bwd_filter(vp(P), xd, vp(P + 0x40000000), Nhwc(64, 56, 56, 64, 0), W, BF16,
                                   vp(P + 0x80000000), vp(P + 0xC0000000), need - 1, None)
    assert st == WORKSPACE
    st = lib.tfk_conv2d_bwd_filter(vp(P), xd, vp(P + 0x40000000), Nhwc(64, 56, 56, 64, 0), W, BF16,
                                   vp(0), vp(P + 0xC0000000), need, None)
    assert st == NULL


def test_conv_bias_relu_maxpool_validation(lib):
    """The convolution fused with the max-pool of its output: bias is required, the pool must fit
    y, py and taps must overlap nothing, before any launch."""
    W = Window(3, 3, 1, 1, 1, 1, 1, 1)
    PW = Window(3, 3, 2, 2, 0, 0, 0, 0)

    def call(bias=P + 0x300000, py=P + 0x400000, taps=P + 0x500000, pyd=(2, 6, 6, 64, 0), pw=PW):
        return lib.tfk_conv2d_fwd_bias_relu_maxpool(vp(P), Nhwc(2, 13, 13, 32, 0), vp(P + 0x100000), 64, vp(bias), W,
                                                    BF16, vp(P + 0x200000), Nhwc(2, 13, 13, 64, 0), pw, vp(py),
                                                    Nhwc(*pyd), vp(taps), None, 0, None)
    assert call(bias=0) == NULL
    assert call(pyd=(2, 7, 6, 64, 0)) == SHAPE                          # not the pool's output shape
    assert call(py=P + 0x200100) == ALIAS                               # py inside y
    assert call(taps=P + 0x400010) == ALIAS                             # taps inside py
    assert call(pw=Window(17, 17, 1, 1, 0, 0, 0, 0), pyd=(2, 1, 1, 64, 0)) == SHAPE   # window past y


def test_conv_bwd_filter_noalloc_validation(lib):
    """The filter gradient without a workspace: bad shapes, and a shape that needs more than the
    library's 128 MiB of device scratch, are refused before any HIP call."""
    W = Window(3, 3, 1, 1, 1, 1, 1, 1)
    st = lib.tfk_conv2d_bwd_filter_noalloc(vp(P), Nhwc(2, 8, 8, 16, 0), vp(P + 0x100000), Nhwc(2, 7, 8, 32, 0), W,
                                           BF16, vp(P + 0x200000), None)
    assert st == SHAPE                                                 # dy is not the output shape
    xd, dyd = Nhwc(512, 224, 224, 3, 0), Nhwc(512, 55, 55, 64, 0)
    W1 = Window(11, 11, 4, 4, 2, 2, 2, 2)
    need = lib.tfk_conv2d_workspace_bytes(2, xd, 64, W1, BF16)
    assert need > 128 << 20
    st = lib.tfk_conv2d_bwd_filter_noalloc(vp(P), xd, vp(P + 0x40000000), dyd, W1, BF16, vp(P + 0x80000000), None)
    assert st == WORKSPACE
    assert b"128" in lib.tfk_last_error() or b"134217728" in lib.tfk_last_error()


def test_conv_bwd_input_relu_bwd_validation(lib):
    """The input gradient fused with the producer's ReLU backward: workspace query (op 3),
    NULL, aliasing and workspace checks, before any launch."""
    W = Window(3, 3, 1, 1, 1, 1, 1, 1)
    xd, dyd = Nhwc(128, 13, 13, 384, 0), Nhwc(128, 13, 13, 256, 0)
    need = lib.tfk_conv2d_workspace_bytes(3, xd, 256, W, BF16)
    # at least one fp32 partial per channel and per 128-pixel tile of the output grid
    assert need >= 384 * 4 * ((128 * 13 * 13 + 127) // 128)
    assert lib.tfk_conv2d_workspace_bytes(1, xd, 256, W, BF16) == 0
    def fused(dy=P, w=P + 0x10000000, y=P + 0x20000000, dpre=P + 0x30000000, db=P + 0x40000000,
              ws=P + 0x50000000, ws_bytes=need, beta=0.0):
        return lib.tfk_conv2d_bwd_input_relu_bwd(vp(dy), dyd, vp(w), W, BF16, vp(y), vp(dpre), xd,
                                                 ctypes.c_float(beta), vp(db), vp(ws), ws_bytes, None)
    assert fused(dy=0) == NULL
    assert fused(y=0) == NULL
    assert fused(beta=0.5) == ARG
    assert fused(db=0, ws_bytes=need - 1) == WORKSPACE                  # deferred: the same checks
    assert fused(dpre=P + 0x20000010) == ALIAS                         # dpre overlaps y
    assert fused(db=P + 0x30000000) == ALIAS                           # dbias inside dpre
    assert fused(ws_bytes=need - 1) == WORKSPACE
    assert fused(ws=P + 0x20000000) == ALIAS                           # workspace over y


def test_pool_validation(lib):
    W = Window(3, 3, 2, 2, 0, 0, 0, 0)
    st = lib.tfk_maxpool_fwd(vp(P), Nhwc(2, 7, 7, 8, 0), W, BF16, vp(P + 0x100000), Nhwc(2, 4, 4, 8, 0),
                             vp(P + 0x200000), None)
    assert st == SHAPE                                                 # 7 -> 3, not 4
    big = Nhwc(1 << 12, 1 << 10, 1 << 8, 4, 0)                         # 2^32 elements: argmax overflows
    st = lib.tfk_maxpool_fwd(vp(P), big, Window(2, 2, 2, 2, 0, 0, 0, 0), BF16, vp(P), Nhwc(1 << 12, 512, 128, 4, 0),
                             vp(P), None)
    assert st == OVERFLOW
    st = lib.tfk_maxpool_bwd(vp(P), vp(P + 0x100000), Nhwc(2, 3, 3, 8, 0), W, BF16, vp(P + 0x200000),
                             Nhwc(2, 7, 7, 8, 0), ctypes.c_float(2.0), None)
    assert st == ARG


def test_bias_relu_validation(lib):
    yd = Nhwc(4, 8, 8, 64, 0)
    need = lib.tfk_bias_relu_bwd_workspace_bytes(yd, BF16)
    assert need >= 64 * 4
    st = lib.tfk_bias_relu_bwd(vp(P), vp(P + 0x100000), yd, vp(P + 0x100010), vp(P + 0x300000), BF16,
                               vp(P + 0x400000), need, None)
    assert st == ALIAS                                                 # dpre partially overlaps dy
    st = lib.tfk_bias_relu_bwd(vp(P), vp(P + 0x100000), yd, vp(P + 0x100000), vp(P + 0x300000), BF16,
                               vp(P + 0x400000), need - 4, None)
    assert st == WORKSPACE
    st = lib.tfk_bias_relu_fwd(vp(P), yd, vp(0), BF16, None)
    assert st == NULL


def test_maxpool_relu_bwd_validation(lib):
    W = Window(3, 3, 2, 2, 0, 0, 0, 0)
    yd, xd = Nhwc(2, 3, 3, 8, 0), Nhwc(2, 7, 7, 8, 0)
    def fused(dy=P, am=P + 0x100000, y=P + 0x200000, dpre=P + 0x300000, beta=0.0, db=P + 0x400000, ws=P + 0x500000,
              ws_bytes=1 << 20, x=xd, py=0, pys=0):
        return lib.tfk_maxpool_bwd_relu_bwd(vp(dy), vp(am), yd, W, BF16, vp(y), vp(py), pys, vp(dpre), x,
                                            ctypes.c_float(beta), vp(db), vp(ws), ws_bytes, None)
    assert fused(dy=0) == NULL
    assert fused(db=0, dpre=P + 0x200010) == ALIAS                     # deferred: the same checks
    assert fused(beta=0.5) == ARG
    assert fused(dpre=P + 0x200010) == ALIAS                           # dpre overlaps y
    assert fused(x=Nhwc(2, 9, 9, 8, 0)) == SHAPE                        # 9 -> 4 with a 3x3/2 window, not 3
    assert fused(ws_bytes=0) == WORKSPACE
    assert fused(ws=P + 0x300000) == ALIAS                              # workspace inside dpre
    # the pool's output as the mask: y may then be NULL (beta = 0), not when beta = 1 (py ignored)
    assert fused(y=0) == NULL
    assert fused(y=0, py=P + 0x600000, pys=8, beta=1.0) == NULL
    assert fused(y=0, py=P + 0x600000, pys=4) == SHAPE                 # pixel stride below the channels
    assert fused(y=0, py=P + 0x300010, pys=8) == ALIAS                 # py inside dpre
    assert fused(y=0, py=P + 0x600001, pys=8) == ALIGN
    assert fused(y=0, py=P + 0x600000, pys=8, ws=P + 0x600000) == ALIAS  # workspace over py


def test_maxpool_taps_validation(lib):
    """The uint8 tap form of the pool's selection: NULL, window size and aliasing checks."""
    W = Window(3, 3, 2, 2, 0, 0, 0, 0)
    yd, xd = Nhwc(2, 3, 3, 8, 0), Nhwc(2, 7, 7, 8, 0)
    fwd = lambda taps, win=W, x=xd, y=yd: lib.tfk_maxpool_fwd_taps(vp(P), x, win, BF16, vp(P + 0x100000), y,
                                                                   vp(taps), None)
    assert fwd(0) == NULL
    assert fwd(P + 0x100010) == ALIAS                                   # taps inside y
    big = Window(17, 16, 1, 1, 0, 0, 0, 0)                              # 272 taps do not fit a byte
    assert fwd(P + 0x200000, big, Nhwc(1, 17, 16, 8, 0), Nhwc(1, 1, 1, 8, 0)) == SHAPE
    assert lib.tfk_maxpool_bwd_taps(vp(P), vp(0), yd, W, BF16, vp(P + 0x200000), xd, ctypes.c_float(0.0),
                                    None) == NULL
    assert lib.tfk_maxpool_bwd_taps(vp(P), vp(P + 0x100000), yd, big, BF16, vp(P + 0x200000), xd,
                                    ctypes.c_float(0.0), None) == SHAPE
    assert lib.tfk_maxpool_bwd_relu_bwd_taps(vp(P), vp(P + 0x100000), yd, W, BF16, vp(P + 0x200000), vp(0), 0,
                                             vp(P + 0x200010), xd, ctypes.c_float(0.0), vp(P + 0x400000),
                                             vp(P + 0x500000), 1 << 20, None) == ALIAS   # dpre overlaps y


def test_sgd_validation(lib):
    assert lib.tfk_apply_sgd(vp(P), vp(P + 0x10), 100, ctypes.c_float(0.01), None, None) == ALIAS
    assert lib.tfk_apply_sgd(vp(P), vp(P + 0x1000), -1, ctypes.c_float(0.01), None, None) == SHAPE
    assert lib.tfk_apply_sgd(vp(P), vp(P + 0x1000), 10, ctypes.c_float(float("nan")), None, None) == ARG
    assert lib.tfk_apply_sgd(vp(P + 1), vp(P + 0x1000), 10, ctypes.c_float(0.01), None, None) == ALIGN
    assert lib.tfk_apply_sgd(vp(0), vp(P), 10, ctypes.c_float(0.01), None, None) == NULL
    # empty update is a no-op that needs no pointers
    assert lib.tfk_apply_sgd(vp(0), vp(0), 0, ctypes.c_float(0.01), None, None) == OK
    VP = ctypes.c_void_p * 2
    NS = ctypes.c_int64 * 2
    st = lib.tfk_apply_sgd_multi(2, VP(P, P + 0x1000), VP(P + 0x2000, P + 0x1000), NS(16, 16),
                                 ctypes.c_float(0.01), None, None)
    assert st == ALIAS                                                 # second var == its grad
    assert b"tensor 1" in lib.tfk_last_error()


def test_momentum_adam_validation(lib):
    f = ctypes.c_float
    mom = lambda var, acc, grad, n, lr=0.01, m=0.9, nest=0, sh=None: lib.tfk_apply_momentum(
        vp(var), vp(acc), vp(grad), n, f(lr), f(m), nest, vp(sh) if sh else None, None)
    assert mom(P, P + 0x1000, P + 0x2000, -1) == SHAPE
    assert mom(P, P + 0x10, P + 0x2000, 100) == ALIAS                 # var overlaps accum
    assert mom(P, P + 0x1000, P + 0x2000, 100, sh=P + 0x2010) == ALIAS  # shadow overlaps grad
    assert mom(P, P + 0x1000, P + 0x2000, 10, lr=float("inf")) == ARG
    assert mom(P, P + 0x1000, P + 0x2000, 10, m=float("nan")) == ARG
    assert mom(P, P + 0x1000, P + 0x2000, 10, nest=2) == ARG
    assert mom(P, 0, P + 0x2000, 10) == NULL
    assert mom(P, P + 0x1002, P + 0x2000, 10) == ALIGN
    assert mom(0, 0, 0, 0) == OK                                       # empty: no pointers needed
    adam = lambda var, m, v, grad, n, lr=0.01, b1=0.9, b2=0.999, eps=1e-8, t=1: lib.tfk_apply_adam(
        vp(var), vp(m), vp(v), vp(grad), n, f(lr), f(b1), f(b2), f(eps), t, None, None)
    args = (P, P + 0x1000, P + 0x2000, P + 0x3000)
    assert adam(*args, -1) == SHAPE
    assert adam(P, P + 0x1000, P + 0x1000, P + 0x3000, 16) == ALIAS    # m is v
    assert adam(*args, 16, b1=1.0) == ARG
    assert adam(*args, 16, b1=-0.1) == ARG
    assert adam(*args, 16, b2=float("nan")) == ARG
    assert adam(*args, 16, eps=-1.0) == ARG
    assert adam(*args, 16, t=0) == ARG
    assert adam(*args, 16, lr=float("nan")) == ARG
    assert adam(P, P + 0x1000, 0, P + 0x3000, 16) == NULL
    assert adam(P, P + 0x1000, P + 0x2001, P + 0x3000, 16) == ALIGN
    assert adam(0, 0, 0, 0, 0) == OK
    assert b"" != lib.tfk_status_string(ARG)


def test_softmax_xent_validation(lib):
    f = ctypes.c_float
    sm = lambda z, n, c, bias=None, lab=P + 0x10000, loss=P + 0x20000, dz=P + 0x30000, scale=1.0, dt=0: \
        lib.tfk_softmax_xent(vp(z), dt, n, c, vp(bias) if bias else None, vp(lab), f(scale), vp(loss), vp(dz), None)
    assert sm(P, -1, 10) == SHAPE
    assert sm(P, 4, 0) == SHAPE
    assert sm(P, 4, 10, dt=7) == DTYPE
    assert sm(P, 4, 10, scale=float("nan")) == ARG
    assert sm(P, 4, 10, dz=P + 8) == ALIAS                     # partial overlap with the logits
    assert sm(P, 4, 10, loss=P + 0x10004) == ALIAS             # loss overlaps the labels
    assert sm(P, 4, 10, bias=P + 0x20000) == ALIAS             # bias overlaps the loss
    assert sm(P, 4, 10, lab=0) == NULL
    assert sm(P + 2, 4, 10) == ALIGN
    assert sm(P, 1 << 30, 1 << 20) == OVERFLOW
    assert sm(0, 0, 10, lab=0, loss=0, dz=0) == OK             # no rows: nothing to touch


def test_sampled_softmax_validation(lib):
    f = ctypes.c_float
    g = lambda table, rows, d, idx, u, u_pad, out, dt=0: lib.tfk_gather_rows_t(vp(table), dt, rows, d, vp(idx), u,
                                                                              u_pad, vp(out), None)
    assert g(P, 100, 8, P + 0x10000, 10, 5, P + 0x20000) == SHAPE            # u_pad < u
    assert g(P, 100, 0, P + 0x10000, 10, 16, P + 0x20000) == SHAPE
    assert g(P, 100, 8, P + 0x10000, 10, 16, P + 0x100) == ALIAS             # out inside the table
    assert g(P, 100, 8, 0, 10, 16, P + 0x20000) == NULL
    assert g(P, 100, 8, P + 0x10000, 10, 16, P + 0x20000, dt=9) == DTYPE
    sx = lambda n, u, u_pad, m, dz=P + 0x40000, loss=P + 0x50000, tp=P + 0x60000, scale=1.0: \
        lib.tfk_sampled_softmax_xent(vp(P), 0, n, u, u_pad, m, None, vp(tp), vp(P + 0x70000), vp(P + 0x80000),
                                     f(scale), vp(loss), vp(dz), None)
    assert sx(4, 10, 16, 11) == SHAPE                                      # m > u
    assert sx(4, 10, 8, 5) == SHAPE                                        # u_pad < u
    assert sx(4, 10, 16, 5, scale=float("inf")) == ARG
    assert sx(4, 10, 16, 5, dz=P + 0x10) == ALIAS                          # dz overlaps z
    assert sx(4, 10, 16, 5, loss=P + 0x60000) == ALIAS                     # loss overlaps true_pos
    assert sx(4, 10, 16, 5, tp=0) == NULL
    assert sx(0, 10, 16, 5) == OK
    sc = lambda rows, d, u, ld, var=P, grad=P + 0x100000, lr=0.1: lib.tfk_scatter_apply_sgd(
        vp(var), None, rows, d, vp(P + 0x200000), u, vp(grad), ld, f(lr), None)
    assert sc(100, 8, 10, 5) == SHAPE                                      # ld < u
    assert sc(100, 8, 10, 16, lr=float("nan")) == ARG
    assert sc(100, 8, 10, 16, grad=P + 0x40) == ALIAS
    assert sc(100, 8, 10, 16, var=P + 2) == ALIGN
    assert sc(100, 8, 0, 16, var=0, grad=0) == OK


def test_empty_batch_conv_fwd_is_noop(lib):
    # n == 0: nothing to read or write, so no launch and no pointers needed
    assert conv_fwd(lib, x=0, w=0, y=0, xd=(0, 8, 8, 16, 0), yd=(0, 8, 8, 32, 0)) == OK


def test_nhwc_view_of_channel_slice():
    buf = torch.zeros(2, 5, 6, 48)
    d = ops.nhwc(buf[..., 16:40])
    assert (d.n, d.h, d.w, d.c, d.pixel_stride) == (2, 5, 6, 24, 48)
    d = ops.nhwc(buf)
    assert (d.c, d.pixel_stride) == (48, 48)
    with pytest.raises(ValueError):
        ops.nhwc(buf.permute(0, 3, 1, 2))


FASTDIV_TEST = r"""
#include <stdio.h>
#include <stdint.h>
#include "fastdiv.h"
int main() {
    const uint32_t ds[] = {1, 2, 3, 5, 6, 7, 11, 13, 27, 55, 169, 729, 3025, 50176, 65535, 65536, 65537,
                           1000003, 46340u * 46340u, 0x7fffffffu};
    uint64_t bad = 0;
    for (uint32_t d : ds) {
        FastDiv f(d);
        for (uint64_t n = 0; n < (1ull << 31); n += (n < 1000000 ? 1 : 7919 + (n >> 20))) {
            uint32_t q, r;
            f.divmod((uint32_t)n, q, r);
            if (q != n / d || r != n % d) ++bad;
        }
        const uint32_t edge[] = {0x7fffffffu, 0x7ffffffeu, d - 1, d, d + 1, 2 * d - 1};
        for (uint32_t n : edge) {
            if (n >= 0x80000000u) continue;
            uint32_t q, r;
            f.divmod(n, q, r);
            if (q != n / d || r != n % d) ++bad;
        }
    }
    printf("%llu\n", (unsigned long long)bad);
    return bad != 0;
}
"""


def test_fastdiv_host_exhaustive_sample():
    with tempfile.TemporaryDirectory() as td:
        src = os.path.join(td, "t.cpp")
        open(src, "w").write(FASTDIV_TEST)
        exe = os.path.join(td, "t")
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-I",
                               os.path.join(ROOT, "paper_1605_08695_amd", "csrc"), src, "-o", exe])
        assert subprocess.run([exe], capture_output=True, text=True).stdout.strip() == "0"


def test_fully_connected_workspace_queries(lib):
    """A whole-window convolution at small batch is flattened and split across blocks: the forward
    and input-gradient queries ask for the split partials (splits x rows x outputs fp32); a large
    batch asks for none, and a strided input gradient (several phases) is never split."""
    lib.tfk_conv2d_workspace_bytes.restype = ctypes.c_size_t
    fc6 = Window(6, 6, 1, 1, 0, 0, 0, 0)
    q = lambda op, n, win=fc6, h=6, c=256, cout=4096, dt=BF16: lib.tfk_conv2d_workspace_bytes(
        op, Nhwc(n, h, h, c, 0), cout, win, dt)
    fwd, bwi = q(0, 4), q(1, 4)
    assert fwd > 0 and fwd % (4 * 4 * 4096) == 0                  # splits x 4 rows x 4096 outputs x 4 B
    assert bwi > 0 and bwi % (4 * 4 * 9216) == 0                  # splits x 4 rows x 9216 inputs x 4 B
    assert q(0, 4, dt=F32) == 0 and q(1, 4, dt=F32) == 0          # the split path is the bf16 kernel's
    assert q(0, 4096) == 0 and q(1, 4096) == 0                    # 32 x 32 tiles: no split
    s3 = q(1, 4, win=Window(3, 3, 1, 1, 1, 1, 1, 1), h=6)          # 3x3, stride 1: split over 36 K tiles
    assert s3 > 0 and s3 % (4 * 36 * 256) == 0                    # splits x 144 pixels x 256 x 4 B
    assert q(1, 4, win=Window(3, 3, 2, 2, 1, 1, 1, 1), h=6) == 0  # stride 2: several phases, no split
    assert q(2, 4) == 0                                           # 4-pixel reduction: no split partials


def test_program_records_successful_calls_only(lib):
    # Recording on the calling thread: calls that pass validation are appended (here no-ops with an
    # empty batch, which enqueue nothing), failing calls are not; a run re-issues the recorded ones.
    prog = ops.Program()
    with prog.recording():
        assert conv_fwd(lib, x=0, w=0, y=0, xd=(0, 8, 8, 16, 0), yd=(0, 8, 8, 32, 0)) == OK
        assert conv_fwd(lib, x=0) == NULL                         # rejected: not recorded
        assert lib.tfk_apply_sgd(None, None, 0, ctypes.c_float(0.1), None, None) == OK
    assert len(prog) == 2
    prog.run()
    assert len(prog) == 2
    with prog.recording():                                       # recording again starts empty
        pass
    assert len(prog) == 0
    prog.close()


def test_program_state_errors(lib):
    a, b = ops.Program(), ops.Program()
    assert lib.tfk_program_begin(a._h) == OK
    assert lib.tfk_program_begin(b._h) == ARG                    # one recording per thread
    assert lib.tfk_program_run(b._h) == ARG                      # no runs while recording
    assert lib.tfk_program_end(b._h) == ARG                      # b is not the one recording
    assert lib.tfk_program_end(a._h) == OK
    assert lib.tfk_program_end(a._h) == ARG
    assert lib.tfk_program_begin(None) == NULL
    assert lib.tfk_program_length(None) == 0
    assert lib.tfk_program_begin(a._h) == OK
    a.close()                                                    # destroying stops its recording
    assert lib.tfk_program_begin(b._h) == OK
    assert lib.tfk_program_end(b._h) == OK
    assert lib.tfk_stream_wait(None, None) == OK                 # same stream: no-op
    b.close()
    # marks: NULL checks only (creating one needs a HIP event)
    assert lib.tfk_mark_create(None) == NULL
    assert lib.tfk_mark_record(None, None) == NULL
    assert lib.tfk_stream_wait_mark(None, None) == NULL
    lib.tfk_mark_destroy(None)


def test_deferred_bias_validation(lib):
    """Deferred bias gradients: where a call given dbias = NULL left its partials (thread-local),
    and the argument checks of the batched finish (nothing is launched in this test)."""
    import threading
    part, rows = ctypes.c_void_p(), ctypes.c_int32()
    assert lib.tfk_last_bias_partials(None, ctypes.byref(rows)) == NULL
    got = []
    t = threading.Thread(target=lambda: got.append(lib.tfk_last_bias_partials(ctypes.byref(part),
                                                                              ctypes.byref(rows))))
    t.start()
    t.join()
    assert got == [ARG]                                 # no deferred call on that thread yet
    # an empty tensor: deferred without a launch, 0 partial rows left at the workspace
    yd = Nhwc(0, 4, 4, 8, 0)
    assert lib.tfk_bias_relu_bwd(vp(P), vp(P + 0x1000), yd, vp(P + 0x1000), vp(0), BF16, vp(P + 0x2000), 0,
                                 None) == OK
    assert lib.tfk_last_bias_partials(ctypes.byref(part), ctypes.byref(rows)) == OK
    assert rows.value == 0 and part.value == P + 0x2000
    Arr = lambda T, *v: (T * len(v))(*v)
    def finish(n=1, parts=(P,), rws=(4,), chans=(8,), dbs=(P + 0x10000,)):
        return lib.tfk_bias_grad_finish(n, Arr(ctypes.c_void_p, *parts) if parts is not None else None,
                                        Arr(ctypes.c_int32, *rws), Arr(ctypes.c_int32, *chans),
                                        Arr(ctypes.c_void_p, *dbs), None)
    assert finish(n=-1) == ARG
    assert lib.tfk_bias_grad_finish(0, None, None, None, None, None) == OK
    assert finish(parts=None) == NULL
    assert finish(parts=(0,)) == NULL                   # rows > 0 need partials
    assert finish(rws=(-1,)) == SHAPE
    assert finish(chans=(0,)) == SHAPE
    assert finish(chans=(16385,)) == SHAPE
    assert finish(dbs=(0,)) == NULL
    assert finish(dbs=(P + 0x10002,)) == ALIGN
    assert finish(dbs=(P + 16,)) == ALIAS               # dbias inside the partials (4 x 8 floats)
    assert finish(n=2, parts=(P, P + 0x1000), rws=(4, 4), chans=(8, 8), dbs=(P + 0x10000, P + 0x10010)) == ALIAS


def test_channel_slices_alias(lib):
    """Two channel slices of one pixel-strided buffer overlap only where their channels do: the
    check rejects sharing channels (nothing launched here)."""
    W = Window(3, 3, 1, 1, 1, 1, 1, 1)
    # x = channels 8..23 and y = channels 0..15 of one 4 x 4 image of 64-channel pixels
    xd, yd = Nhwc(1, 4, 4, 16, 64), Nhwc(1, 4, 4, 16, 64)
    st = lib.tfk_conv2d_fwd(vp(P + 16), xd, vp(P + 0x100000), 16, W, BF16, vp(P), yd, None, 0, None)
    assert st == ALIAS
    # dpre = channels 0..15 and dy = channels 12..27: the fused input gradient rejects them too
    st = lib.tfk_conv2d_bwd_input(vp(P + 24), yd, vp(P + 0x100000), W, BF16, vp(P), xd, ctypes.c_float(0.0),
                                  None, 0, None)
    assert st == ALIAS
