"""Per-op parity of the HIP kernels against the CPU oracle on seeded inputs (GPU).

Shapes span several tiles with ragged tails, odd channel counts (scalar
gather paths), strided and asymmetric windows, channel-slice views (concat
buffers), the stride-phase cases of bwd-input (including a phase with no
taps), empty batches, ties in max-pool and both element types.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_1605_08695_amd import ops
from tests.gpu_parity import BAR, assert_close, err, f64, say, ulp_diff_f32

pytestmark = pytest.mark.gpu

DEV = "cuda"
DTYPES = [torch.float32, torch.bfloat16]

# N, H, W, Cin, Cout, KH, KW, sh, sw, pads
CONV_CASES = [
    ("single_layer", 8, 32, 32, 16, 32, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("ragged_tiles", 3, 13, 11, 24, 136, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("cin3_11x11s4", 2, 35, 35, 3, 64, 11, 11, 4, 4, (2, 2, 2, 2)),
    ("cin3_11x11s4_pairfold", 2, 36, 40, 3, 64, 11, 11, 4, 4, (2, 2, 2, 2)),
    ("cin3_3x3s2_valid_oddw", 2, 15, 17, 3, 32, 3, 3, 2, 2, (0, 0, 0, 0)),
    ("3x3s2_valid", 2, 17, 17, 32, 48, 3, 3, 2, 2, (0, 0, 0, 0)),
    ("1x7_asym", 2, 9, 9, 16, 24, 1, 7, 1, 1, (0, 0, 3, 3)),
    ("7x1_asym", 2, 9, 9, 16, 24, 7, 1, 1, 1, (3, 3, 0, 0)),
    ("1x1s2_empty_phase", 2, 8, 8, 16, 32, 1, 1, 2, 2, (0, 0, 0, 0)),
    ("odd_channels", 2, 7, 7, 5, 7, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("5x5_cout192", 2, 14, 14, 64, 192, 5, 5, 1, 1, (2, 2, 2, 2)),
    ("long_reduction", 16, 28, 28, 64, 64, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("3x3s2_pad_odd", 3, 10, 9, 8, 16, 3, 3, 2, 2, (1, 0, 1, 0)),
    # 64 | Cin: whole 64-channel K tiles, visited channel-chunk outer
    ("tiny_images_c64", 9, 3, 3, 64, 72, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("stride2_c64", 2, 17, 15, 64, 64, 3, 3, 2, 2, (1, 1, 1, 1)),
    ("1x7_c128", 2, 17, 17, 128, 64, 1, 7, 1, 1, (0, 0, 3, 3)),
    ("5x5_valid_c128", 3, 12, 11, 128, 96, 5, 5, 1, 1, (0, 0, 0, 0)),
    ("alexnet_conv3_shape", 4, 13, 13, 192, 384, 3, 3, 1, 1, (1, 1, 1, 1)),
    # widest filter row the pipelined kernel's tap masks hold (31 columns), and one past it
    # (33 columns: the non-pipelined kernel)
    ("1x31_c16", 2, 5, 40, 16, 16, 1, 31, 1, 1, (0, 0, 15, 15)),
    ("1x33_c16", 2, 5, 40, 16, 16, 1, 33, 1, 1, (0, 0, 16, 16)),
    # one output pixel per image: a 64-pixel reduction tile spans 64 images
    ("one_pixel_out_c64", 70, 3, 3, 64, 64, 3, 3, 1, 1, (0, 0, 0, 0)),
    # several 64-channel reduction chunks with tiles spanning image boundaries and uneven
    # padding; a 5x5 filter over 128 channels
    ("chunks_c192_uneven_pad", 3, 11, 9, 192, 128, 3, 3, 1, 1, (1, 1, 0, 2)),
    ("5x5_c128_k192", 2, 14, 14, 128, 192, 5, 5, 1, 1, (2, 2, 2, 2)),
    # enough output pixels (256 tiles of 128) for the 192-channel tiles of the forward pass
    # (192 x 96: 342 blocks fill the last round better than 256 of 128 rows) and the filter
    # gradient
    ("k192_tiles", 32, 32, 32, 64, 192, 3, 3, 1, 1, (1, 1, 1, 1)),
    # ... and of the input gradient (192 input channels)
    ("c192_bwd_tiles", 32, 32, 32, 192, 64, 3, 3, 1, 1, (1, 1, 1, 1)),
    # 192 x 128 tiles: three 192-channel tiles x 170 of 128 pixels fill two rounds of blocks
    ("k576_tiles_192x128", 85, 16, 16, 16, 576, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("c576_bwd_tiles_192x128", 85, 16, 16, 576, 16, 3, 3, 1, 1, (1, 1, 1, 1)),
    # 288 tiles of 128 x 128 (most CUs with one block): 128 x 96 tiles, forward and input gradient
    ("bj96_tiles_fwd", 36, 32, 32, 64, 128, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("bj96_tiles_bwd", 36, 32, 32, 128, 64, 3, 3, 1, 1, (1, 1, 1, 1)),
    # 64 input channels over 75264 pixels (input gradients over many blocks of 64-channel tiles)
    ("c64_bwd_tiles_64x192", 96, 28, 28, 64, 32, 3, 3, 1, 1, (1, 1, 1, 1)),
    # fully connected layers as whole-window convolutions: AlexNet's fc6 (6x6x256 -> 4096) and
    # fc8 (4096 -> 1000 logits), at batch 4
    ("fc6_6x6_window", 4, 6, 6, 256, 4096, 6, 6, 1, 1, (0, 0, 0, 0)),
    ("fc8_1x1_c4096_k1000", 4, 1, 1, 4096, 1000, 1, 1, 1, 1, (0, 0, 0, 0)),
    # at most 32 input channels: 32-channel input-gradient tiles (a GoogLeNet 5x5 branch; a
    # split reduction over few pixels)
    ("5x5_c32_k96", 4, 14, 14, 32, 96, 5, 5, 1, 1, (2, 2, 2, 2)),
    ("narrow_split_c24_k1024", 2, 4, 4, 24, 1024, 1, 1, 1, 1, (0, 0, 0, 0)),
]


def _mk(shape, dtype, rng, scale=1.0):
    a = rng.standard_normal(shape) * scale
    return torch.from_numpy(a).to(dtype).to(DEV)


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("case", CONV_CASES, ids=[c[0] for c in CONV_CASES])
def test_conv_three_directions(case, dtype):
    name, N, H, W, C, K, KH, KW, sh, sw, pads = case
    say("conv case", name, dtype)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    x = _mk((N, H, W, C), dtype, rng)
    w = _mk((KH, KW, C, K), dtype, rng, np.sqrt(2.0 / (KH * KW * C)))
    y = ops.conv2d_fwd(x, w, (sh, sw), pads)
    torch.cuda.synchronize()
    ref = oracle.conv2d_fwd(f64(x), f64(w), (sh, sw), pads)
    assert y.shape == ref.shape
    assert_close(f64(y), ref, dtype, label="fwd")

    # the same convolution with bias + ReLU fused into its epilogue
    bias = torch.from_numpy(rng.standard_normal(K) * 0.5).to(torch.float32).to(DEV)
    yf = ops.conv2d_fwd_bias_relu(x, w, bias, (sh, sw), pads)
    torch.cuda.synchronize()
    ref_f = oracle.bias_relu_fwd(ref, f64(bias))
    assert_close(f64(yf), ref_f, dtype, label="fwd+bias+relu")
    assert not bool(torch.any(torch.signbit(yf))), "fused ReLU must store +0, never -0 or negatives"

    dy = _mk(y.shape, dtype, rng)
    for beta in (0.0, 1.0):
        dx = _mk(x.shape, dtype, rng)
        dx_old = f64(dx)
        ops.conv2d_bwd_input(dy, w, dx, (sh, sw), pads, beta=beta)
        torch.cuda.synchronize()
        ref = oracle.conv2d_bwd_input(f64(dy), f64(w), x.shape, (sh, sw), pads, dx=dx_old, beta=beta)
        assert_close(f64(dx), ref, dtype, label="bwd_input beta=%g" % beta)

    dw = ops.conv2d_bwd_filter(x, dy, (KH, KW), (sh, sw), pads)
    torch.cuda.synchronize()
    ref = oracle.conv2d_bwd_filter(f64(x), f64(dy), (KH, KW), (sh, sw), pads)
    assert_close(f64(dw), ref, torch.float32, dtype, label="bwd_filter")


RELU_BWI_CASES = ["ragged_tiles", "3x3s2_valid", "3x3s2_pad_odd", "1x1s2_empty_phase", "5x5_cout192",
                  "alexnet_conv3_shape", "chunks_c192_uneven_pad", "c192_bwd_tiles", "bj96_tiles_bwd",
                  "c64_bwd_tiles_64x192",
                  "one_pixel_out_c64", "odd_channels", "5x5_c32_k96", "narrow_split_c24_k1024",
                  # a fully connected layer at small batch: split-K partials, then the ReLU
                  # backward and the bias-gradient rows in the epilogue pass
                  "fc8_1x1_c4096_k1000"]


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("name", RELU_BWI_CASES)
def test_conv_bwd_input_relu_bwd_fused(name, dtype):
    """Input gradient fused with the producer's ReLU backward + bias gradient against the
    oracle's two ops (stride phases with empty phases, ragged tiles, 64/128/192-wide tiles)."""
    case = next(c for c in CONV_CASES if c[0] == name)
    _, N, H, W, C, K, KH, KW, sh, sw, pads = case
    say("fused bwd-input + relu case", name, dtype)
    rng = np.random.default_rng(zlib.crc32(("relu" + name).encode()))
    # x is a ReLU output: exact zeros mask the gradient
    y = torch.from_numpy(np.maximum(rng.standard_normal((N, H, W, C)), 0.0)).to(dtype).to(DEV)
    w = _mk((KH, KW, C, K), dtype, rng, np.sqrt(2.0 / (KH * KW * C)))
    out = ops.conv2d_fwd(y, w, (sh, sw), pads)
    dy = _mk(out.shape, dtype, rng)
    dpre = _mk(y.shape, dtype, rng)                            # overwritten
    _, db = ops.conv2d_bwd_input_relu_bwd(dy, w, y, dpre, (sh, sw), pads)
    torch.cuda.synchronize()
    g = oracle.conv2d_bwd_input(f64(dy), f64(w), y.shape, (sh, sw), pads)
    ref_dpre, ref_db = oracle.bias_relu_bwd(f64(y), g)
    assert_close(f64(dpre), ref_dpre, dtype, label="fused dpre")
    assert np.all(f64(dpre)[f64(y) <= 0] == 0) and not bool(torch.any(torch.signbit(dpre)[y <= 0]))
    assert_close(f64(db), ref_db, torch.float32, dtype, label="fused db")
    # the bias gradient is the column sum of the stored dpre
    assert err(f64(db), f64(dpre).sum(axis=(0, 1, 2))) <= 1e-4
    # and the stored dpre is bit-identical to the unfused pair's
    dx = torch.empty_like(y)
    ops.conv2d_bwd_input(dy, w, dx, (sh, sw), pads)
    dp2, _ = ops.bias_relu_bwd(y, dx)
    torch.cuda.synchronize()
    assert torch.equal(dpre, dp2)
    # beta = 1: added to the gradient the input's other readers stored, then masked
    old = _mk(y.shape, dtype, rng)
    dp3 = old.clone()
    _, db3 = ops.conv2d_bwd_input_relu_bwd(dy, w, y, dp3, (sh, sw), pads, beta=1.0)
    dx4 = old.clone()
    ops.conv2d_bwd_input(dy, w, dx4, (sh, sw), pads, beta=1.0)
    dp4, _ = ops.bias_relu_bwd(y, dx4)
    torch.cuda.synchronize()
    g1 = oracle.conv2d_bwd_input(f64(dy), f64(w), y.shape, (sh, sw), pads, dx=f64(old), beta=1.0)
    ref_dpre1, ref_db1 = oracle.bias_relu_bwd(f64(y), g1)
    assert_close(f64(dp3), ref_dpre1, dtype, label="fused dpre beta=1")
    assert_close(f64(db3), ref_db1, torch.float32, dtype, label="fused db beta=1")
    assert torch.equal(dp3, dp4)


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
def test_conv_channel_slice_views(dtype):
    """Input read from and output written into channel slices of wider buffers."""
    rng = np.random.default_rng(7)
    big_in = _mk((2, 9, 9, 48), dtype, rng)
    x = big_in[..., 8:40]                                    # 32 channels, pixel stride 48
    w = _mk((3, 3, 32, 24), dtype, rng, 0.1)
    out = torch.full((2, 9, 9, 64), 7.0, dtype=dtype, device=DEV)
    y = out[..., 16:40]
    ops.conv2d_fwd(x, w, 1, (1, 1, 1, 1), y=y)
    torch.cuda.synchronize()
    ref = oracle.conv2d_fwd(f64(x), f64(w), 1, (1, 1, 1, 1))
    assert_close(f64(y), ref, dtype, label="fwd slice")
    rest = torch.cat([out[..., :16], out[..., 40:]], dim=-1)
    assert bool(torch.all(rest == 7.0))                      # neighbours untouched
    bias = torch.linspace(-1, 1, 24, device=DEV, dtype=torch.float32)
    ops.conv2d_fwd_bias_relu(x, w, bias, 1, (1, 1, 1, 1), y=y)
    torch.cuda.synchronize()
    assert_close(f64(y), oracle.bias_relu_fwd(ref, f64(bias)), dtype, label="fwd+bias+relu slice")
    rest = torch.cat([out[..., :16], out[..., 40:]], dim=-1)
    assert bool(torch.all(rest == 7.0))
    dyb = _mk((2, 9, 9, 64), dtype, rng)
    dy = dyb[..., 16:40]
    dxb = torch.zeros((2, 9, 9, 48), dtype=dtype, device=DEV)
    dx = dxb[..., 8:40]
    ops.conv2d_bwd_input(dy, w, dx, 1, (1, 1, 1, 1))
    dw = ops.conv2d_bwd_filter(x, dy, (3, 3), 1, (1, 1, 1, 1))
    torch.cuda.synchronize()
    assert_close(f64(dx), oracle.conv2d_bwd_input(f64(dy), f64(w), x.shape, 1, (1, 1, 1, 1)), dtype,
                 label="bwd_input slice")
    assert_close(f64(dw), oracle.conv2d_bwd_filter(f64(x), f64(dy), (3, 3), 1, (1, 1, 1, 1)), torch.float32,
                 dtype, label="bwd_filter slice")
    assert bool(torch.all(dxb[..., :8] == 0)) and bool(torch.all(dxb[..., 40:] == 0))


def test_conv_empty_batch_filter_grad_is_zero():
    x = torch.zeros((0, 8, 8, 16), dtype=torch.bfloat16, device=DEV)
    dy = torch.zeros((0, 8, 8, 32), dtype=torch.bfloat16, device=DEV)
    dw = torch.full((3, 3, 16, 32), 5.0, device=DEV)
    ops.conv2d_bwd_filter(x, dy, (3, 3), 1, (1, 1, 1, 1), dw=dw)
    torch.cuda.synchronize()
    assert bool(torch.all(dw == 0))


@pytest.mark.parametrize("shape", [(2, 36, 40, 64, 11, 4, (2, 2, 2, 2)), (2, 15, 17, 32, 3, 2, (0, 0, 0, 0))],
                         ids=["pairfold_in_place", "oddw_padded"])
def test_conv_rgbx_input_view(shape):
    """An RGB input given as a 3-channel view of an RGBx buffer whose fourth channel holds
    finite garbage: read in place when it folds, padded otherwise; the result is that of
    the 3-channel image either way."""
    N, H, W, K, KS, s, pads = shape
    rng = np.random.default_rng(31)
    buf = _mk((N, H, W, 4), torch.bfloat16, rng)             # channel 3: random, finite
    x = buf[..., :3]
    w = _mk((KS, KS, 3, K), torch.bfloat16, rng, 0.1)
    bias = torch.from_numpy(rng.standard_normal(K) * 0.5).to(torch.float32).to(DEV)
    y = ops.conv2d_fwd(x, w, s, pads)
    yf = ops.conv2d_fwd_bias_relu(x, w, bias, s, pads)
    torch.cuda.synchronize()
    ref = oracle.conv2d_fwd(f64(x), f64(w), s, pads)
    assert_close(f64(y), ref, torch.bfloat16, label="fwd rgbx")
    assert_close(f64(yf), oracle.bias_relu_fwd(ref, f64(bias)), torch.bfloat16, label="fwd+bias+relu rgbx")
    dy = _mk(y.shape, torch.bfloat16, rng)
    dw = ops.conv2d_bwd_filter(x, dy, (KS, KS), s, pads)
    torch.cuda.synchronize()
    assert_close(f64(dw), oracle.conv2d_bwd_filter(f64(x), f64(dy), (KS, KS), s, pads), torch.float32,
                 torch.bfloat16, label="bwd_filter rgbx")


# First layers with at most 4 input channels (bf16) run as band kernels that stage input rows in LDS.
# N, H, W, Cin, Cout, KH, KW, sh, sw, pads
BAND_CASES = [
    # AlexNet conv1 at full image size: 4-row bands, a 3-row last band, one band per workgroup
    ("alexnet_conv1_b3", 3, 224, 224, 3, 64, 11, 11, 4, 4, (2, 2, 2, 2)),
    # more bands than workgroups: the double-buffered band loop runs twice on some workgroups
    ("many_bands", 300, 35, 35, 3, 64, 11, 11, 4, 4, (2, 2, 2, 2)),
    # AlexNet conv1 with 280 bands: the register-filter forward kernel runs its band loop twice on
    # some workgroups (and once on the others)
    ("alexnet_conv1_b20", 20, 224, 224, 3, 64, 11, 11, 4, 4, (2, 2, 2, 2)),
    # two output-channel blocks; a partly empty channel block
    ("cin3_k128_5x5s2", 4, 30, 30, 3, 128, 5, 5, 2, 2, (2, 2, 2, 2)),
    ("cin3_k48_5x5s2", 3, 27, 29, 3, 48, 5, 5, 2, 2, (1, 2, 2, 1)),
    # odd horizontal stride (two 8-byte LDS reads per operand), odd width, asymmetric pads
    ("cin3_7x7s1_oddw", 2, 20, 21, 3, 32, 7, 7, 1, 1, (3, 3, 3, 3)),
    ("cin1_5x5s3", 3, 29, 31, 1, 16, 5, 5, 3, 3, (1, 2, 0, 1)),
    ("cin4_9x9s2", 2, 40, 38, 4, 64, 9, 9, 2, 2, (4, 4, 4, 4)),
    ("cin3_8x1_sh2", 2, 20, 12, 3, 32, 8, 1, 2, 1, (3, 4, 0, 0)),
    # 3x3 first layers: forward band kernel, filter gradient on the folded path (too few taps)
    ("cin3_3x3s1_same", 2, 24, 26, 3, 64, 3, 3, 1, 1, (1, 1, 1, 1)),
    ("cin3_3x3s2_valid", 2, 33, 31, 3, 32, 3, 3, 2, 2, (0, 0, 0, 0)),
]


@pytest.mark.parametrize("case", BAND_CASES, ids=[c[0] for c in BAND_CASES])
def test_conv_first_layer_band(case):
    name, N, H, W, C, K, KH, KW, sh, sw, pads = case
    say("band conv case", name)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    x = _mk((N, H, W, C), torch.bfloat16, rng)
    w = _mk((KH, KW, C, K), torch.bfloat16, rng, np.sqrt(2.0 / (KH * KW * C)))
    bias = torch.from_numpy(rng.standard_normal(K) * 0.5).to(torch.float32).to(DEV)
    y = ops.conv2d_fwd(x, w, (sh, sw), pads)
    yf = ops.conv2d_fwd_bias_relu(x, w, bias, (sh, sw), pads)
    torch.cuda.synchronize()
    ref = oracle.conv2d_fwd(f64(x), f64(w), (sh, sw), pads)
    assert y.shape == ref.shape
    assert_close(f64(y), ref, torch.bfloat16, label="fwd")
    assert_close(f64(yf), oracle.bias_relu_fwd(ref, f64(bias)), torch.bfloat16, label="fwd+bias+relu")
    dy = _mk(y.shape, torch.bfloat16, rng)
    dw = torch.full((KH, KW, C, K), 3.0, device=DEV)          # overwritten, never accumulated into
    ops.conv2d_bwd_filter(x, dy, (KH, KW), (sh, sw), pads, dw=dw)
    torch.cuda.synchronize()
    assert_close(f64(dw), oracle.conv2d_bwd_filter(f64(x), f64(dy), (KH, KW), (sh, sw), pads), torch.float32,
                 torch.bfloat16, label="bwd_filter")


def test_conv_misaligned_base_uses_scalar_path():
    """A view whose base is not 16-byte aligned still computes correctly."""
    rng = np.random.default_rng(9)
    flat = _mk((1 + 2 * 6 * 6 * 16,), torch.bfloat16, rng)
    x = flat[1:].view(2, 6, 6, 16)                           # 2-byte offset
    w = _mk((3, 3, 16, 16), torch.bfloat16, rng, 0.2)
    y = ops.conv2d_fwd(x, w, 1, (1, 1, 1, 1))
    torch.cuda.synchronize()
    assert_close(f64(y), oracle.conv2d_fwd(f64(x), f64(w), 1, (1, 1, 1, 1)), torch.bfloat16, label="misaligned")


# ----------------------------------------------------------------------------- bias + relu
@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("shape,slice_", [((2, 7, 7, 64), None), ((3, 5, 5, 13), None),
                                          ((2, 6, 6, 96), (32, 80)), ((64, 13, 13, 384), None)],
                         ids=["c64", "c13_odd", "slice", "alexnet_conv3"])
def test_bias_relu(dtype, shape, slice_):
    rng = np.random.default_rng(11)
    buf = _mk(shape, dtype, rng)
    y = buf if slice_ is None else buf[..., slice_[0]:slice_[1]]
    C = y.shape[-1]
    b = torch.from_numpy(rng.standard_normal(C) * 0.5).float().to(DEV)
    pre = f64(y)
    ops.bias_relu_fwd(y, b)
    torch.cuda.synchronize()
    got = f64(y)
    assert_close(got, oracle.bias_relu_fwd(pre, f64(b)), dtype, label="bias_relu_fwd")
    assert not np.any(np.signbit(got))
    # the backward on a seeded ReLU output (exact zeros where the mask is off)
    y_in = torch.from_numpy(np.maximum(rng.standard_normal(y.shape), 0.0)).to(dtype)
    y.copy_(y_in.to(DEV))
    dybuf = _mk(buf.shape, dtype, rng)
    dy = dybuf if slice_ is None else dybuf[..., slice_[0]:slice_[1]]
    dy0 = f64(dy)
    dpre, db = ops.bias_relu_bwd(y, dy, dpre=dy)          # in place
    torch.cuda.synchronize()
    ref_dpre, ref_db = oracle.bias_relu_bwd(f64(y_in), dy0)
    assert_close(f64(db), ref_db, torch.float32, dtype, label="db")
    # exact: masked entries are exactly zero, passed entries exactly dy
    assert np.array_equal(f64(dpre), ref_dpre)


# ----------------------------------------------------------------------------- max-pool
def _taps_to_dense(taps, x_shape, k, s, pads):
    """uint8 window taps kh * k + kw -> dense NHWC indices into the pool input."""
    a = taps.cpu().numpy().astype(np.int64)
    N, H, W, C = x_shape
    n, oh, ow, c = np.indices(a.shape)
    h = oh * s - pads[0] + a // k
    w = ow * s - pads[2] + a % k
    return ((n * H + h) * W + w) * C + c


POOL_CASES = [
    ("alexnet_pool1", (2, 55, 55, 64), 3, 2, (0, 0, 0, 0)),
    ("same_3s2", (2, 28, 28, 192), 3, 2, (0, 1, 0, 1)),
    ("branch_3s1", (2, 6, 5, 8), 3, 1, (1, 1, 1, 1)),
    # stride-1 3x3 pools: the backward gather loads its nine candidate windows at once; SAME and
    # VALID padding
    ("inception_3s1", (2, 14, 15, 48), 3, 1, (1, 1, 1, 1)),
    ("valid_3s1", (3, 9, 7, 16), 3, 1, (0, 0, 0, 0)),
    ("odd_c", (2, 8, 8, 5), 2, 2, (0, 0, 0, 0)),
    ("vgg_2s2", (2, 14, 14, 128), 2, 2, (0, 0, 0, 0)),
    # trailing rows/columns that no window reaches (gradient 0 there)
    ("uncovered_tail_3s2", (2, 8, 10, 16), 3, 2, (0, 0, 0, 0)),
    ("uncovered_tail_2s2", (2, 9, 7, 8), 2, 2, (0, 0, 0, 0)),
]


@pytest.mark.parametrize("ties", [False, True], ids=["random", "ties"])
@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("case", POOL_CASES, ids=[c[0] for c in POOL_CASES])
def test_maxpool(case, dtype, ties):
    name, shape, k, s, pads = case
    rng = np.random.default_rng(13)
    a = rng.standard_normal(shape)
    if ties:
        a = np.maximum(np.round(a * 2), 0.0)                 # many exact zeros and repeats
    x = torch.from_numpy(a).to(dtype).to(DEV)
    y, am = ops.maxpool_fwd(x, (k, k), s, pads)
    y8, taps = ops.maxpool_fwd(x, (k, k), s, pads, taps=True)
    torch.cuda.synchronize()
    ref_y, ref_am = oracle.maxpool_fwd(f64(x), (k, k), s, pads)
    assert np.array_equal(f64(y), ref_y) and np.array_equal(f64(y8), ref_y)
    assert np.array_equal(am.cpu().numpy(), ref_am)
    assert taps.dtype == torch.uint8 and np.array_equal(_taps_to_dense(taps, shape, k, s, pads), ref_am)
    dy = _mk(y.shape, dtype, rng)
    for beta in (0.0, 1.0):
        dx = _mk(shape, dtype, rng)
        dx8 = dx.clone()
        old = f64(dx)
        ops.maxpool_bwd(dy, am, dx, (k, k), s, pads, beta=beta)
        ops.maxpool_bwd(dy, taps, dx8, (k, k), s, pads, beta=beta)
        torch.cuda.synchronize()
        ref = oracle.maxpool_bwd(f64(dy), ref_am, shape, dx=old, beta=beta)
        assert_close(f64(dx), ref, dtype, label="maxpool_bwd beta=%g" % beta)
        assert torch.equal(dx, dx8), "the tap form routes exactly as the index form"


@pytest.mark.parametrize("stride", [1, 2])
def test_maxpool_bf16_special_values(stride):
    """bf16 3x3 windows over non-negative values -- exact zeros, repeats, subnormals, the largest
    finite value, +inf -- where the uint8-tap forward orders elements by their bit patterns, and
    chunks with a NaN or a sign bit (-0, a negative) that it leaves to the float scan: outputs
    (NaN where the oracle has one) and selections equal the oracle's, in both argmax forms."""
    rng = np.random.default_rng(41)
    shape, pads = (2, 9, 9, 32), (1, 1, 1, 1)
    vals = np.array([0.0, 0.0, 1.0, 2.0, 2.0, 0.5, 1e-40, 3.0e38, np.inf])
    a = rng.choice(vals, size=shape)
    a[0, 2, 2, 0:8] = np.nan                                  # a NaN that a later tap cannot beat
    a[0, 5, 5, 8] = np.nan
    a[1, 3, 3, 16:24] = -0.0                                   # sign bits: the float scan
    a[1, 6, 6, 24] = -1.0
    x = torch.from_numpy(a).to(torch.bfloat16).to(DEV)
    y, am = ops.maxpool_fwd(x, (3, 3), stride, pads)
    y8, taps = ops.maxpool_fwd(x, (3, 3), stride, pads, taps=True)
    torch.cuda.synchronize()
    ref_y, ref_am = oracle.maxpool_fwd(f64(x), (3, 3), stride, pads)
    for got in (y, y8):
        g = f64(got)
        assert np.array_equal(g, ref_y, equal_nan=True)
        assert np.array_equal(np.signbit(g), np.signbit(ref_y))
    assert np.array_equal(am.cpu().numpy(), ref_am)
    assert np.array_equal(_taps_to_dense(taps, shape, 3, stride, pads), ref_am)


@pytest.mark.parametrize("taps", [False, True], ids=["index", "taps"])
@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("case", POOL_CASES, ids=[c[0] for c in POOL_CASES])
def test_maxpool_relu_bwd_fused(case, dtype, taps):
    """Fused max-pool backward + ReLU backward + bias gradient against the oracle's two ops,
    with the selection stored as dense indices or as uint8 window taps.  With the pool's output
    as the mask (beta = 0: y is not read, NULL; beta = 1: ignored) the result is the same bits."""
    name, shape, k, s, pads = case
    rng = np.random.default_rng(29)
    # the pool input is a ReLU output: exact zeros (masked, and ties inside windows)
    y = torch.from_numpy(np.maximum(rng.standard_normal(shape), 0.0)).to(dtype).to(DEV)
    out, am = ops.maxpool_fwd(y, (k, k), s, pads, taps=taps)
    dy = _mk(out.shape, dtype, rng)
    torch.cuda.synchronize()
    ref_am = oracle.maxpool_fwd(f64(y), (k, k), s, pads)[1]
    for beta in (0.0, 1.0):
        dpre = _mk(shape, dtype, rng)
        dpre_p = dpre.clone()
        old = f64(dpre)
        _, db = ops.maxpool_bwd_relu_bwd(dy, am, y, dpre, (k, k), s, pads, beta=beta)
        _, db_p = ops.maxpool_bwd_relu_bwd(dy, am, None if beta == 0 else y, dpre_p, (k, k), s, pads, beta=beta,
                                           py=out)
        torch.cuda.synchronize()
        assert torch.equal(dpre_p, dpre) and torch.equal(db_p, db), "mask from the pool output"
        g = oracle.maxpool_bwd(f64(dy), ref_am, shape, dx=old, beta=beta)
        ref_dpre, ref_db = oracle.bias_relu_bwd(f64(y), g)
        assert_close(f64(dpre), ref_dpre, dtype, label="fused dpre beta=%g" % beta)
        assert np.all(f64(dpre)[f64(y) <= 0] == 0), "masked entries must be exactly zero"
        assert_close(f64(db), ref_db, torch.float32, dtype, label="fused db beta=%g" % beta)
        # the bias gradient is the column sum of the stored dpre (fp32 accumulation of it)
        assert err(f64(db), f64(dpre).sum(axis=(0, 1, 2))) <= 1e-4


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
def test_maxpool_slice_views(dtype):
    """Pool output written into a concat slice; its gradient read from one."""
    rng = np.random.default_rng(17)
    x = _mk((2, 9, 9, 32), dtype, rng)
    cat = torch.zeros((2, 4, 4, 80), dtype=dtype, device=DEV)
    y = cat[..., 40:72]
    _, am = ops.maxpool_fwd(x, (3, 3), 2, (0, 0, 0, 0), y=y)
    torch.cuda.synchronize()
    ref_y, ref_am = oracle.maxpool_fwd(f64(x), (3, 3), 2, (0, 0, 0, 0))
    assert np.array_equal(f64(y), ref_y) and np.array_equal(am.cpu().numpy(), ref_am)
    gcat = _mk((2, 4, 4, 80), dtype, rng)
    dy = gcat[..., 40:72]
    dx = torch.empty_like(x)
    ops.maxpool_bwd(dy, am, dx, (3, 3), 2, (0, 0, 0, 0))
    torch.cuda.synchronize()
    assert_close(f64(dx), oracle.maxpool_bwd(f64(dy), ref_am, x.shape), dtype, label="maxpool_bwd slice")
    # the fused ReLU backward with the mask from the pool output held in the concat slice
    xr = torch.relu(x)
    _, am_r = ops.maxpool_fwd(xr, (3, 3), 2, (0, 0, 0, 0), y=y)
    d1, d2 = torch.empty_like(x), torch.empty_like(x)
    _, db1 = ops.maxpool_bwd_relu_bwd(dy, am_r, xr, d1, (3, 3), 2, (0, 0, 0, 0))
    _, db2 = ops.maxpool_bwd_relu_bwd(dy, am_r, None, d2, (3, 3), 2, (0, 0, 0, 0), py=y)
    torch.cuda.synchronize()
    assert torch.equal(d1, d2) and torch.equal(db1, db2)
    g = oracle.maxpool_bwd(f64(dy), oracle.maxpool_fwd(f64(xr), (3, 3), 2, (0, 0, 0, 0))[1], x.shape)
    assert_close(f64(d2), oracle.bias_relu_bwd(f64(xr), g)[0], dtype, label="maxpool_relu_bwd slice py")


# ----------------------------------------------------------------------------- sgd
@pytest.mark.parametrize("n", [1, 1001, 2469696])
def test_apply_sgd_one_ulp_and_shadow(n):
    rng = np.random.default_rng(19)
    v = torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(DEV)
    g = torch.from_numpy(rng.standard_normal(n).astype(np.float32) * 10).to(DEV)
    v0, g0 = v.cpu().numpy().astype(np.float64), g.cpu().numpy().astype(np.float64)
    sh = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    lr = float(np.float32(0.01))
    ops.apply_sgd(v, g, lr, shadow=sh)
    torch.cuda.synchronize()
    ref = oracle.apply_sgd(v0, g0, lr)
    assert ulp_diff_f32(v.cpu().numpy(), ref) <= 1
    assert torch.equal(sh, v.to(torch.bfloat16))            # bf16 shadow = RNE of the new value


def test_apply_sgd_multi():
    rng = np.random.default_rng(23)
    sizes = [0, 5, 1024, 1025, 3000] + [17] * 20               # more than one launch batch
    vs = [torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(DEV) for n in sizes]
    gs = [torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(DEV) for n in sizes]
    shs = [torch.empty(n, dtype=torch.bfloat16, device=DEV) if i % 2 else None for i, n in enumerate(sizes)]
    before = [v.cpu().numpy().astype(np.float64) for v in vs]
    ops.apply_sgd_multi(vs, gs, 0.045, shs)
    torch.cuda.synchronize()
    for v, g, b, sh in zip(vs, gs, before, shs):
        ref = oracle.apply_sgd(b, g.cpu().numpy().astype(np.float64), float(np.float32(0.045)))
        assert ulp_diff_f32(v.cpu().numpy(), ref) <= 1
        if sh is not None:
            assert torch.equal(sh, v.to(torch.bfloat16))


# ----------------------------------------------------------------------------- momentum, adam
# Error bounds from the fp32 arithmetic of the kernels (u = 2^-24, the unit roundoff), against the
# fp64 oracle fed the same fp32 inputs and the fp32-rounded scalars:
#   velocity  fma(m, a, g)                one rounding                 0.5 ulp -> at most 1 ulp after fp32(ref)
#   var       fma(-lr, s, var)            2u|var'| + lr * (error of s)
#   Adam m    fma(b1, m, fl(fl(1-b1) g))  three roundings              4u (|m'| + (1-b1)|g|)
#   Adam v    sum of non-negative terms                                8u |v'|
#   Adam step lr/(1-b1^t) m / (sqrt(v/(1-b2^t)) + eps): about eight roundings on top of m's error
U = 2.0 ** -24


def _momentum_case(n, seed, offset=0):
    rng = np.random.default_rng(seed)
    mk = lambda scale: torch.from_numpy((rng.standard_normal(n + offset) * scale).astype(np.float32)).to(DEV)[offset:]
    return mk(1.0), mk(0.5), mk(3.0)


@pytest.mark.parametrize("nesterov", [False, True])
@pytest.mark.parametrize("n,offset", [(1, 0), (1001, 0), (1003, 1), (2469696, 0)])
def test_apply_momentum_matches_oracle(n, offset, nesterov):
    say("momentum", n, offset, nesterov)
    var, acc, g = _momentum_case(n, 40 + n % 7, offset)
    v0, a0, g0 = (t.cpu().numpy().astype(np.float64) for t in (var, acc, g))
    lr, mom = float(np.float32(0.01)), float(np.float32(0.9))
    sh = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    ops.apply_momentum(var, acc, g, lr, mom, nesterov=nesterov, shadow=sh)
    torch.cuda.synchronize()
    rv, ra = oracle.apply_momentum(v0, a0, g0, lr, mom, nesterov)
    assert ulp_diff_f32(acc.cpu().numpy(), ra) <= 1
    s_mag = np.abs(g0) + 2 * mom * np.abs(ra) if nesterov else np.abs(ra)
    tol = 2 * U * np.abs(rv) + lr * 4 * U * s_mag + 1e-38
    d = np.abs(var.cpu().numpy().astype(np.float64) - rv)
    assert np.all(d <= tol), float(np.max(d / tol))
    assert torch.equal(sh, var.to(torch.bfloat16))


def _adam_bounds(rv, rm, rvv, g0, lr, b1, b2, eps, t):
    tol_m = 4 * U * (np.abs(rm) + (1 - b1) * np.abs(g0)) + 1e-38
    tol_v = 8 * U * rvv + 1e-38
    c1, c2 = 1 - b1 ** t, 1 - b2 ** t
    den = np.sqrt(rvv / c2) + eps
    step = lr / c1 * np.abs(rm) / den
    tol_var = 2 * U * np.abs(rv) + 16 * U * step + lr / c1 * tol_m / den + 1e-38
    return tol_m, tol_v, tol_var


@pytest.mark.parametrize("t", [1, 2, 1000])
@pytest.mark.parametrize("n,offset", [(1, 0), (1001, 0), (1003, 1), (2469696, 0)])
def test_apply_adam_matches_oracle(n, offset, t):
    say("adam", n, offset, t)
    rng = np.random.default_rng(60 + t)
    mk = lambda x: torch.from_numpy(x.astype(np.float32)).to(DEV)[offset:]
    var = mk(rng.standard_normal(n + offset))
    m = mk(rng.standard_normal(n + offset) * 0.1)
    v = mk(np.abs(rng.standard_normal(n + offset)) * 0.01)
    g = mk(rng.standard_normal(n + offset) * 0.2)
    v0, m0, vv0, g0 = (x.cpu().numpy().astype(np.float64) for x in (var, m, v, g))
    f = lambda x: float(np.float32(x))
    lr, b1, b2, eps = f(0.001), f(0.9), f(0.999), f(1e-8)
    sh = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    ops.apply_adam(var, m, v, g, lr, b1, b2, eps, t, shadow=sh)
    torch.cuda.synchronize()
    rv, rm, rvv = oracle.apply_adam(v0, m0, vv0, g0, lr, b1, b2, eps, t)
    tol_m, tol_v, tol_var = _adam_bounds(rv, rm, rvv, g0, lr, b1, b2, eps, t)
    for name, got, ref, tol in (("m", m, rm, tol_m), ("v", v, rvv, tol_v), ("var", var, rv, tol_var)):
        d = np.abs(got.cpu().numpy().astype(np.float64) - ref)
        assert np.all(d <= tol), (name, float(np.max(d / tol)))
    assert torch.equal(sh, var.to(torch.bfloat16))


def test_adam_and_momentum_steps_from_zero_state():
    """Five steps from zero slots, the way a training loop starts, against five oracle steps."""
    rng = np.random.default_rng(71)
    n = 4099
    gs = [rng.standard_normal(n).astype(np.float32) * 0.3 for _ in range(5)]
    x0 = rng.standard_normal(n).astype(np.float32)
    f = lambda x: float(np.float32(x))
    var = torch.from_numpy(x0).to(DEV)
    m, v = torch.zeros(n, device=DEV), torch.zeros(n, device=DEV)
    rv, rm, rvv = x0.astype(np.float64), np.zeros(n), np.zeros(n)
    for t, g in enumerate(gs, start=1):
        ops.apply_adam(var, m, v, torch.from_numpy(g).to(DEV), f(0.01), f(0.9), f(0.999), f(1e-8), t)
        rv, rm, rvv = oracle.apply_adam(rv, rm, rvv, g.astype(np.float64), f(0.01), f(0.9), f(0.999), f(1e-8), t)
    torch.cuda.synchronize()
    # each step adds its own rounding; the first-order error growth over 5 steps stays linear
    _, _, tol = _adam_bounds(rv, rm, rvv, gs[-1].astype(np.float64), f(0.01), f(0.9), f(0.999), f(1e-8), 5)
    d = np.abs(var.cpu().numpy().astype(np.float64) - rv)
    assert np.all(d <= 5 * tol + 5 * 32 * U * f(0.01)), float(np.max(d))
    var = torch.from_numpy(x0).to(DEV)
    acc = torch.zeros(n, device=DEV)
    rv, ra = x0.astype(np.float64), np.zeros(n)
    for g in gs:
        ops.apply_momentum(var, acc, torch.from_numpy(g).to(DEV), f(0.01), f(0.9), nesterov=True)
        rv, ra = oracle.apply_momentum(rv, ra, g.astype(np.float64), f(0.01), f(0.9), True)
    torch.cuda.synchronize()
    bound = 5 * (2 * U * np.abs(rv) + 0.01 * 16 * U * (np.abs(ra) * 6 + 2.0))
    assert np.all(np.abs(var.cpu().numpy().astype(np.float64) - rv) <= bound)
    # the velocity is a signed sum over the steps: each step's rounding (at most u times the
    # magnitudes it adds) is carried forward, so the bound is absolute, not in ulps of the result
    gmax = max(float(np.max(np.abs(g))) for g in gs)
    vbound = 5 * 2 * U * (np.abs(ra) + 5 * gmax)
    assert np.all(np.abs(acc.cpu().numpy().astype(np.float64) - ra) <= vbound)


# ----------------------------------------------------------------------------- softmax cross-entropy
SOFTMAX_CASES = [("one_class", 1, 1), ("small", 5, 13), ("alexnet_b128", 128, 1000), ("ragged_rows", 7, 1000),
                 ("wide_rows", 3, 4097)]


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("bias", [False, True], ids=["nobias", "bias"])
@pytest.mark.parametrize("case", SOFTMAX_CASES, ids=[c[0] for c in SOFTMAX_CASES])
def test_softmax_xent(case, bias, dtype):
    name, n, c = case
    say("softmax_xent", name, bias, dtype)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    z = _mk((n, c), dtype, rng, 3.0)
    b = torch.from_numpy(rng.standard_normal(c)).float().to(DEV) if bias else None
    lab_np = rng.integers(0, c, size=n).astype(np.int32)
    lab_np[0] = c - 1                              # the edge classes
    if n > 1:
        lab_np[1] = 0
    lab = torch.from_numpy(lab_np).to(DEV)
    loss, dz = ops.softmax_xent(z, lab, 1.0 / n, bias=b)
    torch.cuda.synchronize()
    rows, ref = oracle.softmax_xent(f64(z), lab_np, 1.0 / n, bias=None if b is None else f64(b))
    assert_close(f64(loss), rows, torch.float32, label="loss rows")
    assert_close(f64(dz), ref, dtype, torch.float32, label="dlogits")
    # in place, and shifted by +1000 (the max is taken out: the same loss and gradient)
    z2 = z.clone()
    loss2, _ = ops.softmax_xent(z2, lab, 1.0 / n, bias=b, dlogits=z2)
    torch.cuda.synchronize()
    assert torch.equal(loss2, loss) and torch.equal(z2, dz)
    if dtype == torch.float32 and b is None:
        # (without a bias: with one, the kernel's fp32 sum logit + bias at magnitude 1000 rounds by
        # up to 2^-14, an error of the inputs' scale that the oracle's fp64 sum does not make)
        zs = z + 1000.0
        loss3, dz3 = ops.softmax_xent(zs, lab, 1.0 / n, bias=b)
        torch.cuda.synchronize()
        rows3, ref3 = oracle.softmax_xent(f64(zs), lab_np, 1.0 / n, bias=None if b is None else f64(b))
        assert np.all(np.isfinite(f64(loss3)))
        # the shifted fp32 logits carry an absolute rounding of up to 2^-14: the bound is the
        # oracle's on those same rounded logits
        assert_close(f64(loss3), rows3, torch.float32, label="loss rows +1000")
        assert_close(f64(dz3), ref3, torch.float32, label="dlogits +1000")


def test_softmax_xent_bad_labels_give_nan_rows():
    rng = np.random.default_rng(77)
    z = _mk((4, 10), torch.float32, rng)
    lab = torch.tensor([3, -1, 10, 0], dtype=torch.int32, device=DEV)
    loss, dz = ops.softmax_xent(z, lab, 0.25)
    torch.cuda.synchronize()
    l = loss.cpu().numpy()
    assert np.isnan(l[1]) and np.isnan(l[2]) and np.all(np.isfinite(l[[0, 3]]))
    assert bool(torch.isnan(dz[1:3]).all()) and bool(torch.isfinite(dz[[0, 3]]).all())


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", [(128, 1, 1, 1000), (64, 1, 1, 40000)], ids=["c1000", "c40000"])
def test_bias_only_backward(dtype, shape):
    """y = NULL: dpre = dy and the bias gradient is the column sums of dy (a logits layer; 40000
    classes: wider than one block's LDS holds)."""
    rng = np.random.default_rng(78)
    dy = _mk(shape, dtype, rng)
    dy0 = dy.clone()
    dpre, db = ops.bias_relu_bwd(None, dy, dpre=dy)
    torch.cuda.synchronize()
    assert torch.equal(dpre, dy0)
    assert_close(f64(db), f64(dy0).sum(axis=(0, 1, 2)), torch.float32, dtype, label="db")


# x shape, cout, conv (k, stride, pads), pool (k, stride, pads), dtype, pool output as a channel slice
CONV_POOL_CASES = [
    # one kernel: one band per image (13 x 13 of 192 rows), bands sharing a row (3x3/2 windows, four
    # 7-row bands of 18 columns), non-overlapping 2x2/2 windows in 4-row bands, a last output row no
    # window reaches (a band that only writes y), several channel tiles, ragged channel tiles
    ("alexnet_conv5_pool5", (3, 13, 13, 256), 256, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("bands_sharing_rows", (2, 25, 18, 32), 64, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("bands_2x2s2", (2, 32, 32, 32), 128, (3, 1, (1, 1, 1, 1)), (2, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("uncovered_last_row", (2, 33, 32, 32), 64, (3, 1, (1, 1, 1, 1)), (2, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("ragged_channels", (2, 13, 13, 64), 72, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("pool_into_channel_slice", (2, 13, 13, 64), 128, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 0, 0, 0)), torch.bfloat16,
     True),
    # two kernels: too many recomputed rows (AlexNet conv2 + pool2), a grid of several rounds of
    # blocks (588 128 x 128 tiles), rows too wide for a band, a padded pool, fp32
    ("alexnet_conv2_pool2", (3, 27, 27, 64), 192, (5, 1, (2, 2, 2, 2)), (3, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("several_rounds", (24, 56, 56, 16), 128, (3, 1, (1, 1, 1, 1)), (2, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("wide_rows", (2, 10, 100, 32), 64, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 0, 0, 0)), torch.bfloat16, False),
    ("same_pool", (2, 14, 14, 32), 64, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 1, 0, 1)), torch.bfloat16, False),
    ("f32", (2, 13, 13, 32), 64, (3, 1, (1, 1, 1, 1)), (3, 2, (0, 0, 0, 0)), torch.float32, False),
]


@pytest.mark.parametrize("ties", [False, True], ids=["random", "ties"])
@pytest.mark.parametrize("case", CONV_POOL_CASES, ids=[c[0] for c in CONV_POOL_CASES])
def test_conv_bias_relu_maxpool(case, ties):
    """The convolution with bias + ReLU and the max-pool of its output in one call: bit for bit the
    two calls it replaces (tfk_conv2d_fwd_bias_relu, then tfk_maxpool_fwd_taps), and against the
    oracle (y within the gate; the pool of the oracle's rounded y, taps equal wherever the window's
    two largest values are not within the gate of each other).  With ties, a third of the channels
    get a bias that zeroes them after the ReLU (every window a tie)."""
    name, xs, cout, (k, st, pads), (pk, ps, ppads), dt, sliced = case
    say("conv + bias + relu + maxpool", name, "ties" if ties else "")
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    x = torch.from_numpy(np.maximum(rng.standard_normal(xs), 0)).to(dt).to(DEV)
    w = torch.from_numpy(rng.standard_normal((k, k, xs[3], cout)) * np.sqrt(2.0 / (k * k * xs[3]))).to(dt).to(DEV)
    b = rng.standard_normal(cout) * 0.1
    if ties:
        b[::3] = -1e4
    bias = torch.from_numpy(b.astype(np.float32)).to(DEV)
    y, py, taps = ops.conv2d_fwd_bias_relu_maxpool(x, w, bias, st, pads, (pk, pk), ps, ppads)
    if sliced:
        big = torch.full(py.shape[:3] + (cout + 48,), -7.0, dtype=dt, device=DEV)
        pys = big[..., 16:16 + cout]
        ops.conv2d_fwd_bias_relu_maxpool(x, w, bias, st, pads, (pk, pk), ps, ppads, py=pys, taps=taps)
        torch.cuda.synchronize()
        assert torch.equal(pys, py) and bool((big[..., :16] == -7).all()) and bool((big[..., 16 + cout:] == -7).all())
    y2 = ops.conv2d_fwd_bias_relu(x, w, bias, st, pads)
    py2, taps2 = ops.maxpool_fwd(y2, (pk, pk), ps, ppads, taps=True)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16) if dt == torch.bfloat16 else y.view(torch.int32),
                       y2.view(torch.int16) if dt == torch.bfloat16 else y2.view(torch.int32))
    assert torch.equal(py, py2) and torch.equal(taps, taps2)
    ref = oracle.bias_relu_fwd(oracle.conv2d_fwd(f64(x), f64(w), st, pads), b.astype(np.float32).astype(np.float64))
    assert_close(f64(y), ref, dt, label=name + " y")
    yr = torch.from_numpy(ref).to(dt).to(torch.float64).numpy()
    pref, am = oracle.maxpool_fwd(yr, (pk, pk), ps, ppads)
    assert_close(f64(py), pref, dt, label=name + " pool")
    n, oh, ow, c = pref.shape
    t = taps.cpu().numpy().astype(np.int64)
    nn, qq, ww, cc = np.indices(t.shape)
    h = qq * ps - ppads[0] + t // pk
    wv = ww * ps - ppads[2] + t % pk
    dense = ((nn * yr.shape[1] + h) * yr.shape[2] + wv) * c + cc
    yp = np.pad(yr, ((0, 0), (ppads[0], ppads[1]), (ppads[2], ppads[3]), (0, 0)), constant_values=-np.inf)
    wins = np.sort(np.stack([yp[:, i:i + ps * (oh - 1) + 1:ps, j:j + ps * (ow - 1) + 1:ps, :]
                             for i in range(pk) for j in range(pk)]), axis=0)
    rms = float(np.sqrt(np.mean(yr * yr)))
    tie = (wins[-1] - wins[-2]) <= 2 * (2.0 ** -7 * np.abs(wins[-1]) + 1e-3 * rms)
    bad = (dense != am) & ~tie
    say("  taps: %d differ from the oracle, all at near-ties" % int(np.sum(dense != am)))
    assert not bad.any()


# ----------------------------------------------------------------------------- deferred bias gradients
def test_deferred_bias_gradients_bitwise():
    """Every bias-gradient producer called with defer=True leaves its partials in its own
    workspace; one bias_grad_finish over all of them (more than one launch batch of 32, an empty
    tensor among them) must give the bits the immediate calls give, and the same dpre."""
    rng = np.random.default_rng(41)
    bf = torch.bfloat16
    jobs, want, keep = [], [], []

    def ws_for(need):
        # (each workspace holds its call's partials until the finish: kept alive here)
        keep.append(torch.zeros(max(16, need), dtype=torch.uint8, device=DEV))
        return keep[-1]

    for rep in range(9):
        # ReLU backward, a channel slice of a wider tensor, and bias only
        buf = torch.from_numpy(np.maximum(rng.standard_normal((4, 13, 13, 96)), 0)).to(bf).to(DEV)
        y = buf[..., 16:80]
        dy = _mk(buf.shape, bf, rng)[..., 16:80]
        d1 = torch.empty_like(buf)[..., 16:80]
        d2 = torch.empty_like(buf)[..., 16:80]
        _, db1 = ops.bias_relu_bwd(y, dy, dpre=d1)
        _, part = ops.bias_relu_bwd(y, dy, dpre=d2, ws=ws_for(ops.bias_relu_bwd_workspace_bytes(y)), defer=True)
        assert torch.equal(d1, d2)
        jobs.append((part, torch.empty(64, device=DEV))); want.append(db1)
        g = _mk((3, 5, 7, 24), bf, rng)
        _, db1 = ops.bias_relu_bwd(None, g, dpre=g.clone())
        _, part = ops.bias_relu_bwd(None, g, dpre=g.clone(), ws=ws_for(ops.bias_relu_bwd_workspace_bytes(g)),
                                    defer=True)
        jobs.append((part, torch.empty(24, device=DEV))); want.append(db1)
        # pool + ReLU backward (tap and index selections)
        x = torch.from_numpy(np.maximum(rng.standard_normal((2, 27, 27, 64)), 0)).to(bf).to(DEV)
        for taps in (True, False):
            out, am = ops.maxpool_fwd(x, (3, 3), 2, (0, 0, 0, 0), taps=taps)
            dyp = _mk(out.shape, bf, rng)
            p1, p2 = torch.empty_like(x), torch.empty_like(x)
            _, db1 = ops.maxpool_bwd_relu_bwd(dyp, am, x, p1, (3, 3), 2, (0, 0, 0, 0))
            _, part = ops.maxpool_bwd_relu_bwd(dyp, am, x, p2, (3, 3), 2, (0, 0, 0, 0),
                                               ws=ws_for(ops.bias_relu_bwd_workspace_bytes(p2)), defer=True)
            assert torch.equal(p1, p2)
            jobs.append((part, torch.empty(64, device=DEV))); want.append(db1)
        # input gradient fused with the ReLU backward: the pipelined kernel and the split path
        for (n, h, cin, cout, k) in ((4, 13, 192, 384, 3), (2, 4, 24, 1024, 1)):
            yv = torch.from_numpy(np.maximum(rng.standard_normal((n, h, h, cin)), 0)).to(bf).to(DEV)
            w = (torch.from_numpy(rng.standard_normal((k, k, cin, cout)) * 0.05)).to(bf).to(DEV)
            dyc = _mk((n, h, h, cout), bf, rng)
            p1, p2 = torch.empty_like(yv), torch.empty_like(yv)
            pd = k // 2
            _, db1 = ops.conv2d_bwd_input_relu_bwd(dyc, w, yv, p1, (1, 1), (pd, pd, pd, pd))
            need = ops.conv2d_workspace_bytes(3, yv, cout, k, k, (1, 1), (pd, pd, pd, pd))
            _, part = ops.conv2d_bwd_input_relu_bwd(dyc, w, yv, p2, (1, 1), (pd, pd, pd, pd), ws=ws_for(need),
                                                    defer=True)
            assert torch.equal(p1, p2)
            jobs.append((part, torch.empty(cin, device=DEV))); want.append(db1)
    # an empty tensor: no partials, bias gradient 0
    e = torch.zeros((0, 4, 4, 8), dtype=bf, device=DEV)
    _, part = ops.bias_relu_bwd(e, e, dpre=e, ws=ws_for(16), defer=True)
    assert part.rows == 0
    jobs.append((part, torch.full((8,), 7.0, device=DEV))); want.append(torch.zeros(8, device=DEV))
    assert len(jobs) > 32
    ops.bias_grad_finish(jobs)
    torch.cuda.synchronize()
    for i, ((_, got), ref) in enumerate(zip(jobs, want)):
        assert torch.equal(got.view(torch.int32), ref.view(torch.int32)), i
