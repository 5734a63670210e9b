"""Synthetic convnet workloads and their seeded inputs.

This module is shared by the HIP step driver, the tests, the bench and the
CPU oracle's step composition.  It holds *descriptions* only: layer tables,
tensor shapes used for buffer bookkeeping, and seeded random draws.  It does no
convolution, pooling, activation or update arithmetic of its own.

Network description
-------------------
A net is a list of ops in forward (topological) order over named NHWC tensors.

* ``Conv``: 2-D cross-correlation of a whole source tensor with an HWIO filter,
  followed by bias-add and ReLU (every conv in these workloads is followed by
  both).  Its result lands in ``dst`` at channel offset ``dst_c0``; a ``dst``
  wider than ``cout`` is a channel-concat buffer shared by the branches of an
  inception module (the paper's "mini-batch 2-D convolution takes two 4-D
  tensors and produces another", Section 3.1; concatenation is expressed as
  writes into channel slices instead of a copy).
* ``Pool``: max-pool of a whole source tensor into ``dst`` at ``dst_c0``.

Padding is always explicit ``(top, bottom, left, right)``.  The "SAME" helper
below puts the odd extra row/column at the bottom/right.

Seeded inputs (one PCG64 stream per workload, default seed 0): the image ``x``
is drawn first, then every conv filter in op order (He-normal, untruncated,
std = sqrt(2 / (KH*KW*Cin))), then the upstream gradient ``g`` of the net's
output tensor.  Biases are zeros and are not drawn.  All draws are float64.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import numpy as np

Pads = Tuple[int, int, int, int]


@dataclass(frozen=True)
class Conv:
    name: str
    src: str
    dst: str
    dst_c0: int
    cout: int
    kh: int
    kw: int
    sh: int
    sw: int
    pads: Pads
    relu: bool = True               # False: bias only (the logits layer of a classifier)


@dataclass(frozen=True)
class Pool:
    name: str
    src: str
    dst: str
    dst_c0: int
    kh: int
    kw: int
    sh: int
    sw: int
    pads: Pads


@dataclass
class Net:
    """A workload: input tensor ``x``, ops in forward order, output tensor."""

    name: str
    dtype: str                      # "f32" or "bf16": activation / filter storage type
    lr: float                       # SGD learning rate (fp32 value)
    input_grad: bool                # compute dX of convs that read the step input
    tensors: Dict[str, Tuple[int, int, int, int]] = field(default_factory=dict)
    ops: List[object] = field(default_factory=list)
    output: str = ""
    loss: str = "surrogate"         # "surrogate": L = <g, out>; "softmax_xent": mean cross-entropy
    classes: int = 0                # softmax_xent: the output tensor is (N, 1, 1, classes) logits

    @property
    def convs(self) -> List[Conv]:
        return [o for o in self.ops if isinstance(o, Conv)]

    def param_count(self) -> int:
        n = 0
        for c in self.convs:
            cin = self.tensors[c.src][3]
            n += c.kh * c.kw * cin * c.cout + c.cout
        return n


def out_len(n: int, k: int, s: int, p0: int, p1: int) -> int:
    """Window count along one axis: floor((n + p0 + p1 - k) / s) + 1 (buffer bookkeeping)."""
    return (n + p0 + p1 - k) // s + 1


def same_pads(h: int, w: int, kh: int, kw: int, sh: int, sw: int) -> Pads:
    """SAME padding: ceil(n/s) outputs, the odd extra pad row/column at the bottom/right."""
    def one(n, k, s):
        o = -(-n // s)
        tot = max((o - 1) * s + k - n, 0)
        return tot // 2, tot - tot // 2
    pt, pb = one(h, kh, sh)
    pl, pr = one(w, kw, sw)
    return (pt, pb, pl, pr)


VALID: Pads = (0, 0, 0, 0)


class _Builder:
    def __init__(self, name, dtype, lr, input_grad, x_shape):
        self.net = Net(name, dtype, lr, input_grad)
        self.net.tensors["x"] = tuple(x_shape)
        self._k = 0

    def _fresh(self, prefix):
        self._k += 1
        return f"{prefix}{self._k}"

    def _spatial(self, src, kh, kw, sh, sw, pads):
        n, h, w, _ = self.net.tensors[src]
        if pads == "SAME":
            pads = same_pads(h, w, kh, kw, sh, sw)
        oh = out_len(h, kh, sh, pads[0], pads[1])
        ow = out_len(w, kw, sw, pads[2], pads[3])
        return n, oh, ow, tuple(pads)

    def conv(self, src, cout, kh, kw=None, s=1, pads=VALID, dst=None, c0=0, name=None):
        kw = kh if kw is None else kw
        n, oh, ow, pads = self._spatial(src, kh, kw, s, s, pads)
        name = name or self._fresh("conv")
        if dst is None:
            dst = name
            self.net.tensors[dst] = (n, oh, ow, cout)
        else:
            assert self.net.tensors[dst][:3] == (n, oh, ow), (name, dst)
        self.net.ops.append(Conv(name, src, dst, c0, cout, kh, kw, s, s, pads))
        return dst

    def fc(self, src, cout, relu=True, name=None):
        """A fully connected layer: a VALID convolution whose window is the whole input image."""
        n, h, w, _ = self.net.tensors[src]
        name = name or self._fresh("fc")
        self.net.tensors[name] = (n, 1, 1, cout)
        self.net.ops.append(Conv(name, src, name, 0, cout, h, w, 1, 1, VALID, relu))
        return name

    def pool(self, src, k, s, pads=VALID, dst=None, c0=0, name=None):
        n, oh, ow, pads = self._spatial(src, k, k, s, s, pads)
        name = name or self._fresh("pool")
        c = self.net.tensors[src][3]
        if dst is None:
            dst = name
            self.net.tensors[dst] = (n, oh, ow, c)
        else:
            assert self.net.tensors[dst][:3] == (n, oh, ow), (name, dst)
        self.net.ops.append(Pool(name, src, dst, c0, k, k, s, s, pads))
        return dst

    def concat_buffer(self, like_spatial_of, hw, c):
        name = self._fresh("cat")
        n = self.net.tensors[like_spatial_of][0]
        self.net.tensors[name] = (n, hw[0], hw[1], c)
        return name

    def done(self, out):
        self.net.output = out
        return self.net

    def softmax_done(self, logits, classes):
        self.net.output = logits
        self.net.loss = "softmax_xent"
        self.net.classes = classes
        assert self.net.tensors[logits][1:] == (1, 1, classes)
        return self.net


# ----------------------------------------------------------------------------- C1
def single_layer(batch=8, hw=32, cin=16, cout=32) -> Net:
    """Single conv layer SGD step, fp32: conv3x3/1 SAME, bias+ReLU, 2x2/2 max-pool."""
    b = _Builder("single_layer_fp32", "f32", 0.01, True, (batch, hw, hw, cin))
    y = b.conv("x", cout, 3, s=1, pads="SAME", name="conv1")
    p = b.pool(y, 2, 2, VALID, name="pool1")
    return b.done(p)


# ----------------------------------------------------------------------------- C2
def alexnet(batch=128, classifier=False) -> Net:
    """AlexNet-shaped conv stack, bf16: 11x11/4 p2 64, pool 3/2, 5x5 p2 192, pool, 3x3 384, 256, 256, pool.
    With ``classifier``: then fc 4096 + ReLU, fc 4096 + ReLU, fc 1000 logits and the softmax
    cross-entropy of 1000 classes (no dropout)."""
    # (the He-initialised classifier on N(0, 1) images diverges at lr 0.01; 1e-4 lowers its loss)
    b = _Builder("alexnet%s_b%d" % ("_cls" if classifier else "", batch), "bf16", 1e-4 if classifier else 0.01,
                 False, (batch, 224, 224, 3))
    t = b.conv("x", 64, 11, s=4, pads=(2, 2, 2, 2), name="conv1")
    t = b.pool(t, 3, 2, name="pool1")
    t = b.conv(t, 192, 5, pads=(2, 2, 2, 2), name="conv2")
    t = b.pool(t, 3, 2, name="pool2")
    t = b.conv(t, 384, 3, pads=(1, 1, 1, 1), name="conv3")
    t = b.conv(t, 256, 3, pads=(1, 1, 1, 1), name="conv4")
    t = b.conv(t, 256, 3, pads=(1, 1, 1, 1), name="conv5")
    t = b.pool(t, 3, 2, name="pool5")
    if classifier:
        t = b.fc(t, 4096, name="fc6")
        t = b.fc(t, 4096, name="fc7")
        t = b.fc(t, 1000, relu=False, name="fc8")
        return b.softmax_done(t, 1000)
    return b.done(t)


def classifier_small(batch=4, dtype="f32") -> Net:
    """A small classifier for finite differences and parity: conv3x3 p1 8 + pool 2/2, fc 16 + ReLU,
    fc 10 logits, softmax cross-entropy (input gradient included)."""
    b = _Builder("classifier_small_%s" % dtype, dtype, 0.01, True, (batch, 8, 8, 4))
    t = b.conv("x", 8, 3, pads=(1, 1, 1, 1), name="conv1")
    t = b.pool(t, 2, 2, name="pool1")
    t = b.fc(t, 16, name="fc1")
    t = b.fc(t, 10, relu=False, name="fc2")
    return b.softmax_done(t, 10)


# ----------------------------------------------------------------------------- C3
def vgg16(batch=64, hw=224) -> Net:
    """VGG-16-shaped stack, bf16: 13 conv3x3 p1, 2x2/2 pool after each block."""
    b = _Builder("vgg16_b%d" % batch, "bf16", 0.01, False, (batch, hw, hw, 3))
    t = "x"
    k = 0
    for blk, widths in enumerate([(64, 64), (128, 128), (256,) * 3, (512,) * 3, (512,) * 3]):
        for c in widths:
            k += 1
            t = b.conv(t, c, 3, pads=(1, 1, 1, 1), name="conv%d" % k)
        t = b.pool(t, 2, 2, name="pool%d" % (blk + 1))
    return b.done(t)


# ----------------------------------------------------------------------------- C4
GOOGLENET_MODULES = [
    # name, #1x1, #3x3red, #3x3, #5x5red, #5x5, pool-proj
    ("3a", 64, 96, 128, 16, 32, 32),
    ("3b", 128, 128, 192, 32, 96, 64),
    ("4a", 192, 96, 208, 16, 48, 64),
    ("4b", 160, 112, 224, 24, 64, 64),
    ("4c", 128, 128, 256, 24, 64, 64),
    ("4d", 112, 144, 288, 32, 64, 64),
    ("4e", 256, 160, 320, 32, 128, 128),
    ("5a", 256, 160, 320, 32, 128, 128),
    ("5b", 384, 192, 384, 48, 128, 128),
]


def _inception_v1(b: _Builder, src, m):
    name, c1, c3r, c3, c5r, c5, cp = m
    n, h, w, _ = b.net.tensors[src]
    cat = b.concat_buffer(src, (h, w), c1 + c3 + c5 + cp)
    b.net.tensors[cat] = (n, h, w, c1 + c3 + c5 + cp)
    b.conv(src, c1, 1, dst=cat, c0=0, name=f"m{name}_1x1")
    r = b.conv(src, c3r, 1, name=f"m{name}_3x3r")
    b.conv(r, c3, 3, pads=(1, 1, 1, 1), dst=cat, c0=c1, name=f"m{name}_3x3")
    r = b.conv(src, c5r, 1, name=f"m{name}_5x5r")
    b.conv(r, c5, 5, pads=(2, 2, 2, 2), dst=cat, c0=c1 + c3, name=f"m{name}_5x5")
    p = b.pool(src, 3, 1, pads=(1, 1, 1, 1), name=f"m{name}_pool")
    b.conv(p, cp, 1, dst=cat, c0=c1 + c3 + c5, name=f"m{name}_pproj")
    return cat


def googlenet(batch=128) -> Net:
    """GoogLeNet-style: 9 inception modules at 28/14/7 from a 28x28x192 input, 3x3/2 SAME stage pools."""
    b = _Builder("googlenet_b%d" % batch, "bf16", 0.01, False, (batch, 28, 28, 192))
    t = "x"
    for m in GOOGLENET_MODULES:
        if m[0] in ("4a", "5a"):
            t = b.pool(t, 3, 2, pads="SAME", name="pool_" + m[0])
        t = _inception_v1(b, t, m)
    return b.done(t)


# ----------------------------------------------------------------------------- C5
def _block_35(b, src, pool_proj, tag):
    n, h, w, _ = b.net.tensors[src]
    cat = b.concat_buffer(src, (h, w), 64 + 64 + 96 + pool_proj)
    b.conv(src, 64, 1, dst=cat, c0=0, name=f"{tag}_1x1")
    r = b.conv(src, 48, 1, name=f"{tag}_5x5r")
    b.conv(r, 64, 5, pads=(2, 2, 2, 2), dst=cat, c0=64, name=f"{tag}_5x5")
    r = b.conv(src, 64, 1, name=f"{tag}_dblr")
    r = b.conv(r, 96, 3, pads=(1, 1, 1, 1), name=f"{tag}_dbl1")
    b.conv(r, 96, 3, pads=(1, 1, 1, 1), dst=cat, c0=128, name=f"{tag}_dbl2")
    p = b.pool(src, 3, 1, pads=(1, 1, 1, 1), name=f"{tag}_pool")
    b.conv(p, pool_proj, 1, dst=cat, c0=224, name=f"{tag}_pproj")
    return cat


def _reduction_17(b, src, tag):
    n, h, w, cin = b.net.tensors[src]
    oh = out_len(h, 3, 2, 0, 0)
    cat = b.concat_buffer(src, (oh, oh), 384 + 96 + cin)
    b.conv(src, 384, 3, s=2, dst=cat, c0=0, name=f"{tag}_3x3")
    r = b.conv(src, 64, 1, name=f"{tag}_dblr")
    r = b.conv(r, 96, 3, pads=(1, 1, 1, 1), name=f"{tag}_dbl1")
    b.conv(r, 96, 3, s=2, dst=cat, c0=384, name=f"{tag}_dbl2")
    b.pool(src, 3, 2, dst=cat, c0=480, name=f"{tag}_pool")
    return cat


def _block_17(b, src, c7, tag):
    n, h, w, _ = b.net.tensors[src]
    cat = b.concat_buffer(src, (h, w), 768)
    p17 = (0, 0, 3, 3)    # 1x7: pad along width
    p71 = (3, 3, 0, 0)    # 7x1: pad along height
    b.conv(src, 192, 1, dst=cat, c0=0, name=f"{tag}_1x1")
    r = b.conv(src, c7, 1, name=f"{tag}_7r")
    r = b.conv(r, c7, 1, 7, pads=p17, name=f"{tag}_7a")
    b.conv(r, 192, 7, 1, pads=p71, dst=cat, c0=192, name=f"{tag}_7b")
    r = b.conv(src, c7, 1, name=f"{tag}_d7r")
    r = b.conv(r, c7, 7, 1, pads=p71, name=f"{tag}_d7a")
    r = b.conv(r, c7, 1, 7, pads=p17, name=f"{tag}_d7b")
    r = b.conv(r, c7, 7, 1, pads=p71, name=f"{tag}_d7c")
    b.conv(r, 192, 1, 7, pads=p17, dst=cat, c0=384, name=f"{tag}_d7d")
    p = b.pool(src, 3, 1, pads=(1, 1, 1, 1), name=f"{tag}_pool")
    b.conv(p, 192, 1, dst=cat, c0=576, name=f"{tag}_pproj")
    return cat


def _reduction_8(b, src, tag):
    n, h, w, cin = b.net.tensors[src]
    oh = out_len(h, 3, 2, 0, 0)
    cat = b.concat_buffer(src, (oh, oh), 320 + 192 + cin)
    r = b.conv(src, 192, 1, name=f"{tag}_3r")
    b.conv(r, 320, 3, s=2, dst=cat, c0=0, name=f"{tag}_3x3")
    r = b.conv(src, 192, 1, name=f"{tag}_7r")
    r = b.conv(r, 192, 1, 7, pads=(0, 0, 3, 3), name=f"{tag}_7a")
    r = b.conv(r, 192, 7, 1, pads=(3, 3, 0, 0), name=f"{tag}_7b")
    b.conv(r, 192, 3, s=2, dst=cat, c0=320, name=f"{tag}_7c")
    b.pool(src, 3, 2, dst=cat, c0=512, name=f"{tag}_pool")
    return cat


def _block_8(b, src, tag):
    n, h, w, _ = b.net.tensors[src]
    cat = b.concat_buffer(src, (h, w), 2048)
    b.conv(src, 320, 1, dst=cat, c0=0, name=f"{tag}_1x1")
    r = b.conv(src, 384, 1, name=f"{tag}_3r")
    b.conv(r, 384, 1, 3, pads=(0, 0, 1, 1), dst=cat, c0=320, name=f"{tag}_3a")
    b.conv(r, 384, 3, 1, pads=(1, 1, 0, 0), dst=cat, c0=704, name=f"{tag}_3b")
    r = b.conv(src, 448, 1, name=f"{tag}_d3r")
    r = b.conv(r, 384, 3, pads=(1, 1, 1, 1), name=f"{tag}_d3")
    b.conv(r, 384, 1, 3, pads=(0, 0, 1, 1), dst=cat, c0=1088, name=f"{tag}_d3a")
    b.conv(r, 384, 3, 1, pads=(1, 1, 0, 0), dst=cat, c0=1472, name=f"{tag}_d3b")
    p = b.pool(src, 3, 1, pads=(1, 1, 1, 1), name=f"{tag}_pool")
    b.conv(p, 192, 1, dst=cat, c0=1856, name=f"{tag}_pproj")
    return cat


def inception_v3(batch=32) -> Net:
    """Inception-v3-shaped replica step at 299x299x3, bf16, lr 0.045 (average pools become 3x3/1 max pools)."""
    b = _Builder("inception_v3_b%d" % batch, "bf16", 0.045, False, (batch, 299, 299, 3))
    t = b.conv("x", 32, 3, s=2, name="stem1")
    t = b.conv(t, 32, 3, name="stem2")
    t = b.conv(t, 64, 3, pads=(1, 1, 1, 1), name="stem3")
    t = b.pool(t, 3, 2, name="stem_pool1")
    t = b.conv(t, 80, 1, name="stem4")
    t = b.conv(t, 192, 3, name="stem5")
    t = b.pool(t, 3, 2, name="stem_pool2")
    for i, pp in enumerate((32, 64, 64)):
        t = _block_35(b, t, pp, "a%d" % i)
    t = _reduction_17(b, t, "r17")
    for i, c7 in enumerate((128, 160, 160, 192)):
        t = _block_17(b, t, c7, "c%d" % i)
    t = _reduction_8(b, t, "r8")
    for i in range(2):
        t = _block_8(b, t, "e%d" % i)
    return b.done(t)


WORKLOADS = {
    "single_layer": single_layer,
    "alexnet": alexnet,
    "vgg16": vgg16,
    "googlenet": googlenet,
    "inception_v3": inception_v3,
}


def conv_flops(net: Net) -> float:
    """Direct-convolution FLOPs of one step: 2*N*OH*OW*KH*KW*Cin*Cout per direction.

    Three directions per conv, except that dX of a conv reading the step input
    is skipped unless ``net.input_grad``.
    """
    tot = 0.0
    for c in net.convs:
        n, oh, ow, _ = net.tensors[c.dst]
        cin = net.tensors[c.src][3]
        f = 2.0 * n * oh * ow * c.kh * c.kw * cin * c.cout
        dirs = 2 if (c.src == "x" and not net.input_grad) else 3
        tot += f * dirs
    return tot


# ----------------------------------------------------------------------------- inputs
@dataclass
class Inputs:
    x: np.ndarray                 # float64 NHWC
    weights: Dict[str, np.ndarray]  # conv name -> float64 HWIO
    biases: Dict[str, np.ndarray]   # conv name -> float64 zeros [Cout]
    g: np.ndarray                 # float64 upstream gradient, shape of the output tensor (surrogate loss)
    labels: np.ndarray | None = None  # int32 class per image (softmax cross-entropy; g is then None)


def make_inputs(net: Net, seed: int = 0, batch_slice: int | None = None) -> Inputs:
    """Seeded inputs in the fixed draw order: x, then filters in op order, then g (or, for a
    softmax classifier, one uniform class label per image).

    ``batch_slice`` keeps only the first images of x and g (the filters are
    drawn from the same stream in the same order, so they are identical).
    """
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(net.tensors["x"])
    weights, biases = {}, {}
    for c in net.convs:
        cin = net.tensors[c.src][3]
        std = math.sqrt(2.0 / (c.kh * c.kw * cin))
        weights[c.name] = rng.standard_normal((c.kh, c.kw, cin, c.cout)) * std
        biases[c.name] = np.zeros(c.cout)
    if net.loss == "softmax_xent":
        g = None
        labels = rng.integers(0, net.classes, size=net.tensors["x"][0]).astype(np.int32)
    else:
        g = rng.standard_normal(net.tensors[net.output])
        labels = None
    if batch_slice is not None:
        x = x[:batch_slice].copy()
        g = None if g is None else g[:batch_slice].copy()
        labels = None if labels is None else labels[:batch_slice].copy()
    return Inputs(x, weights, biases, g, labels)


def with_batch(net_fn, batch):
    """The same workload at another batch size (used for bounded CPU samples)."""
    return net_fn(batch=batch)


# ----------------------------------------------------------------------------- sampled softmax inputs
def log_uniform_sample(rng, vocab: int, m: int):
    """m distinct classes from the log-uniform proposal Q(c) = log((c + 2) / (c + 1)) / log(vocab + 1),
    drawn (inverse CDF) until m distinct ones appear.  Returns (sampled ids int32, the log of each
    class's expected count among those draws, as a function of an id array).  These are the
    random numbers of the method, drawn on the host and handed to both implementations."""
    out, seen, draws = [], set(), 0
    while len(out) < m:
        c = np.minimum((np.exp(rng.random(2 * m) * math.log(vocab + 1.0)) - 1.0).astype(np.int64), vocab - 1)
        for x in c:
            draws += 1
            if x not in seen:
                seen.add(int(x))
                out.append(int(x))
                if len(out) == m:
                    break

    def log_expected(ids):
        q = np.log((np.asarray(ids, np.float64) + 2.0) / (np.asarray(ids, np.float64) + 1.0)) / math.log(vocab + 1.0)
        return np.log(-np.expm1(draws * np.log1p(-q)))
    return np.asarray(out, np.int32), log_expected


@dataclass
class SampledInputs:
    h: np.ndarray               # n x d classifier input
    W: np.ndarray               # vocab x d weights
    b: np.ndarray               # vocab biases
    labels: np.ndarray          # n int32
    sampled: np.ndarray         # m int32, distinct
    lq_true: np.ndarray         # n: log expected count of each row's true class
    lq_sampled: np.ndarray      # m


def make_sampled_inputs(n: int, d: int, vocab: int, m: int, seed: int = 0) -> SampledInputs:
    """Seeded sampled-softmax inputs: h ~ N(0, 1), W ~ N(0, 1/d), b ~ N(0, 0.1^2), labels from the
    same log-uniform law (word frequencies of a language model are Zipfian), then the sample."""
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((n, d))
    W = rng.standard_normal((vocab, d)) / math.sqrt(d)
    b = rng.standard_normal(vocab) * 0.1
    labels = np.minimum((np.exp(rng.random(n) * math.log(vocab + 1.0)) - 1.0).astype(np.int64), vocab - 1)
    sampled, log_expected = log_uniform_sample(rng, vocab, m)
    return SampledInputs(h, W, b, labels.astype(np.int32), sampled, log_expected(labels), log_expected(sampled))
