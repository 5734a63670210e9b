"""Parity harness between the HIP path and the CPU oracle (GPU tests only).

Error metrics (fixed for every floating-point comparison; ``r`` is the fp64
oracle result, ``a`` the GPU result):

    rel_l2(a, r) = ||a - r||_2 / ||r||_2          relative error normalised by
                                                  the tensor's L2 norm
    err(a, r)    = max_i |a_i - r_i| / RMS(r)     worst element in units of
                                                  the reference's RMS
    ulp(a, r)    = max_i |a_i - r_i| / (2^-7 |r_i| + 1e-3 RMS(r))

Gates:
* outputs stored in fp32 by an fp32 path: err <= 1e-4 (this also bounds
  rel_l2 by 1e-4);
* outputs stored in fp32 by a bf16-input path (filter and bias gradients):
  err <= 2e-2;
* outputs stored in bf16: rel_l2 <= 2e-2 and ulp <= 1, i.e. every element is
  within one bf16 ulp of the exact value (round-to-nearest on store costs half
  an ulp; a different fp32 summation order can move a value across a rounding
  midpoint), plus a slack of 1e-3 RMS for cancellation.  A max-over-RMS gate
  would count the storage rounding itself as error: on a sparse or
  heavy-tailed tensor half a bf16 ulp of its largest element alone exceeds
  2e-2 RMS.
Argmax indices and max-pool values must match exactly.  SGD results must be
within 1 ulp of the fp32 rounding of the fp64 oracle.

Comparisons are teacher-forced: the oracle receives the exact values the GPU
op consumed (bf16 widened to fp64), so kernel error is isolated from the
compounding of bf16 storage across layers.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle

BAR = {torch.float32: 1e-4, torch.bfloat16: 2e-2}


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


def err(a, r) -> float:
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if r.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(r * r)))
    d = float(np.max(np.abs(a - r)))
    return d / rms if rms > 0 else d


def rel_l2(a, r) -> float:
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    nr = float(np.linalg.norm(r.ravel()))
    d = float(np.linalg.norm((a - r).ravel()))
    return d / nr if nr > 0 else d


def ulp_bf16(a, r) -> float:
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if r.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(r * r)))
    tol = 2.0 ** -7 * np.abs(r) + 1e-3 * rms
    tol = np.where(tol > 0, tol, 1e-30)
    return float(np.max(np.abs(a - r) / tol))


def compare(a, r, storage, path=None):
    """Gate of one output tensor; returns (ok, metrics)."""
    path = storage if path is None else path
    m = {"err": err(a, r), "rel_l2": rel_l2(a, r)}
    if storage == torch.bfloat16:
        m["ulp"] = ulp_bf16(a, r)
        ok = m["rel_l2"] <= 2e-2 and m["ulp"] <= 1.0
    else:
        ok = m["err"] <= BAR[path]
    return ok, m


def assert_close(a, r, storage, path=None, label=""):
    ok, m = compare(a, r, storage, path)
    say("  %-28s %s" % (label, " ".join("%s=%.2e" % kv for kv in m.items())))
    assert ok, (label, m)


def ulp_diff_f32(a: np.ndarray, r64: np.ndarray) -> int:
    """Max distance in fp32 ulps between fp32 array a and fp32(r64)."""
    a = np.ascontiguousarray(a, dtype=np.float32).view(np.int32).astype(np.int64)
    b = np.ascontiguousarray(r64.astype(np.float32)).view(np.int32).astype(np.int64)
    a = np.where(a < 0, -(a & 0x7fffffff), a)
    b = np.where(b < 0, -(b & 0x7fffffff), b)
    return int(np.max(np.abs(a - b))) if a.size else 0


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


class ParityTracer:
    """Step-driver hook: snapshots each op's inputs, then checks its outputs.

    ``sample_images``: None checks whole tensors; a list of image indices checks
    only those images (outputs of every op but the filter/bias gradients depend
    on one image each) and evaluates ``filter_samples`` filter-gradient entries
    through the oracle's sampled entry point.
    """

    def __init__(self, dtype, sample_images=None, filter_samples=256, seed=0, label=""):
        self.dtype = dtype
        self.bar = BAR[dtype]
        self.sample = sample_images
        self.filter_samples = filter_samples
        self.rng = np.random.default_rng(seed)
        self.pending = None
        self.results = []           # (kind, op name, metric, value, bar, ok)
        self.label = label

    # -------------------------------------------------------------- helpers
    def _imgs(self, a: np.ndarray) -> np.ndarray:
        return a if self.sample is None else a[self.sample]

    def _x64(self, t: torch.Tensor) -> np.ndarray:
        if self.sample is None:
            return f64(t)
        idx = torch.tensor(self.sample, device=t.device)
        return f64(t.index_select(0, idx))

    def _index_shift(self, x_shape):
        """Argmax indices of image sample[j] in the full batch minus those of image j of the slice."""
        n, h, w, c = x_shape
        j = np.arange(len(self.sample))
        return ((np.asarray(self.sample) - j) * (h * w * c))[:, None, None, None]

    def record(self, kind, name, metric, value, bar):
        ok = value <= bar
        self.results.append((kind, name, metric, value, bar, ok))

    def record_tensor(self, kind, name, a, r, storage, path=None):
        path = self.dtype if path is None else path
        ok, m = compare(a, r, storage, path)
        if storage == torch.bfloat16:
            self.record(kind, name, "rel_l2", m["rel_l2"], 2e-2)
            self.record(kind, name, "ulp", m["ulp"], 1.0)
            self.results.append((kind, name, "err(info)", m["err"], float("inf"), True))
        else:
            self.record(kind, name, "err", m["err"], BAR[path])

    def failures(self):
        return [r for r in self.results if not r[5]]

    def summary(self):
        worst = {}
        for kind, name, metric, value, bar, ok in self.results:
            key = (kind, metric)
            score = value / bar if bar > 0 else value
            if key not in worst or score > worst[key][3]:
                worst[key] = (value, bar, name, score)
        return worst

    # -------------------------------------------------------------- hook
    def __call__(self, event, op, **t):
        if not event.endswith(":end"):
            snap = {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in t.items()}
            self.pending = (event, op, snap)
            return
        kind, op0, inp = self.pending
        assert kind == event[:-4] and op0 is op
        torch.cuda.synchronize()
        getattr(self, "_check_" + kind)(op, inp, t)
        self.pending = None

    # -------------------------------------------------------------- checks
    def _check_conv_fwd(self, op, inp, out):
        ref = oracle.conv2d_fwd(self._x64(inp["x"]), f64(inp["w"]), (op.sh, op.sw), op.pads)
        self.record_tensor("conv_fwd", op.name, self._x64(out["y"]), ref, self.dtype)

    def _check_conv_bias_relu_fwd(self, op, inp, out):
        pre = oracle.conv2d_fwd(self._x64(inp["x"]), f64(inp["w"]), (op.sh, op.sw), op.pads)
        ref = oracle.bias_relu_fwd(pre, f64(inp["b"]))
        y = self._x64(out["y"])
        self.record_tensor("conv_bias_relu_fwd", op.name, y, ref, self.dtype)
        self.record("conv_bias_relu_fwd", op.name, "negatives", float(np.sum(np.signbit(y))), 0.0)

    def _check_bias_relu_fwd(self, op, inp, out):
        ref = oracle.bias_relu_fwd(self._x64(inp["y"]), f64(inp["b"]))
        y = self._x64(out["y"])
        self.record_tensor("bias_relu_fwd", op.name, y, ref, self.dtype)
        self.record("bias_relu_fwd", op.name, "negatives", float(np.sum(np.signbit(y))), 0.0)

    @staticmethod
    def _dense(argmax, x_shape, op):
        """A pool's selection as dense NHWC indices into its input: int32 argmax as stored, uint8
        window taps kh * KW + kw decoded."""
        a = argmax.cpu().numpy().astype(np.int64)
        if argmax.dtype != torch.uint8:
            return a
        N, H, W, C = x_shape
        n, oh, ow, c = np.indices(a.shape)
        h = oh * op.sh - op.pads[0] + a // op.kw
        w = ow * op.sw - op.pads[2] + a % op.kw
        return ((n * H + h) * W + w) * C + c

    def _check_maxpool_fwd(self, op, inp, out):
        x = self._x64(inp["x"])
        ref, am = oracle.maxpool_fwd(x, (op.kh, op.kw), (op.sh, op.sw), op.pads)
        got_am = self._dense(out["argmax"], inp["x"].shape, op)
        if self.sample is not None:
            got_am = got_am[self.sample] - self._index_shift(inp["x"].shape)
        self.record("maxpool_fwd", op.name, "err", err(self._x64(out["y"]), ref), 0.0)
        self.record("maxpool_fwd", op.name, "argmax_mismatch", float(np.sum(got_am != am)), 0.0)

    def _check_bias_relu_bwd(self, op, inp, out):
        y, dy = f64(inp["y"]), f64(inp["dy"])
        ref_dpre, ref_db = oracle.bias_relu_bwd(y, dy)
        self.record("bias_relu_bwd", op.name, "dpre_mismatch", float(np.sum(f64(out["dpre"]) != ref_dpre)), 0.0)
        self.record_tensor("bias_relu_bwd:db", op.name, f64(out["db"]), ref_db, torch.float32)

    def _check_conv_bwd_filter(self, op, inp, out):
        dw = f64(out["dw"])
        if self.sample is None:
            ref = oracle.conv2d_bwd_filter(f64(inp["x"]), f64(inp["dy"]), (op.kh, op.kw), (op.sh, op.sw), op.pads)
            self.record_tensor("conv_bwd_filter", op.name, dw, ref, torch.float32)
        else:
            idx = self.rng.integers(0, dw.size, size=min(self.filter_samples, dw.size))
            ref = oracle.conv2d_bwd_filter_at(f64(inp["x"]), f64(inp["dy"]), (op.kh, op.kw), (op.sh, op.sw),
                                              op.pads, idx)
            self.record_tensor("conv_bwd_filter:sampled", op.name, dw.ravel()[idx], ref, torch.float32)

    def _check_conv_bwd_input(self, op, inp, out):
        dy = self._x64(inp["dy"])
        dx_old = self._x64(inp["dx"])
        ref = oracle.conv2d_bwd_input(dy, f64(inp["w"]), dx_old.shape, (op.sh, op.sw), op.pads,
                                      dx=dx_old, beta=inp["beta"])
        self.record_tensor("conv_bwd_input", op.name, self._x64(out["dx"]), ref, self.dtype)

    def _check_conv_bwd_input_relu_bwd(self, op, inp, out):
        # the input gradient of op fused with the ReLU backward of the layer that produced its input
        dy, y = self._x64(inp["dy"]), self._x64(inp["y"])
        g = oracle.conv2d_bwd_input(dy, f64(inp["w"]), y.shape, (op.sh, op.sw), op.pads)
        ref_dpre, ref_db = oracle.bias_relu_bwd(y, g)
        self.record_tensor("conv_bwd_input_relu_bwd", op.name, self._x64(out["dpre"]), ref_dpre, self.dtype)
        if self.sample is None:              # (the bias gradient sums over every image)
            self.record_tensor("conv_bwd_input_relu_bwd:db", op.name, f64(out["db"]), ref_db, torch.float32)

    def _check_maxpool_bwd(self, op, inp, out):
        dy = self._x64(inp["dy"])
        am = self._dense(inp["argmax"], inp["dx"].shape, op)
        dx_old = self._x64(inp["dx"])
        if self.sample is not None:
            am = am[self.sample] - self._index_shift(inp["dx"].shape)
        ref = oracle.maxpool_bwd(dy, am.astype(np.int32), dx_old.shape, dx=dx_old, beta=inp["beta"])
        self.record_tensor("maxpool_bwd", op.name, self._x64(out["dx"]), ref, self.dtype)

    def _check_maxpool_relu_bwd(self, op, inp, out):
        # whole tensors: the bias gradient sums over every image
        y = f64(inp["y"])
        am = self._dense(inp["argmax"], inp["y"].shape, op).astype(np.int32)
        dpre_old = f64(inp["dpre"])
        g = oracle.maxpool_bwd(f64(inp["dy"]), am, y.shape, dx=dpre_old, beta=inp["beta"])
        ref_dpre, ref_db = oracle.bias_relu_bwd(y, g)
        self.record_tensor("maxpool_relu_bwd", op.name, f64(out["dpre"]), ref_dpre, self.dtype)
        self.record_tensor("maxpool_relu_bwd:db", op.name, f64(out["db"]), ref_db, torch.float32)

    def _check_apply_sgd(self, op, inp, out):
        var, grad = inp["var"].cpu().numpy(), inp["grad"].cpu().numpy()
        ref = oracle.apply_sgd(var.astype(np.float64), grad.astype(np.float64), self.lr)
        self.record("apply_sgd", "all", "ulp", float(ulp_diff_f32(out["var"].cpu().numpy(), ref)), 1.0)

    lr = 0.01
