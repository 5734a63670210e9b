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

Whole-step comparisons are oracle-forced: the oracle runs the step op by op on
the seeded inputs, and before each GPU op the harness overwrites that op's
input buffers with the oracle's values, rounded to the buffer's storage type;
the oracle op then runs on the same rounded values.  Values flow only from the
oracle to the GPU, never back, and each kernel's error is isolated from the
compounding of bf16 storage across layers.
"""
from __future__ import annotations

import sys
import time

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
    """Step-driver hook that forces every op's inputs from the oracle and checks its outputs.

    ``rep`` is the Replica being stepped and ``inputs`` its seeded inputs.  With ``distinct``
    set, the oracle runs on the first ``distinct`` images only and every input buffer holds
    those images repeated along the batch (the batch must be a multiple): the GPU runs the
    full-size step in its own launch configuration, per-image outputs are checked on the
    distinct images (and must repeat bit for bit), and batch sums (filter and bias
    gradients) are the oracle's sums times the repeat count.
    """

    def __init__(self, rep, inputs, distinct=None, label=""):
        self.rep = rep
        self.dtype = rep.dtype
        self.bar = BAR[rep.dtype]
        n = inputs.x.shape[0]
        self.k = n if distinct is None else distinct
        assert n % self.k == 0
        self.tile = n // self.k
        self.label = label
        self.lr = rep.lr
        self.pending = None
        self._t0 = time.perf_counter()
        self.results = []           # (kind, op name, metric, value, bar, ok)
        net, k = rep.net, self.k
        self.state = {("act", "x"): np.asarray(inputs.x[:k], np.float64)}
        if inputs.g is not None:
            self.state[("grad", net.output)] = np.asarray(inputs.g[:k], np.float64)
        self.labels = None if inputs.labels is None else np.asarray(inputs.labels[:k], np.int32)
        for c in net.convs:
            self.state[("W", c.name)] = np.asarray(inputs.weights[c.name], np.float64)
            self.state[("b", c.name)] = np.asarray(inputs.biases[c.name], np.float64)
        # merged 1x1 groups: their filters side by side, as the replica holds them
        self.member_of = {}
        for g in getattr(rep, "merges", []):
            name = g["op"].name
            self.state[("W", name)] = np.concatenate([self.state[("W", m.name)] for m in g["members"]], axis=3)
            a = 0
            for m in g["members"]:
                self.member_of[m.name] = (name, a)
                a += m.cout
        # every buffer an op reads or writes, under the oracle state key that mirrors it;
        # NHWC batch buffers may be viewed as channel slices, the variables only whole
        self.batched = [(("act", nm), t) for nm, t in rep.act.items()]
        self.batched += [(("grad", nm), t) for nm, t in rep.grad.items()]
        self.batched += [(("dpre_out",), rep.dpre_out)]
        self.whole = [(("W", nm), t) for nm, t in rep.Wlp.items()]
        self.whole += [(("b", nm), t) for nm, t in rep.b.items()]
        self.whole += [(("dW", nm), t) for nm, t in rep.dW.items()]
        self.whole += [(("db", nm), t) for nm, t in rep.db.items()]
        self.whole += [(("W", nm), t) for nm, t in getattr(rep, "mWlp", {}).items()]
        self.whole += [(("dW", nm), t) for nm, t in getattr(rep, "mdW", {}).items()]

    # -------------------------------------------------------------- buffers
    def _lookup(self, t):
        """(state key, first channel, buffer shape) of the buffer t views: a channel slice of an
        NHWC batch buffer, or a whole variable (first channel None)."""
        p, es = t.data_ptr(), t.element_size()
        for key, b in self.whole:
            if b.dtype == t.dtype and p == b.data_ptr() and tuple(t.shape) == tuple(b.shape):
                return key, None, tuple(b.shape)
        for key, b in self.batched:
            off = p - b.data_ptr()
            if b.dtype != t.dtype or t.dim() != 4 or off < 0 or off % es:
                continue
            c0 = off // es
            if (tuple(t.shape[:3]) == tuple(b.shape[:3]) and c0 + t.shape[3] <= b.shape[3]
                    and t.stride() == b.stride()):
                return key, c0, tuple(b.shape)
        raise KeyError("tensor at %#x %s is none of the replica's buffers" % (p, tuple(t.shape)))

    def _chan_spans(self, t):
        """A 4-D view whose channels are several batch buffers side by side in one allocation (a
        merged group's outputs or gradients): [(key, first channel in the buffer, first channel
        in t, width)] covering t's channels in order, or None."""
        if t.dim() != 4:
            return None
        es, p, width = t.element_size(), t.data_ptr(), t.shape[3]
        parts = []
        for key, b in self.batched:
            if (b.dtype != t.dtype or b.dim() != 4 or tuple(b.shape[:3]) != tuple(t.shape[:3])
                    or b.stride() != t.stride()):
                continue
            d = (b.data_ptr() - p) // es                 # b's channel 0 in t's channel numbering
            if (b.data_ptr() - p) % es or d >= width or d + b.shape[3] <= 0:
                continue
            lo, hi = max(0, d), min(width, d + b.shape[3])
            parts.append((lo, key, lo - d, hi - lo))
        parts.sort(key=lambda e: e[0])
        at = 0
        for lo, _, _, w in parts:
            if lo != at:
                return None
            at += w
        return [(key, bc0, lo, w) for lo, key, bc0, w in parts] if at == width and len(parts) > 1 else None

    def _get(self, t):
        spans = self._chan_spans(t)
        if spans is not None:
            return np.concatenate([self.state[key][..., bc0:bc0 + w] for key, bc0, _, w in spans], axis=3)
        vspans = self._spans(t)
        if vspans is not None:                           # (a merged group's biases side by side)
            return np.concatenate([np.asarray(self.state[key], np.float64).reshape(-1) for key, _, _ in vspans])
        key, c0, _ = self._lookup(t)
        v = self.state[key]
        return v if c0 is None else v[..., c0:c0 + t.shape[3]]

    def _spans(self, t):
        """The whole variables a 1-D slice covers exactly, side by side (the bias gradients of a
        group of concat branches): [(key, first element of t, length)], or None."""
        if t.dim() != 1:
            return None
        p, es, n = t.data_ptr(), t.element_size(), t.numel()
        parts = sorted(((b.data_ptr() - p) // es, key, b.numel()) for key, b in self.whole
                       if b.dtype == t.dtype and b.dim() == 1 and p <= b.data_ptr() < p + n * es)
        at = 0
        for off, _, m in parts:
            if off != at:
                return None
            at += m
        return [(key, off, m) for off, key, m in parts] if at == n and len(parts) > 1 else None

    def _set(self, t, v):
        spans = self._spans(t)
        if spans is not None:
            for key, off, m in spans:
                self.state[key] = np.array(v[off:off + m], np.float64)
            return
        cspans = self._chan_spans(t)
        if cspans is not None:
            for key, bc0, tc0, w in cspans:
                if key not in self.state:
                    shape = next(tuple(b.shape) for k, b in self.batched if k == key)
                    self.state[key] = np.zeros((self.k,) + shape[1:])
                self.state[key][..., bc0:bc0 + w] = v[..., tc0:tc0 + w]
            return
        key, c0, shape = self._lookup(t)
        if c0 is None:
            self.state[key] = np.array(v, np.float64)
            return
        if key not in self.state:
            self.state[key] = np.zeros((self.k,) + shape[1:])
        self.state[key][..., c0:c0 + t.shape[3]] = v

    def _round(self, v, dtype):
        return torch.from_numpy(np.ascontiguousarray(v)).to(dtype)

    def _write(self, t, r, batched):
        """Copy host tensor r into t; a batch tensor of k images is repeated along the batch."""
        if batched and self.tile > 1:
            r = r.repeat(self.tile, 1, 1, 1)
        t.copy_(r.to(t.device))

    def _force(self, t):
        """Overwrite t with the oracle's value of its buffer rounded to t's type; returns the
        rounded value (k images for a batch tensor) in fp64."""
        r = self._round(self._get(t), t.dtype)
        if self._chan_spans(t) is not None:
            batched = True
        elif self._spans(t) is not None:
            batched = False
        else:
            batched = self._lookup(t)[1] is not None
        self._write(t, r, batched)
        return r.to(torch.float64).numpy()

    def _force_argmax(self, t, op, x_shape):
        """Overwrite a pool's selection buffer with the oracle's (dense indices into the k-image
        input), in the buffer's format: uint8 window taps or int32 dense indices."""
        dense = self.state[("argmax", op.name)].astype(np.int64)
        _, H, W, C = x_shape
        if t.dtype == torch.uint8:
            n, oh, ow, c = np.indices(dense.shape)
            h = dense // (W * C) % H
            w = dense // C % W
            taps = (h - (oh * op.sh - op.pads[0])) * op.kw + (w - (ow * op.sw - op.pads[2]))
            assert np.all((taps >= 0) & (taps < op.kh * op.kw))
            self._write(t, torch.from_numpy(taps.astype(np.uint8)), True)
        else:
            full = np.concatenate([dense + r * self.k * H * W * C for r in range(self.tile)])
            t.copy_(torch.from_numpy(full.astype(np.int32)).to(t.device))
        return dense

    def _got(self, kind, name, t):
        """GPU output of the k distinct images in fp64; with repeated images, checks that every
        repeat of an image's output equals the first bit for bit."""
        if t.dim() == 4 and self.tile > 1:
            first = t[:self.k]
            bad = sum(int((t[r * self.k:(r + 1) * self.k] != first).sum()) for r in range(1, self.tile))
            self.record(kind, name, "repeat_mismatch", float(bad), 0.0)
            t = first
        return f64(t)

    # -------------------------------------------------------------- results
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

    # -------------------------------------------------------------- hook
    def __call__(self, event, op, stream=None, **t):
        torch.cuda.synchronize()
        if not event.endswith(":end"):
            used = getattr(self, "_force_" + event)(op, t)
            torch.cuda.synchronize()
            self.pending = (event, op, used)
            return
        kind, op0, used = self.pending
        assert kind == event[:-4] and op0 is op
        getattr(self, "_check_" + kind)(op, used, t)
        self.pending = None
        now = time.perf_counter()
        say("    %-28s %-20s checked (%.1f s)" % (kind, op.name if op is not None else "all", now - self._t0))
        self._t0 = now

    # -------------------------------------------------------------- forward
    def _force_conv_bias_relu_fwd(self, op, t):
        return {"x": self._force(t["x"]), "w": self._force(t["w"]), "b": self._force(t["b"])}

    def _check_conv_bias_relu_fwd(self, op, u, out):
        pre = oracle.conv2d_fwd(u["x"], u["w"], (op.sh, op.sw), op.pads)
        ref = oracle.bias_relu_fwd(pre, u["b"])
        y = self._got("conv_bias_relu_fwd", op.name, out["y"])
        self.record_tensor("conv_bias_relu_fwd", op.name, y, ref, self.dtype)
        self.record("conv_bias_relu_fwd", op.name, "negatives", float(np.sum(np.signbit(y))), 0.0)
        self._set(out["y"], ref)

    def _force_conv_bias_relu_maxpool_fwd(self, op, t):
        return {"x": self._force(t["x"]), "w": self._force(t["w"]), "b": self._force(t["b"])}

    def _check_conv_bias_relu_maxpool_fwd(self, op, u, out):
        pool = self.rep.conv_pool[op.name]
        ref = oracle.bias_relu_fwd(oracle.conv2d_fwd(u["x"], u["w"], (op.sh, op.sw), op.pads), u["b"])
        y = self._got("conv_bias_relu_maxpool_fwd", op.name, out["y"])
        self.record_tensor("conv_bias_relu_maxpool_fwd", op.name, y, ref, self.dtype)
        self.record("conv_bias_relu_maxpool_fwd", op.name, "negatives", float(np.sum(np.signbit(y))), 0.0)
        self._set(out["y"], ref)
        yr = self._round(ref, self.dtype).to(torch.float64).numpy()
        pref, am = oracle.maxpool_fwd(yr, (pool.kh, pool.kw), (pool.sh, pool.sw), pool.pads)
        py = self._got("conv_bias_relu_maxpool_fwd:py", pool.name, out["py"])
        got_am = self._dense(out["argmax"][:self.k], yr.shape, pool)
        if out["argmax"].dtype == torch.uint8:
            self._got("conv_bias_relu_maxpool_fwd:argmax", pool.name, out["argmax"])
        self._check_fused_pool(pool, yr, pref, am, py, got_am)
        self._set(out["py"], pref)
        self.state[("argmax", pool.name)] = am

    def _check_fused_pool(self, pool, yr, pref, am, py, got_am):
        """A max-pool fused after its convolution pools the convolution's own output, which is not
        forced to the oracle's: values are held to the bf16 gate, and the selected tap must be the
        oracle's wherever the window's two largest oracle values differ by more than the two can
        move under that gate (2 x (2^-7 |v| + 1e-3 RMS)); near-ties are counted, not gated."""
        kh, kw, sh, sw = pool.kh, pool.kw, pool.sh, pool.sw
        n, oh, ow, c = pref.shape
        pt, pb, pl, pr = pool.pads
        yp = np.pad(yr, ((0, 0), (pt, pb), (pl, pr), (0, 0)), constant_values=-np.inf) if any(pool.pads) else yr
        wins = np.stack([yp[:, i:i + sh * (oh - 1) + 1:sh, j:j + sw * (ow - 1) + 1:sw, :]
                         for i in range(kh) for j in range(kw)])
        wins.sort(axis=0)
        top1, top2 = wins[-1], wins[-2] if wins.shape[0] > 1 else wins[-1] - np.inf
        rms = float(np.sqrt(np.mean(yr * yr))) if yr.size else 0.0
        tie = (top1 - top2) <= 2 * (2.0 ** -7 * np.abs(top1) + 1e-3 * rms)
        mism = got_am != am
        self.record_tensor("fused_maxpool_fwd", pool.name, py, pref, self.dtype)
        self.record("fused_maxpool_fwd", pool.name, "argmax_mismatch", float(np.sum(mism & ~tie)), 0.0)
        self.results.append(("fused_maxpool_fwd", pool.name, "near_tie_mismatch(info)", float(np.sum(mism & tie)),
                             float("inf"), True))

    def _force_maxpool_fwd(self, op, t):
        return {"x": self._force(t["x"]), "x_shape": tuple(t["x"].shape)}

    def _check_maxpool_fwd(self, op, u, out):
        ref, am = oracle.maxpool_fwd(u["x"], (op.kh, op.kw), (op.sh, op.sw), op.pads)
        y = self._got("maxpool_fwd", op.name, out["y"])
        got_am = self._dense(out["argmax"][:self.k], (self.k,) + u["x_shape"][1:], op)
        self.record("maxpool_fwd", op.name, "err", err(y, ref), 0.0)
        self.record("maxpool_fwd", op.name, "argmax_mismatch", float(np.sum(got_am != am)), 0.0)
        if out["argmax"].dtype == torch.uint8:          # (dense indices differ by the image offset)
            self._got("maxpool_fwd:argmax", op.name, out["argmax"])
        self._set(out["y"], ref)
        self.state[("argmax", op.name)] = am

    def _force_conv_fwd(self, op, t):
        return {"x": self._force(t["x"]), "w": self._force(t["w"])}

    def _check_conv_fwd(self, op, u, out):
        ref = oracle.conv2d_fwd(u["x"], u["w"], (op.sh, op.sw), op.pads)
        self.record_tensor("conv_fwd", op.name, self._got("conv_fwd", op.name, out["y"]), ref, self.dtype)
        self._set(out["y"], ref)

    # -------------------------------------------------------------- loss
    def _force_softmax_xent(self, op, t):
        lab = t["labels"]
        lab.copy_(torch.from_numpy(np.tile(self.labels, self.tile)).to(lab.device))
        return {"logits": self._force(t["logits"]), "bias": self._force(t["bias"]), "n": lab.numel()}

    def _check_softmax_xent(self, op, u, out):
        z = u["logits"].reshape(self.k, -1)
        rows, dz = oracle.softmax_xent(z, self.labels, 1.0 / u["n"], bias=u["bias"])
        loss = out["loss"]
        if self.tile > 1:
            first = loss[:self.k]
            bad = sum(int((loss[r * self.k:(r + 1) * self.k] != first).sum()) for r in range(1, self.tile))
            self.record("softmax_xent", op.name, "repeat_mismatch", float(bad), 0.0)
        self.record_tensor("softmax_xent:loss", op.name, f64(loss[:self.k]), rows, torch.float32, torch.float32)
        got = self._got("softmax_xent", op.name, out["dlogits"]).reshape(self.k, -1)
        self.record_tensor("softmax_xent", op.name, got, dz, self.dtype, torch.float32)
        self._set(out["dlogits"], dz.reshape((self.k,) + tuple(out["dlogits"].shape[1:])))

    # -------------------------------------------------------------- backward
    def _force_bias_bwd(self, op, t):
        return {"dy": self._force(t["dy"])}

    def _check_bias_bwd(self, op, u, out):
        dpre = self._got("bias_bwd", op.name, out["dpre"])
        self.record("bias_bwd", op.name, "dpre_mismatch", float(np.sum(dpre != u["dy"])), 0.0)
        ref_db = u["dy"].sum(axis=(0, 1, 2)) * self.tile
        self.record_tensor("bias_bwd:db", op.name, f64(out["db"]), ref_db, torch.float32)
        self._set(out["dpre"], u["dy"])
        self._set(out["db"], ref_db)

    def _force_bias_relu_bwd(self, op, t):
        return {"y": self._force(t["y"]), "dy": self._force(t["dy"])}

    def _check_bias_relu_bwd(self, op, u, out):
        ref_dpre, ref_db = oracle.bias_relu_bwd(u["y"], u["dy"])
        dpre = self._got("bias_relu_bwd", op.name, out["dpre"])
        self.record("bias_relu_bwd", op.name, "dpre_mismatch", float(np.sum(dpre != ref_dpre)), 0.0)
        self.record_tensor("bias_relu_bwd:db", op.name, f64(out["db"]), ref_db * self.tile, torch.float32)
        self._set(out["dpre"], ref_dpre)
        self._set(out["db"], ref_db * self.tile)

    def _force_conv_bwd_filter(self, op, t):
        return {"x": self._force(t["x"]), "dy": self._force(t["dy"])}

    def _check_conv_bwd_filter(self, op, u, out):
        ref = oracle.conv2d_bwd_filter(u["x"], u["dy"], (op.kh, op.kw), (op.sh, op.sw), op.pads) * self.tile
        self.record_tensor("conv_bwd_filter", op.name, f64(out["dw"]), ref, torch.float32)
        self._set(out["dw"], ref)

    def _force_conv_bwd_input(self, op, t):
        u = {"dy": self._force(t["dy"]), "w": self._force(t["w"]), "beta": t["beta"],
             "dx_shape": (self.k,) + tuple(t["dx"].shape[1:])}
        u["dx"] = self._force(t["dx"]) if t["beta"] else None
        return u

    def _check_conv_bwd_input(self, op, u, out):
        ref = oracle.conv2d_bwd_input(u["dy"], u["w"], u["dx_shape"], (op.sh, op.sw), op.pads,
                                      dx=u["dx"], beta=u["beta"])
        self.record_tensor("conv_bwd_input", op.name, self._got("conv_bwd_input", op.name, out["dx"]), ref,
                           self.dtype)
        self._set(out["dx"], ref)

    def _force_conv_bwd_input_relu_bwd(self, op, t):
        u = {"dy": self._force(t["dy"]), "w": self._force(t["w"]), "y": self._force(t["y"]),
             "beta": t.get("beta", 0.0)}
        u["dpre"] = self._force(t["dpre"]) if u["beta"] else None
        return u

    def _check_conv_bwd_input_relu_bwd(self, op, u, out):
        # the input gradient of op (added to what the input's other readers stored, beta = 1) fused
        # with the ReLU backward of the layers that produced its input
        g = oracle.conv2d_bwd_input(u["dy"], u["w"], u["y"].shape, (op.sh, op.sw), op.pads, dx=u["dpre"],
                                    beta=u["beta"])
        ref_dpre, ref_db = oracle.bias_relu_bwd(u["y"], g)
        got = self._got("conv_bwd_input_relu_bwd", op.name, out["dpre"])
        self.record_tensor("conv_bwd_input_relu_bwd", op.name, got, ref_dpre, self.dtype)
        self.record("conv_bwd_input_relu_bwd", op.name, "masked_nonzero", float(np.sum(got[u["y"] <= 0] != 0)), 0.0)
        self.record_tensor("conv_bwd_input_relu_bwd:db", op.name, f64(out["db"]), ref_db * self.tile, torch.float32)
        self._set(out["dpre"], ref_dpre)
        self._set(out["db"], ref_db * self.tile)

    def _force_maxpool_bwd(self, op, t):
        x_shape = tuple(t["dx"].shape)
        u = {"dy": self._force(t["dy"]), "am": self._force_argmax(t["argmax"], op, x_shape), "beta": t["beta"],
             "dx_shape": (self.k,) + x_shape[1:]}
        u["dx"] = self._force(t["dx"]) if t["beta"] else None
        return u

    def _check_maxpool_bwd(self, op, u, out):
        ref = oracle.maxpool_bwd(u["dy"], u["am"].astype(np.int32), u["dx_shape"], dx=u["dx"], beta=u["beta"])
        self.record_tensor("maxpool_bwd", op.name, self._got("maxpool_bwd", op.name, out["dx"]), ref, self.dtype)
        self._set(out["dx"], ref)

    def _force_maxpool_relu_bwd(self, op, t):
        y_shape = tuple(t["y"].shape)
        u = {"dy": self._force(t["dy"]), "am": self._force_argmax(t["argmax"], op, y_shape), "y": self._force(t["y"]),
             "beta": t["beta"]}
        # the pool's output, which may stand in for y as the mask: the state the forward check left,
        # the oracle's pool of the state of y (the check below still takes the mask from y)
        if t.get("py") is not None:
            self._force(t["py"])
        u["dpre"] = self._force(t["dpre"]) if t["beta"] else None
        return u

    def _check_maxpool_relu_bwd(self, op, u, out):
        g = oracle.maxpool_bwd(u["dy"], u["am"].astype(np.int32), u["y"].shape, dx=u["dpre"], beta=u["beta"])
        ref_dpre, ref_db = oracle.bias_relu_bwd(u["y"], g)
        got = self._got("maxpool_relu_bwd", op.name, out["dpre"])
        self.record_tensor("maxpool_relu_bwd", op.name, got, ref_dpre, self.dtype)
        self.record_tensor("maxpool_relu_bwd:db", op.name, f64(out["db"]), ref_db * self.tile, torch.float32)
        self._set(out["dpre"], ref_dpre)
        self._set(out["db"], ref_db * self.tile)

    # -------------------------------------------------------------- update
    def _flat(self, kind_w, kind_b, wdtype):
        """The oracle's per-layer values laid out like the replica's flat variable buffer (fp32;
        weights first rounded to wdtype, the type the step's convolutions read them in)."""
        rep = self.rep
        flat = np.zeros(rep.n_params, np.float64)
        for c in rep.net.convs:
            wo, wshape, bo, bn = rep._layout[c.name]
            key = (kind_w, c.name)
            if key not in self.state and c.name in self.member_of:
                # (a merged group's member: its channels of the group's filter gradient)
                name, a = self.member_of[c.name]
                w = self.state[(kind_w, name)][..., a:a + c.cout]
            else:
                w = self.state[key]
            wv = self._round(w, wdtype).to(torch.float32).to(torch.float64).numpy()
            rep.place_filter(flat, c.name, wv)
            flat[bo:bo + bn] = self._round(self.state[(kind_b, c.name)], torch.float32).to(torch.float64).numpy()
        return flat

    def _force_apply_sgd(self, op, t):
        var = self._flat("W", "b", self.dtype)
        grad = self._flat("dW", "db", torch.float32)
        t["var"].copy_(torch.from_numpy(var).to(torch.float32).to(t["var"].device))
        t["grad"].copy_(torch.from_numpy(grad).to(torch.float32).to(t["grad"].device))
        return {"var": var, "grad": grad}

    def _check_apply_sgd(self, op, u, out):
        ref = oracle.apply_sgd(u["var"], u["grad"], self.lr)
        self.record("apply_sgd", "all", "ulp", float(ulp_diff_f32(out["var"].cpu().numpy(), ref)), 1.0)
        if self.rep.shadow is not None:
            same = torch.equal(self.rep.shadow, out["var"].to(torch.bfloat16))
            self.record("apply_sgd", "shadow", "mismatch", 0.0 if same else 1.0, 0.0)


class SampledParityTracer(ParityTracer):
    """Full-size, all-distinct step check for workloads whose whole-batch oracle step is too slow.

    Every buffer holds distinct images (the seeded inputs, no repetition), and every op's inputs
    are forced from the harness state before it runs, as in ParityTracer.  The state holds the
    whole batch:

    * ops whose oracle is cheap at full size (max-pool forward and backward, ReLU backward, bias
      gradients) are computed by the oracle over the whole batch and checked on every image
      (argmax and max-pool values bit-exact);
    * convolution outputs are computed by the oracle only for the images in ``sample`` and
      checked there element by element; the other images of that output are filled with seeded
      N(0, rms^2) draws (passed through max(., 0) after a ReLU), so every later op still reads
      distinct, known values and never a GPU result;
    * filter gradients are checked at ``n_entries`` seeded HWIO entries, each summed by the oracle
      over the whole batch; the rest of the filter-gradient state is filled the same way;
    * an input gradient fused with the ReLU backward is checked on the sampled images and, for
      its mask, on every image (zero wherever the forced ReLU output is not positive); its bias
      gradient sums the GPU's own input gradient of the unsampled images, which the oracle does
      not form, so it is left to the repeated-image full-size test.

    A kernel that reads another image's data (a wrong batch offset or image advance) fails the
    sampled comparisons, since no two images hold the same values.
    """

    def __init__(self, rep, inputs, sample, n_entries=256, seed=1234, label=""):
        super().__init__(rep, inputs, distinct=None, label=label)
        n = inputs.x.shape[0]
        self.sample = sorted({int(s) % n for s in sample})
        self.n_entries = n_entries
        self.rng = np.random.default_rng(seed)
        self.skipped = []

    def _gs(self, t):
        """GPU values of the sampled images of batch tensor t, fp64."""
        return f64(t[self.sample])

    def _fill(self, shape, ref, relu):
        """Whole-batch state of a convolution output: seeded draws with the RMS of the oracle's
        sampled values, the sampled images set to those values."""
        rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 1.0
        full = self.rng.standard_normal(shape, dtype=np.float32).astype(np.float64) * (rms or 1.0)
        if relu:
            np.maximum(full, 0.0, out=full)
        full[self.sample] = ref
        return full

    def _set_fill(self, t, ref, relu):
        shape = (self.k,) + tuple(t.shape[1:])
        self._set(t, self._fill(shape, ref, relu))

    # -------------------------------------------------------------- forward
    def _check_conv_bias_relu_fwd(self, op, u, out):
        s = self.sample
        ref = oracle.bias_relu_fwd(oracle.conv2d_fwd(u["x"][s], u["w"], (op.sh, op.sw), op.pads), u["b"])
        y = self._gs(out["y"])
        self.record_tensor("conv_bias_relu_fwd", op.name, y, ref, self.dtype)
        self.record("conv_bias_relu_fwd", op.name, "negatives", float(np.sum(np.signbit(y))), 0.0)
        self._set_fill(out["y"], ref, relu=True)

    def _check_conv_bias_relu_maxpool_fwd(self, op, u, out):
        s = self.sample
        pool = self.rep.conv_pool[op.name]
        ref = oracle.bias_relu_fwd(oracle.conv2d_fwd(u["x"][s], u["w"], (op.sh, op.sw), op.pads), u["b"])
        y = self._gs(out["y"])
        self.record_tensor("conv_bias_relu_maxpool_fwd", op.name, y, ref, self.dtype)
        self.record("conv_bias_relu_maxpool_fwd", op.name, "negatives", float(np.sum(np.signbit(y))), 0.0)
        yr = self._round(ref, self.dtype).to(torch.float64).numpy()
        pref, am = oracle.maxpool_fwd(yr, (pool.kh, pool.kw), (pool.sh, pool.sw), pool.pads)
        got_am = self._dense(out["argmax"][s], yr.shape, pool)
        self._check_fused_pool(pool, yr, pref, am, self._gs(out["py"]), got_am)
        self._set_fill(out["y"], ref, relu=True)
        # the whole batch's pool state: the oracle's pool of the (filled) state, as stored
        full = self._round(self.state[self._lookup(out["y"])[0]], self.dtype).to(torch.float64).numpy()
        pfull, amfull = oracle.maxpool_fwd(full, (pool.kh, pool.kw), (pool.sh, pool.sw), pool.pads)
        self._set(out["py"], pfull)
        self.state[("argmax", pool.name)] = amfull

    def _check_conv_fwd(self, op, u, out):
        s = self.sample
        ref = oracle.conv2d_fwd(u["x"][s], u["w"], (op.sh, op.sw), op.pads)
        self.record_tensor("conv_fwd", op.name, self._gs(out["y"]), ref, self.dtype)
        self._set_fill(out["y"], ref, relu=False)

    # -------------------------------------------------------------- backward
    def _check_conv_bwd_filter(self, op, u, out):
        dw = out["dw"]
        numel = dw.numel()
        idx = self.rng.choice(numel, size=min(self.n_entries, numel), replace=False)
        idx = np.unique(np.concatenate([idx, [0, numel - 1]])).astype(np.int64)
        ref = oracle.conv2d_bwd_filter_at(u["x"], u["dy"], (op.kh, op.kw), (op.sh, op.sw), op.pads, idx)
        got = dw.reshape(-1)[torch.from_numpy(idx).to(dw.device)].to(torch.float64).cpu().numpy()
        self.record_tensor("conv_bwd_filter@entries", op.name, got, ref, torch.float32)
        rms = float(np.sqrt(np.mean(ref * ref))) or 1.0
        full = self.rng.standard_normal(numel) * rms
        full[idx] = ref
        self._set(dw, full.reshape(tuple(dw.shape)))

    def _check_conv_bwd_input(self, op, u, out):
        s = self.sample
        dx0 = u["dx"][s] if u["beta"] else None
        ref = oracle.conv2d_bwd_input(u["dy"][s], u["w"], (len(s),) + u["dx_shape"][1:], (op.sh, op.sw), op.pads,
                                      dx=dx0, beta=u["beta"])
        self.record_tensor("conv_bwd_input", op.name, self._gs(out["dx"]), ref, self.dtype)
        self._set_fill(out["dx"], ref, relu=False)

    def _check_conv_bwd_input_relu_bwd(self, op, u, out):
        s = self.sample
        g = oracle.conv2d_bwd_input(u["dy"][s], u["w"], (len(s),) + u["y"].shape[1:], (op.sh, op.sw), op.pads,
                                    dx=u["dpre"][s] if u["beta"] else None, beta=u["beta"])
        ref_dpre, _ = oracle.bias_relu_bwd(u["y"][s], g)
        self.record_tensor("conv_bwd_input_relu_bwd", op.name, self._gs(out["dpre"]), ref_dpre, self.dtype)
        # the ReLU mask on every image: zero wherever the forced y is not positive
        masked = out["dpre"][torch.from_numpy(u["y"] <= 0).to(out["dpre"].device)]
        self.record("conv_bwd_input_relu_bwd", op.name, "masked_nonzero", float((masked != 0).sum()), 0.0)
        self.skipped.append(("conv_bwd_input_relu_bwd:db", op.name))
        full = self._fill((self.k,) + u["y"].shape[1:], ref_dpre, relu=False)
        full[u["y"] <= 0] = 0.0
        self._set(out["dpre"], full)
        db_ref = self.rng.standard_normal(out["db"].numel())
        self._set(out["db"], db_ref)
