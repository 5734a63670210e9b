"""Benchmark: one replica's synchronous SGD step of the AlexNet-shaped convnet.

Workload: batch 128, 224x224x3 synthetic N(0,1) images, bf16 storage with fp32
accumulation, conv 11x11/4 64 -> pool 3/2 -> 5x5 192 -> pool -> 3x3 384 ->
3x3 256 -> 3x3 256 -> pool, bias+ReLU after each conv, He-normal filters, an
N(0,1) upstream gradient of the last pool, plain SGD (lr 0.01) of every filter
and bias.  All inputs are resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--launch program|streams|graph|serial] [--no-cpu-baseline]

Prints one JSON line: ms per step (the timed region is K whole steps between
two device synchronisations), conv TFLOP/s against the bf16 MFMA peak, the
roofline entry of the dominant convolution kernel measured with HIP events on
the stream it runs on, warm (the step's cache state) and cold (caches flushed
before every op) per-op figures, and the CPU oracle timed on a bounded batch
slice, with its host's CPU model and a single-thread one-layer time.

Launch modes: ``streams`` (default) launches every op from the host, the filter
gradients on a second stream that overlaps the rest of the backward pass;
``graph`` replays the same two-stream step captured as one HIP graph; ``serial``
launches every op in order on one stream.
"""
from __future__ import annotations

import argparse
import ctypes
import faulthandler
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA: 256 CU x 4096 FLOP/clk x 2.4 GHz
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
METRIC = "ms per training step + conv TFLOP/s (% bf16 MFMA peak), AlexNet-shape b=128"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # (defaults: about 0.14 s of warm-up steps, by which the AlexNet step has reached its sustained
    # rate -- the first hundred steps after start-up run a few per cent slower -- then 200 timed)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--launch", choices=("program", "streams", "graph", "serial"), default="program",
                    help="the two-stream step recorded once and issued again from C++ (default), two streams "
                         "launched from Python, the two-stream step as a HIP graph, or one stream")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sampled", action="store_true", help="skip the sampled-softmax comparison")
    ap.add_argument("--metric-only", action="store_true",
                    help="only the metric's workload: no update, classifier or sampled-softmax figures "
                         "(for profiles of the step's kernels)")
    ap.add_argument("--classifier-steps", type=int, default=10,
                    help="also time this many steps of AlexNet with its classifier (fc layers + softmax "
                         "cross-entropy); 0 skips it")
    ap.add_argument("--cpu-sample", type=int, default=128, help="images of the batch the oracle steps through")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--gemm-reference", action="store_true",
                    help="only time the vendor bf16 GEMM (torch.matmul) on the GEMM shapes of the workload's convolutions "
                         "(no im2col), as a reference point, and exit")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain copy kernel over this many MiB (HBM counter calibration) and exit")
    return ap.parse_args()


def elementwise_bytes(net, op_kind, op, D, A=4):
    """Algorithmic HBM bytes of one elementwise op (read + write of its operands); A: bytes per
    stored pool selection (4 for dense indices, 1 for window taps)."""
    t = net.tensors
    if op_kind == "bias_relu_fwd":
        n = int(np.prod(t[op.dst][:3])) * op.cout
        return 2 * n * D
    if op_kind == "bias_relu_bwd":
        n = int(np.prod(t[op.dst][:3])) * op.cout
        return 3 * n * D
    if op_kind == "maxpool_fwd":
        nx = int(np.prod(t[op.src]))
        ny = int(np.prod(t[op.dst][:3])) * t[op.src][3]
        return nx * D + ny * (D + A)
    if op_kind == "maxpool_bwd":
        nx = int(np.prod(t[op.src]))
        ny = int(np.prod(t[op.dst][:3])) * t[op.src][3]
        return ny * (D + A) + nx * D
    if op_kind == "maxpool_relu_bwd":         # + read the ReLU output y, write dpre
        nx = int(np.prod(t[op.src]))
        ny = int(np.prod(t[op.dst][:3])) * t[op.src][3]
        return ny * (D + A) + 2 * nx * D
    raise KeyError(op_kind)


def kernel_source_sha():
    """Hash of the HIP sources: HBM counters recorded for other sources are not reported."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1605_08695_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


def recorded_traffic(kind):
    """HBM bytes per launch of the dominant kernel measured with rocprofv3 --pmc (FETCH_SIZE and
    WRITE_SIZE, scaled by a plain-copy calibration), if recorded for the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "alexnet_b128_conv_traffic.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_sha") != kernel_source_sha():
        return None
    return rec.get("bytes_per_launch", {}).get(kind)


# Algorithmic HBM bytes per fp32 variable of each in-place update (reads + writes, the bf16
# shadow of the new value included): SGD var,grad -> var; Momentum var,accum,grad -> var,accum;
# Adam var,m,v,grad -> var,m,v.
UPDATE_BYTES = {"sgd": 4 + 4 + 4 + 2, "momentum": 12 + 8 + 2, "adam": 16 + 12 + 2}


class HipEvent:
    """A timing event recorded without the system-scope fence (hipEventDisableSystemFence, the flag
    HIP gives events that only time work).  An ordinary event's fence writes back and invalidates
    the caches when it is reached, which also slows the work enqueued after it.  Same interface as
    torch.cuda.Event for what is used here: record(stream) and elapsed_time(end) in ms."""
    _hip = None

    def __init__(self):
        if HipEvent._hip is None:
            # the HIP runtime torch has loaded (the library's kernels run on the same one)
            path = next(l.split()[-1] for l in open("/proc/self/maps") if "libamdhip64" in l)
            h = ctypes.CDLL(path)
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._hip = h
        self.e = ctypes.c_void_p()
        if HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.e), 0x20000000) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream=None):
        import torch
        st = stream if stream is not None else torch.cuda.current_stream()
        if HipEvent._hip.hipEventRecord(self.e, ctypes.c_void_p(st.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        if HipEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.e, end.e) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if self.e.value and HipEvent._hip is not None:
            HipEvent._hip.hipEventDestroy(self.e)


def time_updates(torch, ops, n, reps=20):
    """Average launch time of each update over n fp32 variables (HIP events on the current stream)."""
    dev = "cuda"
    g = torch.Generator(device=dev).manual_seed(5)
    var = torch.randn(n, device=dev, generator=g)
    grad = torch.randn(n, device=dev, generator=g) * 1e-3
    s1, s2 = torch.zeros(n, device=dev), torch.zeros(n, device=dev)
    sh = torch.empty(n, dtype=torch.bfloat16, device=dev)
    calls = {
        "sgd": lambda t: ops.apply_sgd(var, grad, 1e-3, shadow=sh),
        "momentum": lambda t: ops.apply_momentum(var, s1, grad, 1e-3, 0.9, shadow=sh),
        "adam": lambda t: ops.apply_adam(var, s1, s2, grad, 1e-3, 0.9, 0.999, 1e-8, t, shadow=sh),
    }
    res = {}
    for name, fn in calls.items():
        for t in range(1, 4):
            fn(t)
        e0, e1 = HipEvent(), HipEvent()
        e0.record()
        for t in range(4, 4 + reps):
            fn(t)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        gbs = UPDATE_BYTES[name] * n / (us * 1e-6) / 1e9
        res[name] = {"us": round(us, 2), "gbs": round(gbs, 1), "pct_hbm_peak": round(100 * gbs / PEAK_HBM_GBS, 1)}
    del var, grad, s1, s2, sh
    return res


def conv_flops(net, op):
    n, oh, ow, _ = net.tensors[op.dst]
    cin = net.tensors[op.src][3]
    return 2.0 * n * oh * ow * op.kh * op.kw * cin * op.cout


class EventTrace:
    """Step-driver hook that brackets every op with HIP events on the stream it runs on.

    Before each start event the stream is given work that keeps the GPU busy while the host
    enqueues the event, the op and the end event, so the pair measures the op's kernels and no
    host launch gap: ``pad`` (a spin kernel of a few tens of microseconds, caches untouched:
    warm figures), or with ``flush`` (a byte buffer larger than the 256 MiB last-level cache)
    a fill of that buffer, which also evicts the op's inputs from every cache (cold figures)."""

    def __init__(self, torch, pad_cycles=0, flush=None):
        self.torch = torch
        self.pad_cycles = pad_cycles
        self.flush = flush
        self.rec = []           # (kind, op, start, end)

    def _stream(self, stream):
        return stream if stream is not None else self.torch.cuda.current_stream()

    def _event(self, stream):
        e = HipEvent()
        e.record(self._stream(stream))
        return e

    def _prefill(self, stream):
        with self.torch.cuda.stream(self._stream(stream)):
            if self.flush is not None:
                self.flush.fill_(1)
            elif self.pad_cycles:
                self.torch.cuda._sleep(self.pad_cycles)

    def __call__(self, event, op, stream=None, **t):
        if event.endswith(":end"):
            kind, op0, s = self.open
            assert kind == event[:-4] and op0 is op
            self.rec.append((kind, op0, s, self._event(stream)))
        else:
            self._prefill(stream)
            self.open = (event, op, self._event(stream))


def sleep_cycles_for(torch, us):
    """Spin-kernel cycles that take about ``us`` microseconds on this GPU (measured)."""
    torch.cuda._sleep(1000)
    torch.cuda.synchronize()
    e0, e1 = HipEvent(), HipEvent()
    n = 200000
    e0.record()
    torch.cuda._sleep(n)
    e1.record()
    torch.cuda.synchronize()
    per_us = n / max(e0.elapsed_time(e1) * 1e3, 1e-3)
    return max(1000, int(per_us * us))


def measure_classifier(args, torch, W, Replica):
    """AlexNet with its classifier at the same batch: the two-stream step, and each classifier op
    alone on one stream (HIP events), as a secondary figure (not the metric's workload)."""
    net = W.alexnet(batch=args.batch, classifier=True)
    inp = W.make_inputs(net, seed=args.seed)
    rep = Replica(net, inp)
    for _ in range(3):
        rep.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.classifier_steps):
        rep.step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.classifier_steps
    tr = EventTrace(torch)
    per = {}
    reps = 3
    for _ in range(reps):
        tr.rec.clear()
        rep.step(trace=tr, concurrent=False)
        torch.cuda.synchronize()
        for kind, op, s, e in tr.rec:
            if op is not None and op.name.startswith("fc") or kind == "softmax_xent":
                key = "%s/%s" % (kind, op.name)
                per[key] = per.get(key, 0.0) + s.elapsed_time(e) / reps
    fc_flop = 0.0
    for op in net.convs:
        if op.name.startswith("fc"):
            f = conv_flops(net, op)
            fc_flop += 3 * f if op.src != "x" else 2 * f
    fc_gemm_ms = sum(v for k, v in per.items() if k.split("/")[0].startswith("conv"))
    return {"workload": net.name, "ms_per_step": round(ms, 4), "images_per_s": round(args.batch / (ms * 1e-3), 1),
            "params": rep.n_params, "loss_last_step": round(rep.loss_value(), 4),
            "fc_gemm_tflops": round(fc_flop / (fc_gemm_ms * 1e-3) / 1e12, 1),
            "per_op_ms": {k: round(v, 4) for k, v in sorted(per.items())}}


def measure_sampled(args, torch, W):
    """The language-model classifier of the paper's second workload in miniature: 2560 rows (128
    sequences x 20 steps) of a 512-wide output, 40000 classes, 512 sampled per batch; one sampled-
    softmax step against one full-softmax step (HIP events on the current stream)."""
    from paper_1605_08695_amd.sampled import FullSoftmaxHead, SampledSoftmaxHead
    n, d, vocab, m = 2560, 512, 40000, 512
    inp = W.make_sampled_inputs(n, d, vocab, m, seed=args.seed)
    h = torch.from_numpy(inp.h).to(torch.bfloat16).cuda()
    sh = SampledSoftmaxHead(inp.W, inp.b, lr=0.1)
    bt = sh.prepare(inp.labels, inp.sampled, inp.lq_true, inp.lq_sampled)
    fh = FullSoftmaxHead(inp.W, inp.b, lr=0.1)
    lab = torch.from_numpy(inp.labels).cuda()

    def timed(fn, reps=10):
        for _ in range(3):
            fn()
        e0, e1 = HipEvent(), HipEvent()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps
    ms_s = timed(lambda: sh.run(h, bt))
    ms_f = timed(lambda: fh.run(h, lab))
    return {"rows": n, "dim": d, "classes": vocab, "sampled": m, "candidates": bt["u"],
            "sampled_ms": round(ms_s, 4), "full_ms": round(ms_f, 4), "full_over_sampled": round(ms_f / ms_s, 1),
            "classes_over_candidates": round(vocab / bt["u"], 1)}


def measure_workloads(args, torch, W, Replica):
    """The other step configurations at their full sizes (two-stream launch): ms per step and the
    direct-convolution FLOP rate of the whole step (every op's time included)."""
    out = {}
    for make in (W.single_layer, W.vgg16, W.googlenet, W.inception_v3):
        net = make()
        print("bench: workload %s" % net.name, file=sys.stderr, flush=True)
        rep = Replica(net, W.make_inputs(net, seed=args.seed))
        for _ in range(2):
            rep.step()
        torch.cuda.synchronize()
        steps = 5
        t0 = time.perf_counter()
        for _ in range(steps):
            rep.step()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        # the same step captured once as a HIP graph and replayed: no per-launch host cost
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            rep.step()
        torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            rep.step()
        g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            g.replay()
        torch.cuda.synchronize()
        ms_g = (time.perf_counter() - t0) * 1e3 / steps
        # the step recorded once into a program and issued again from C++
        prog = rep.record_step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            rep.run_program(prog)
        torch.cuda.synchronize()
        ms_p = (time.perf_counter() - t0) * 1e3 / steps
        prog.close()
        fl = W.conv_flops(net)
        best = min(ms, ms_g, ms_p)
        out[net.name] = {"batch": net.tensors["x"][0], "dtype": net.dtype, "ms_per_step": round(ms, 3),
                         "ms_per_step_graph": round(ms_g, 3), "ms_per_step_program": round(ms_p, 3),
                         "ops": len(net.ops),
                         "conv_gflop_per_step": round(fl / 1e9, 1),
                         "step_tflops": round(fl / (best * 1e-3) / 1e12, 1)}
        del g
        del rep
        torch.cuda.empty_cache()
    return out


def gemm_reference(net, torch):
    """Vendor-library bf16 GEMMs with the (M, N, K) of every convolution direction, for reference only."""
    def t(fn, it=20):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = HipEvent(), HipEvent()
        a.record()
        for _ in range(it):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / it * 1e3
    out = {}
    for op in net.convs:
        n, h, w, c = net.tensors[op.src]
        _, oh, ow, k = net.tensors[op.dst][:3] + (op.cout,)
        M, N, K = n * oh * ow, op.cout, op.kh * op.kw * c
        fl = 2.0 * M * N * K
        A = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
        B = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
        G = torch.randn(M, N, device="cuda", dtype=torch.bfloat16)
        Bt, At = B.t().contiguous(), A.t().contiguous()
        us = {"fwd [M,K]x[K,N]": t(lambda: A @ B), "bwd_input [M,N]x[N,K]": t(lambda: G @ Bt),
              "bwd_filter [K,M]x[M,N]": t(lambda: At @ G)}
        out[op.name] = {"M": M, "N": N, "K": K,
                        "us": {k2: round(v, 1) for k2, v in us.items()},
                        "tflops": {k2: round(fl / v / 1e6, 1) for k2, v in us.items()}}
        del A, B, G, Bt, At
    print(json.dumps({"gemm_reference": out}))


CONV_CALLS = {"conv2d_fwd_bias_relu": "conv_fwd", "conv2d_fwd_bias_relu_maxpool": "conv_fwd", "conv2d_fwd": "conv_fwd",
              "conv2d_bwd_input": "conv_bwd_input",
              "conv2d_bwd_input_relu_bwd": "conv_bwd_input", "conv2d_bwd_filter": "conv_bwd_filter"}


def record_conv_calls(torch, ops, rep):
    """The convolution calls of one one-stream step, in order: (kind, function, args, kwargs).  A
    convolution called with the max-pool of its output is recorded as the convolution alone (bias +
    ReLU epilogue, same output), so that the group times the implicit-GEMM kernel only."""
    calls, saved = [], {}
    conv_only = ops.conv2d_fwd_bias_relu
    for name, kind in CONV_CALLS.items():
        fn = getattr(ops, name)
        saved[name] = fn

        def wrap(*a, _fn=fn, _kind=kind, _name=name, **k):
            if _name == "conv2d_fwd_bias_relu_maxpool":
                calls.append((_kind, conv_only, a[:5], {"y": k["y"], "ws": k["ws"], "stream": k["stream"]}))
            else:
                calls.append((_kind, _fn, a, k))
            return _fn(*a, **k)
        setattr(ops, name, wrap)
    try:
        rep.step(concurrent=False)
        torch.cuda.synchronize()
    finally:
        for name, fn in saved.items():
            setattr(ops, name, fn)
    return calls


def time_back_to_back(torch, calls, pad, reps=20):
    """Average duration of each call launched reps times back to back on the current stream, between
    two HIP events on that stream (after a spin kernel that covers the host's enqueueing)."""
    out = []
    for kind, fn, a, k in calls:
        fn(*a, **k)
        torch.cuda.synchronize()
        torch.cuda._sleep(pad)
        e0, e1 = HipEvent(), HipEvent()
        e0.record()
        for _ in range(reps):
            fn(*a, **k)
        e1.record()
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) * 1e3 / reps)
    return out


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def per_op_pass(torch, rep, tr, reps):
    """Average event duration of every op (one-stream step, ``tr`` brackets each op), by kind and
    by (kind, layer)."""
    per_kind, per_layer = {}, {}
    for r in range(reps):
        tr.rec.clear()
        rep.step(trace=tr, concurrent=False)
        torch.cuda.synchronize()
        for kind, op, s, e in tr.rec:
            ms = s.elapsed_time(e)
            if kind in ("conv_bias_relu_fwd", "conv_bias_relu_maxpool_fwd"):
                kind = "conv_fwd"       # the forward convolution with its bias + ReLU (+ max-pool) epilogue
            if kind == "conv_bwd_input_relu_bwd":
                kind = "conv_bwd_input"  # the input gradient with the producer's ReLU backward epilogue
            per_kind[kind] = per_kind.get(kind, 0.0) + ms / reps
            key = (kind, op.name if op is not None else "all")
            per_layer[key] = per_layer.get(key, 0.0) + ms / reps
    return per_kind, per_layer


def step_figures(net, rep, per_kind, per_layer, D):
    """Conv FLOP rates and elementwise HBM rates of one per-op pass."""
    conv_kinds = ("conv_fwd", "conv_bwd_input", "conv_bwd_filter")
    conv_ms = sum(per_kind.get(k, 0.0) for k in conv_kinds)
    flops = {k: 0.0 for k in conv_kinds}
    for op in net.convs:
        f = conv_flops(net, op)
        flops["conv_fwd"] += f
        flops["conv_bwd_filter"] += f
        if op.src != "x" or net.input_grad:
            flops["conv_bwd_input"] += f
    conv_flop = sum(flops.values())
    ew_kinds = ("bias_relu_fwd", "bias_relu_bwd", "maxpool_fwd", "maxpool_bwd", "maxpool_relu_bwd")
    ew_bytes = {k: 0.0 for k in ew_kinds}
    for op in net.ops:
        # the kinds this op actually ran as (bias + ReLU forward runs in the conv epilogue; a pool
        # fused with the ReLU backward of its producer replaces that conv's bias_relu_bwd)
        if hasattr(op, "cout"):
            kinds = [] if op.name in rep.relu_fused else ["bias_relu_bwd"]
        else:
            kinds = [] if op.name in rep.pool_in_conv else ["maxpool_fwd"]
            if op.name in rep.pool_relu:
                kinds.append("maxpool_relu_bwd")
            elif op.src != "x":
                kinds.append("maxpool_bwd")
        A = rep.argmax[op.name].element_size() if op.name in rep.argmax else 4
        for k in kinds:
            ew_bytes[k] += elementwise_bytes(net, k, op, D, A)
    sgd_bytes = rep.n_params * 14.0
    ew_ms = sum(per_kind.get(k, 0.0) for k in ew_kinds) + per_kind.get("apply_sgd", 0.0)
    ew_total = sum(ew_bytes.values()) + sgd_bytes
    by_kind = {}
    for k in ew_kinds:
        if per_kind.get(k):
            by_kind[k] = round(ew_bytes[k] / (per_kind[k] * 1e-3) / 1e9, 1)
    if per_kind.get("apply_sgd"):
        by_kind["apply_sgd"] = round(sgd_bytes / (per_kind["apply_sgd"] * 1e-3) / 1e9, 1)
    return {"flops": flops, "conv_flop": conv_flop, "conv_ms": conv_ms,
            "conv_tflops": conv_flop / (conv_ms * 1e-3) / 1e12,
            "conv_tflops_by_direction": {k: round(flops[k] / (per_kind[k] * 1e-3) / 1e12, 1) for k in conv_kinds},
            "ew_ms": ew_ms, "ew_bytes": ew_total, "ew_gbs": ew_total / (ew_ms * 1e-3) / 1e9,
            "ew_gbs_by_kind": by_kind}


def main():
    faulthandler.enable()            # a crash prints where every thread was
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs one replica on one GPU; multi-GPU data parallelism is not built "
              "(requested --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1605_08695_amd import ops
    from paper_1605_08695_amd import workloads as W
    from paper_1605_08695_amd.step import Replica

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy_mib:
        # A plain elementwise copy of known size: reads and writes n * 4 bytes per launch.
        n = args.calibrate_copy_mib * (1 << 20) // 4
        a = torch.ones(n, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            torch.neg(a, out=b)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes_read": n * 4, "calibration_copy_bytes_written": n * 4}))
        return
    net = W.alexnet(batch=args.batch)
    if args.gemm_reference:
        gemm_reference(net, torch)
        return
    inp = W.make_inputs(net, seed=args.seed)
    rep = Replica(net, inp)
    D = 2
    torch.cuda.synchronize()
    print("bench: %s, %d params, %.1f GFLOP/step" % (net.name, rep.n_params, W.conv_flops(net) / 1e9),
          file=sys.stderr, flush=True)

    # ---------------------------------------------------------------- timed region
    graph = None
    if args.launch == "graph":
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(2):
                rep.step()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            rep.step()
        run = graph.replay
    elif args.launch == "program":
        prog = rep.record_step()           # the recording run is the first warm-up step
        run = lambda: rep.run_program(prog)
    else:
        concurrent = args.launch == "streams"
        run = lambda: rep.step(concurrent=concurrent)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    # The K timed steps run back to back with nothing between them; a timing event records with a
    # system-scope fence (a cache write-back and invalidation that also slows the work after it),
    # so the per-step distribution (median, p10, p90) comes from K more steps, each bracketed by
    # events, after the timed region.
    t0 = time.perf_counter()
    for i in range(args.steps):
        run()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    ev = [HipEvent() for _ in range(args.steps + 1)]
    ev[0].record()
    for i in range(args.steps):
        run()
        ev[i + 1].record()
    torch.cuda.synchronize()
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    print("bench: timed %d steps, %.3f ms/step (median %.3f)" % (args.steps, ms_per_step, np.median(step_ms)),
          file=sys.stderr, flush=True)

    # ---------------------------------------------------------------- host enqueue time
    # Wall time of the host call that enqueues one step, with the GPU kept busy by a spin kernel
    # queued first (so the call never waits for the device): Python launches on two streams or
    # one, and the recorded program issued from C++.
    def host_ms(fn, reps=5):
        out = []
        for _ in range(reps):
            torch.cuda.synchronize()
            torch.cuda._sleep(20_000_000)
            h0 = time.perf_counter()
            fn()
            out.append((time.perf_counter() - h0) * 1e3)
        torch.cuda.synchronize()
        return round(float(np.median(out)), 4)
    hprog = prog if args.launch == "program" else rep.record_step()
    host_enqueue = {"streams": host_ms(lambda: rep.step(concurrent=True)),
                    "serial": host_ms(lambda: rep.step(concurrent=False)),
                    "program": host_ms(lambda: rep.run_program(hprog))}
    print("bench: host enqueue ms per step %s" % host_enqueue, file=sys.stderr, flush=True)

    # ---------------------------------------------------------------- per-op events
    # Every op launched alone, in order, on one stream and bracketed by HIP events on that
    # stream: the duration of each op's kernels by themselves (in the two-stream step the filter
    # gradients share the GPU with the input gradients), from which the roofline is taken.  Each
    # op's start event is preceded on its stream by work that keeps the GPU busy while the host
    # enqueues the op (so no launch gap is counted): a spin kernel for the warm figures (the
    # step's real cache state), a 512 MiB fill for the cold ones (every cache flushed).
    reps = max(3, min(10, args.steps))
    pad = sleep_cycles_for(torch, 200.0)
    print("bench: per-op pass (warm, cold)", file=sys.stderr, flush=True)
    warm = per_op_pass(torch, rep, EventTrace(torch, pad_cycles=pad), reps)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold = per_op_pass(torch, rep, EventTrace(torch, flush=flush), reps)
    del flush
    per_kind, per_layer = warm
    # the roofline groups' launches again, each repeated back to back (event overhead amortised)
    conv_calls = record_conv_calls(torch, ops, rep)
    fig_w = step_figures(net, rep, *warm, D)
    fig_c = step_figures(net, rep, *cold, D)
    conv_kinds = ("conv_fwd", "conv_bwd_input", "conv_bwd_filter")
    flops, conv_flop = fig_w["flops"], fig_w["conv_flop"]
    conv_tflops = fig_w["conv_tflops"]
    ew_gbs = fig_w["ew_gbs"]

    # ---------------------------------------------------------------- in-place updates alone
    # over this network's variables and over 61.1M variables (AlexNet with its classifier)
    updates = None
    if not args.metric_only:
        updates = {"bytes_per_variable": UPDATE_BYTES,
                   "this_net": dict(n=rep.n_params, **time_updates(torch, ops, rep.n_params)),
                   "alexnet_with_classifier": dict(n=61_100_840, **time_updates(torch, ops, 61_100_840))}

    classifier = None
    if args.classifier_steps > 0 and not args.metric_only:
        print("bench: AlexNet with its classifier", file=sys.stderr, flush=True)
        classifier = measure_classifier(args, torch, W, Replica)
    if not (args.no_sampled or args.metric_only):
        print("bench: sampled softmax", file=sys.stderr, flush=True)
    sampled = None if args.no_sampled or args.metric_only else measure_sampled(args, torch, W)
    others = None if args.metric_only else measure_workloads(args, torch, W, Replica)

    # ---------------------------------------------------------------- CPU baseline: the oracle
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        from oracle import net as onet
        oracle.build()
        k = max(1, min(args.cpu_sample, args.batch))
        snet = W.alexnet(batch=k)
        sinp = W.make_inputs(net, seed=args.seed, batch_slice=k)
        print("bench: oracle step on %d images ..." % k, file=sys.stderr, flush=True)
        c0 = time.perf_counter()
        onet.step(snet, sinp.x, sinp.weights, sinp.biases, sinp.g)
        c1 = time.perf_counter()
        # one layer on one thread: AlexNet conv3 forward (3x3, 192 -> 384 channels at 13x13) on 4 images
        lay = next(op for op in net.convs if op.name == "conv3")
        nt = oracle.num_threads()
        xs = np.random.default_rng(1).standard_normal((4,) + net.tensors[lay.src][1:])
        ws = sinp.weights[lay.name]
        oracle.set_num_threads(1)
        try:
            t0 = time.perf_counter()
            oracle.conv2d_fwd(xs, ws, (lay.sh, lay.sw), lay.pads)
            t_one = time.perf_counter() - t0
        finally:
            oracle.set_num_threads(nt)
        f_one = conv_flops(net, lay) * 4 / args.batch
        cpu = {"value": round((c1 - c0) * 1e3 * args.batch / k, 1), "unit": "ms/step",
               "cores": nt, "kind": "oracle", "cpu_model": cpu_model(),
               "sample": "%d of the %d images of one step (fp64 loop nests, %.1f s); oracle cost is linear "
                         "in batch, scaled x%g" % (k, args.batch, c1 - c0, args.batch / k),
               "single_thread_layer": {"layer": "conv3 forward, 4 images", "s": round(t_one, 3),
                                       "gflops": round(f_one / t_one / 1e9, 3),
                                       "full_batch_s_scaled": round(t_one * args.batch / 4, 1)}}

    # The roofline kernel: the convolution kernel with the most time per step.  The first layer
    # (3 input channels) runs the band kernels, every other layer of a direction the implicit-GEMM
    # kernel, so a group is one direction over the layers after the first.  Each group's launches
    # (in step order) are timed back to back and the slowest group is the roofline's: the three
    # directions carry the same FLOPs and their one-at-a-time figures lie within event noise of
    # each other, so the back-to-back time is the stable choice.
    groups = {}
    for (kind, name), ms in per_layer.items():
        if kind in conv_kinds and name != net.convs[0].name:
            g = groups.setdefault(kind, [0.0, 0, 0.0])
            g[0] += ms
            g[1] += 1
            g[2] += conv_flops(net, next(op for op in net.convs if op.name == name))
    b2b_by_group = {}
    for kind in groups:
        dcalls = [c for c in conv_calls if c[0] == kind]
        if kind == "conv_fwd":
            dcalls = dcalls[1:]
        elif kind == "conv_bwd_filter":
            dcalls = dcalls[:-1]
        b2b_by_group[kind] = time_back_to_back(torch, dcalls, pad)
    dom = max(groups, key=lambda k: sum(b2b_by_group[k]))
    dom_ms, n_dom, dom_flop = groups[dom]
    b2b_us = b2b_by_group[dom]
    cold_ms = sum(v for (kind, name), v in cold[1].items() if kind == dom and name != net.convs[0].name)
    dom_layers = [op.name for op in net.convs[1:]]
    out = {
        "metric": METRIC,
        "value": round(ms_per_step, 4),
        "unit": "ms/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "alexnet_b%d" % args.batch, "global_batch": args.batch, "image": [224, 224, 3],
                   "layers": "conv11x11/4-64,pool3/2,conv5x5-192,pool3/2,conv3x3-384,conv3x3-256,conv3x3-256,pool3/2",
                   "launch": {"streams": "host launches, two streams", "graph": "hip_graph, two streams",
                              "program": "recorded program issued from C++, two streams",
                              "serial": "host launches, one stream"}[args.launch]},
        "host_enqueue_ms": host_enqueue,
        "step_ms_median": round(float(np.median(step_ms)), 4),
        "step_ms_p10": round(float(np.percentile(step_ms, 10)), 4),
        "step_ms_p90": round(float(np.percentile(step_ms, 90)), 4),
        "images_per_s": round(args.batch / (ms_per_step * 1e-3), 1),
        "conv_gflop_per_step": round(conv_flop / 1e9, 2),
        "conv_tflops": round(conv_tflops, 1),
        "conv_pct_bf16_peak": round(100 * conv_tflops / PEAK_BF16_TFLOPS, 2),
        "conv_tflops_by_direction": fig_w["conv_tflops_by_direction"],
        "eltwise_gbs": round(ew_gbs, 1),
        "eltwise_pct_hbm_peak": round(100 * ew_gbs / PEAK_HBM_GBS, 2),
        "eltwise_gbs_by_kind": fig_w["ew_gbs_by_kind"],
        "cold": {"what": "every op after a 512 MiB fill of a scratch buffer on its stream (caches flushed)",
                 "conv_tflops": round(fig_c["conv_tflops"], 1),
                 "conv_pct_bf16_peak": round(100 * fig_c["conv_tflops"] / PEAK_BF16_TFLOPS, 2),
                 "conv_tflops_by_direction": fig_c["conv_tflops_by_direction"],
                 "eltwise_gbs": round(fig_c["ew_gbs"], 1),
                 "eltwise_pct_hbm_peak": round(100 * fig_c["ew_gbs"] / PEAK_HBM_GBS, 2),
                 "eltwise_gbs_by_kind": fig_c["ew_gbs_by_kind"],
                 "per_op_ms": {k: round(v, 4) for k, v in sorted(cold[0].items())}},
        "per_op_ms": {k: round(v, 4) for k, v in sorted(per_kind.items())},
        "roofline": {"kernel": "%s implicit-GEMM kernel of %s (%d launches/step)" % (dom, ",".join(dom_layers), n_dom),
                     "bound": "mfma",
                     "achieved": round(dom_flop / (sum(b2b_us) * 1e-6) / 1e12, 1),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(dom_flop / (sum(b2b_us) * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
                     "traffic": recorded_traffic(dom),
                     "avg_launch_us": round(sum(b2b_us) / len(b2b_us), 2),
                     "avg_launch_us_by_layer": [round(u, 2) for u in b2b_us],
                     "measured": "HIP events on the launch stream around 20 back-to-back launches of each of "
                                 "the group's calls (the stream kept busy ahead of the start event; a "
                                 "convolution the step runs with its max-pool is timed without the pool)",
                     "avg_launch_us_isolated": round(dom_ms * 1e3 / n_dom, 2),
                     "avg_launch_us_cold": round(cold_ms * 1e3 / n_dom, 2),
                     "avg_launch_us_by_group": {k: round(sum(v) / len(v), 2) for k, v in sorted(b2b_by_group.items())},
                     "flop_per_launch": round(dom_flop / n_dom)},
        "cpu_baseline": cpu,
        "updates": updates,
        "classifier": classifier,
        "sampled_softmax": sampled,
        "other_workloads": others,
    }
    print(json.dumps(out))
    print("per-layer ms:", json.dumps({"%s/%s" % k: round(v, 4) for k, v in sorted(per_layer.items())}),
          file=sys.stderr)


if __name__ == "__main__":
    main()
