"""Whole-step parity of the HIP path against the CPU oracle (GPU).

* single-layer fp32 step end to end against the oracle's own step;
* single-layer fp32 steps with Momentum and Adam updates against the oracle's;
* every op of every workload oracle-forced (its inputs overwritten with the
  oracle's values before it runs), at reduced batch (and, for VGG, reduced
  image size) so the oracle finishes in seconds;
* the AlexNet-shaped step at its full size (batch 128, the bench's launch
  configuration) on 4 distinct images repeated 32 times, whole tensors, and on
  128 distinct images (the oracle steps through the whole batch);
* the VGG-16, GoogLeNet and Inception-v3 steps at their configured sizes on a
  few repeated images (whole tensors), and every configured step at full size
  on all-distinct images with sampled convolution outputs and filter-gradient
  entries (SampledParityTracer);
* determinism, restore-and-rerun, the two-stream step against the one-stream
  step, and a captured HIP graph replayed against eager steps.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import net as onet
from paper_1605_08695_amd import workloads as W
from paper_1605_08695_amd.step import Replica
from tests.gpu_parity import ParityTracer, SampledParityTracer, err, f64, say, ulp_diff_f32

pytestmark = pytest.mark.gpu


def bitwise_equal(a, b):
    bits = {2: torch.int16, 4: torch.int32}[a.element_size()]
    return torch.equal(a.view(bits), b.view(bits))


def _report(tr):
    for (kind, metric), (value, bar, name, _) in sorted(tr.summary().items()):
        say("  %-24s %-14s worst %.3e (bar %.0e) at %s" % (kind, metric, value, bar, name))
    bad = tr.failures()
    for b in bad[:20]:
        say("  FAIL", b)
    return bad


def test_single_layer_step_end_to_end():
    """fp32 single-layer step (x[8,32,32,16]) against the oracle's fp64 step, end to end."""
    net = W.single_layer()
    inp = W.make_inputs(net, seed=0)
    rep = Replica(net, inp)
    rep.step()
    torch.cuda.synchronize()
    ref = onet.step(net, inp.x, inp.weights, inp.biases, inp.g)
    c = net.convs[0].name
    e = {
        "conv_out": err(f64(rep.act[c]), ref["acts"][c]),
        "pool": err(f64(rep.act[net.output]), ref["acts"][net.output]),
        "dW": err(f64(rep.dW[c]), ref["dW"][c]),
        "db": err(f64(rep.db[c]), ref["db"][c]),
        "dx": err(f64(rep.grad["x"]), ref["grads"]["x"]),
    }
    say("single layer end-to-end:", {k: "%.2e" % v for k, v in e.items()})
    assert all(v <= 1e-4 for v in e.values()), e
    # argmax: mismatches allowed only where the oracle's window top-2 gap is tiny
    am = ParityTracer._dense(rep.argmax[net.ops[1].name], rep.act[c].shape, net.ops[1])
    ref_am = ref["argmax"][net.ops[1].name]
    mism = np.argwhere(am != ref_am)
    y = ref["acts"][c]
    rms = np.sqrt(np.mean(y ** 2))
    for (n, oh, ow, ch) in mism:
        win = np.sort(y[n, 2 * oh:2 * oh + 2, 2 * ow:2 * ow + 2, ch].ravel())
        assert win[-1] - win[-2] <= 1e-5 * rms
    say("  argmax mismatches (near-ties only):", len(mism))
    # the updated variables against the oracle's: the fp32 rounding of the update plus lr times
    # the gradient bar (the replica starts from the fp32 values of the weights)
    lr = float(np.float32(net.lr))
    w0 = inp.weights[c].astype(np.float32).astype(np.float64)
    dw_ref = ref["dW"][c]
    w_ref = oracle.apply_sgd(w0, dw_ref, lr)
    tol = 2.0 ** -23 * np.abs(w_ref) + lr * 1e-4 * np.sqrt(np.mean(dw_ref ** 2))
    assert np.all(np.abs(f64(rep.W[c]) - w_ref) <= tol)


@pytest.mark.parametrize("opt", ["momentum", "nesterov", "adam"])
def test_single_layer_steps_with_momentum_and_adam(opt):
    """Two fp32 single-layer steps with a Momentum or Adam update against the oracle's two steps
    (forward, backward, then the same update rule), from zero optimizer slots."""
    say("optimizer step", opt)
    net = W.single_layer(batch=4, hw=16)
    inp = W.make_inputs(net, seed=4)
    c = net.convs[0].name
    lr = float(np.float32(net.lr))
    f = lambda v: float(np.float32(v))
    g1 = onet.step(net, inp.x, inp.weights, inp.biases, inp.g)
    # Adam's step is nearly sign(g) when eps is tiny; an eps of the gradient's size keeps the
    # update Lipschitz in the gradient, so the gradient bar carries over to the variables
    eps = f(max(np.sqrt(np.mean(g1["dW"][c] ** 2)), np.sqrt(np.mean(g1["db"][c] ** 2))))
    kw = dict(momentum=f(0.9), nesterov=(opt == "nesterov"), beta1=f(0.9), beta2=f(0.999), epsilon=eps)
    rep = Replica(net, inp, optimizer="adam" if opt == "adam" else "momentum", **kw)
    w = {c: inp.weights[c].astype(np.float32).astype(np.float64)}
    b = {c: inp.biases[c].astype(np.float32).astype(np.float64)}
    slots = {k: [np.zeros_like(w[c]), np.zeros_like(w[c])] if k == "w" else [np.zeros_like(b[c])] * 2
             for k in ("w", "b")}
    for t in (1, 2):
        rep.step()
        ref = onet.step(net, inp.x, w, b, inp.g)
        for key, var, grad in (("w", w, ref["dW"][c]), ("b", b, ref["db"][c])):
            s0 = slots[key]
            if opt == "adam":
                var[c], s0[0], s0[1] = oracle.apply_adam(var[c], s0[0], s0[1], grad, lr, kw["beta1"], kw["beta2"],
                                                         eps, t)
            else:
                var[c], s0[0] = oracle.apply_momentum(var[c], s0[0], grad, lr, kw["momentum"], kw["nesterov"])
    torch.cuda.synchronize()
    w0 = inp.weights[c].astype(np.float32).astype(np.float64)
    b0 = inp.biases[c].astype(np.float32).astype(np.float64)
    e_w = err(f64(rep.W[c]) - w0, w[c] - w0)
    e_b = err(f64(rep.b[c]) - b0, b[c] - b0)
    say("  variable change err: W %.2e  b %.2e" % (e_w, e_b))
    assert e_w <= 1e-3 and e_b <= 1e-3, (e_w, e_b)
    assert rep.t == 2


SMALL = [
    ("single_layer", lambda: W.single_layer(batch=4, hw=16)),
    ("alexnet_b2", lambda: W.alexnet(batch=2)),
    ("vgg16_b2_32px", lambda: W.vgg16(batch=2, hw=32)),
    ("googlenet_b2", lambda: W.googlenet(batch=2)),
    ("inception_v3_b1", lambda: W.inception_v3(batch=1)),
    ("classifier_small_f32", lambda: W.classifier_small(batch=4)),
    ("classifier_small_bf16", lambda: W.classifier_small(batch=4, dtype="bf16")),
    ("alexnet_classifier_b2", lambda: W.alexnet(batch=2, classifier=True)),
]


@pytest.mark.parametrize("name,make", SMALL, ids=[s[0] for s in SMALL])
def test_step_every_op_oracle_forced(name, make):
    net = make()
    say("oracle-forced step:", net.name, "ops", len(net.ops))
    inp = W.make_inputs(net, seed=0)
    rep = Replica(net, inp)
    tr = ParityTracer(rep, inp, label=name)
    rep.step(trace=tr)
    torch.cuda.synchronize()
    bad = _report(tr)
    n_checked = len(tr.results)
    assert n_checked >= 4 * len(net.convs)
    assert not bad


def test_alexnet_full_size_repeated_images():
    """The bench workload at full size (batch 128) and launch configuration (two streams), with
    4 distinct images repeated 32 times: every op's output against the oracle's, per-image
    outputs repeating bit for bit, and whole filter and bias gradients (32 times the oracle's
    4-image sums)."""
    net = W.alexnet(batch=128)
    inp = W.make_inputs(net, seed=0)
    rep = Replica(net, inp)
    tr = ParityTracer(rep, inp, distinct=4, label="alexnet_b128")
    rep.step(trace=tr)
    torch.cuda.synchronize()
    bad = _report(tr)
    assert not bad


FULL_REPEATED = [
    ("vgg16_b64", lambda: W.vgg16(batch=64), 2),
    ("googlenet_b128", lambda: W.googlenet(batch=128), 4),
    ("inception_v3_b32", lambda: W.inception_v3(batch=32), 2),
]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,make,distinct", FULL_REPEATED, ids=[c[0] for c in FULL_REPEATED])
def test_full_size_repeated_images(name, make, distinct):
    """The VGG-16 (batch 64, 224x224), GoogLeNet (batch 128) and Inception-v3 (batch 32) steps at
    their configured sizes and launch configuration (two streams), with a few distinct images
    repeated along the batch so the oracle steps through them in seconds: every op's output
    against the oracle's (whole tensors, repeats bit for bit), whole filter and bias gradients."""
    net = make()
    say("full-size repeated-image step:", name, "ops", len(net.ops), "distinct", distinct)
    inp = W.make_inputs(net, seed=0)
    rep = Replica(net, inp)
    tr = ParityTracer(rep, inp, distinct=distinct, label=name)
    rep.step(trace=tr)
    torch.cuda.synchronize()
    bad = _report(tr)
    assert len(tr.results) >= 4 * len(net.convs)
    assert not bad


@pytest.mark.timeout(900)
def test_alexnet_full_size_all_distinct():
    """The bench workload at full size (batch 128, two streams) with 128 distinct images: the
    oracle steps through the whole batch, every op's whole output is compared (a kernel reading
    another image's data cannot pass), whole filter and bias gradients."""
    net = W.alexnet(batch=128)
    inp = W.make_inputs(net, seed=7)
    rep = Replica(net, inp)
    tr = ParityTracer(rep, inp, label="alexnet_b128_distinct")
    rep.step(trace=tr)
    torch.cuda.synchronize()
    bad = _report(tr)
    assert not bad


FULL_SAMPLED = [
    ("vgg16_b64", lambda: W.vgg16(batch=64), (0, 29, 63)),
    ("googlenet_b128", lambda: W.googlenet(batch=128), (0, 77, 127)),
    ("inception_v3_b32", lambda: W.inception_v3(batch=32), (0, 13, 31)),
    ("alexnet_b128", lambda: W.alexnet(batch=128), (0, 64, 127)),
]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,make,sample", FULL_SAMPLED, ids=[c[0] for c in FULL_SAMPLED])
def test_full_size_all_distinct_sampled(name, make, sample):
    """Every configured step at full size with all-distinct images (SampledParityTracer): pools,
    ReLU backward and bias gradients against the oracle on every image; convolution outputs on the
    sampled images; filter gradients at 256 seeded entries summed over the whole batch."""
    net = make()
    say("full-size all-distinct sampled step:", name, "sample", sample)
    inp = W.make_inputs(net, seed=11)
    rep = Replica(net, inp)
    tr = SampledParityTracer(rep, inp, sample=sample, label=name)
    rep.step(trace=tr)
    torch.cuda.synchronize()
    bad = _report(tr)
    say("  unchecked here (left to the repeated-image test):", len(tr.skipped), "fused bias gradients")
    assert len(tr.results) >= 3 * len(net.convs)
    assert not bad


def test_alexnet_classifier_full_size_repeated_images():
    """AlexNet with its classifier (fc 4096, 4096, 1000 and the softmax cross-entropy) at batch 128,
    4 distinct images repeated 32 times, every op against the oracle."""
    net = W.alexnet(batch=128, classifier=True)
    inp = W.make_inputs(net, seed=0)
    rep = Replica(net, inp)
    tr = ParityTracer(rep, inp, distinct=4, label="alexnet_cls_b128")
    rep.step(trace=tr)
    torch.cuda.synchronize()
    bad = _report(tr)
    assert not bad


def test_classifier_step_end_to_end():
    """fp32 classifier step (conv, pool, fc + ReLU, fc logits, softmax cross-entropy) against the
    oracle's step, end to end with no forcing: loss, every gradient and the input gradient."""
    net = W.classifier_small(batch=4)
    inp = W.make_inputs(net, seed=6)
    rep = Replica(net, inp)
    rep.step()
    torch.cuda.synchronize()
    ref = onet.step(net, inp.x, inp.weights, inp.biases, None, labels=inp.labels)
    e = {"loss": abs(rep.loss_value() - ref["loss"]) / abs(ref["loss"]), "dx": err(f64(rep.grad["x"]), ref["grads"]["x"])}
    for c in net.convs:
        e["dW_" + c.name] = err(f64(rep.dW[c.name]), ref["dW"][c.name])
        e["db_" + c.name] = err(f64(rep.db[c.name]), ref["db"][c.name])
    say("classifier end-to-end:", {k: "%.2e" % v for k, v in e.items()})
    assert all(v <= 1e-4 for v in e.values()), e


@pytest.mark.parametrize("make", [lambda: W.single_layer(), lambda: W.googlenet(batch=4)],
                         ids=["single_layer", "googlenet_b4"])
def test_step_deterministic_and_restorable(make):
    net = make()
    net.lr = 1e-6            # keep the linear surrogate loss from driving values to inf
    inp = W.make_inputs(net, seed=1)
    rep = Replica(net, inp)
    snap = rep.snapshot()
    rep.step()
    p1, g1 = rep.params.clone(), rep.grads.clone()
    rep.restore(snap)
    rep.step()
    torch.cuda.synchronize()
    assert bool(torch.isfinite(rep.params).all())
    assert bitwise_equal(p1, rep.params) and bitwise_equal(g1, rep.grads)


@pytest.mark.parametrize("make", [lambda: W.alexnet(batch=8), lambda: W.googlenet(batch=4),
                                  lambda: W.inception_v3(batch=2)],
                         ids=["alexnet_b8", "googlenet_b4", "inception_v3_b2"])
def test_two_stream_step_matches_one_stream(make):
    """Forward branches on the lane streams and filter gradients on the second stream
    (overlapping the input gradients) must give bit-identical activations, gradients and
    variables to the same step with every op on one stream, over several steps in a row."""
    net = make()
    net.lr = 1e-6
    inp = W.make_inputs(net, seed=3)
    one, two = Replica(net, inp), Replica(net, inp)
    for r in range(3):
        one.step(concurrent=False)
        two.step(concurrent=True)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(two.params).all()), r
        assert bitwise_equal(one.grads, two.grads), r
        assert bitwise_equal(one.params, two.params), r
        for t in one.act:
            assert bitwise_equal(one.act[t], two.act[t]), (r, t)


@pytest.mark.parametrize("make", [lambda: W.googlenet(), lambda: W.inception_v3()],
                         ids=["googlenet_b128", "inception_v3_b32"])
def test_full_size_lanes_match_one_stream(make):
    """At the benchmarked sizes, two steps with the forward and backward branches on the lane
    streams -- the first recorded into a program, the second issued from it -- must give the
    same bits as two steps with every op on one stream, from the same variables."""
    net = make()
    net.lr = 1e-6
    rep = Replica(net, W.make_inputs(net, seed=6))
    snap = rep.snapshot()
    for _ in range(2):
        rep.step(concurrent=False)
    torch.cuda.synchronize()
    p1, g1 = rep.params.clone(), rep.grads.clone()
    a1 = {t: v.clone() for t, v in rep.act.items()}
    rep.restore(snap)
    prog = rep.record_step()
    rep.run_program(prog)
    torch.cuda.synchronize()
    say("lanes", net.name, "recorded calls:", len(prog))
    assert bool(torch.isfinite(rep.params).all())
    assert bitwise_equal(g1, rep.grads) and bitwise_equal(p1, rep.params)
    for t, v in a1.items():
        assert bitwise_equal(v, rep.act[t]), t
    prog.close()


@pytest.mark.parametrize("make", [lambda: W.alexnet(batch=8), lambda: W.googlenet(batch=4)],
                         ids=["alexnet_b8", "googlenet_b4"])
def test_graph_capture_replays_match_eager(make):
    """The whole step captured once in a HIP graph; every replay (with eager steps and
    synchronisations in between) must equal the eager step from the same state.  (A network
    with branches runs its forward and backward passes without the lane streams under capture;
    its eager steps use them.)"""
    net = make()
    net.lr = 1e-6            # keep the linear surrogate loss from driving values to inf
    inp = W.make_inputs(net, seed=2)
    eager = Replica(net, inp)
    graphed = Replica(net, inp)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        graphed.step()                     # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    eager.step()
    torch.cuda.synchronize()
    assert bitwise_equal(eager.params, graphed.params)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.step()
    for r in range(3):
        eager.step()
        g.replay()
        torch.cuda.synchronize()
        assert bool(torch.isfinite(eager.params).all()), r
        assert bitwise_equal(eager.params, graphed.params), r
        assert bitwise_equal(eager.grads, graphed.grads), r
        _ = torch.ones(1024, device="cuda").sum().item()      # unrelated eager work between replays


@pytest.mark.parametrize("make,opt", [(lambda: W.alexnet(batch=8), "sgd"), (lambda: W.googlenet(batch=4), "sgd"),
                                      (lambda: W.inception_v3(batch=2), "sgd"),
                                      (lambda: W.alexnet(batch=8), "momentum"), (lambda: W.alexnet(batch=8), "adam")],
                         ids=["alexnet_b8_sgd", "googlenet_b4_sgd", "inception_v3_b2_sgd", "alexnet_b8_momentum",
                              "alexnet_b8_adam"])
def test_program_replays_match_eager(make, opt):
    """The step recorded once into a native program (its library calls, stream joins included)
    and issued again from C++: every replay, with eager steps and synchronisations in between,
    must equal the eager two-stream step from the same state (the Adam update, whose step count
    changes, runs eagerly after the recorded calls)."""
    net = make()
    net.lr = 1e-6
    inp = W.make_inputs(net, seed=4)
    eager, prog_rep = Replica(net, inp, optimizer=opt), Replica(net, inp, optimizer=opt)
    eager.step()
    prog = prog_rep.record_step()
    torch.cuda.synchronize()
    say("program", net.name, opt, "recorded calls:", len(prog))
    assert len(prog) > len(net.ops)
    assert bitwise_equal(eager.params, prog_rep.params)
    for r in range(3):
        eager.step()
        prog_rep.run_program(prog)
        torch.cuda.synchronize()
        assert eager.t == prog_rep.t, r
        assert bool(torch.isfinite(prog_rep.params).all()), r
        assert bitwise_equal(eager.grads, prog_rep.grads), r
        assert bitwise_equal(eager.params, prog_rep.params), r
        for a, b in zip(eager.slots, prog_rep.slots):
            assert bitwise_equal(a, b), r
        _ = torch.ones(1024, device="cuda").sum().item()      # unrelated eager work between replays
    prog.close()


@pytest.mark.parametrize("make", [lambda: W.alexnet(batch=8), lambda: W.googlenet(batch=4),
                                  lambda: W.alexnet(batch=4, classifier=True)],
                         ids=["alexnet_b8", "googlenet_b4", "alexnet_cls_b4"])
def test_deferred_bias_gradients_match_immediate(make):
    """The untraced step leaves every main-stream bias gradient's partials in a workspace of its
    own and sums them all in one launch before the update; it must equal, bit for bit, the step
    that sums each one as it is formed (the same per-channel order), over two steps."""
    net = make()
    net.lr = 1e-6
    inp = W.make_inputs(net, seed=8)
    a, b = Replica(net, inp), Replica(net, inp)
    b.defer_bias = False
    for r in range(2):
        a.step()
        b.step()
        torch.cuda.synchronize()
        assert len(a.bias_ws) > 0 and len(b.bias_ws) == 0
        assert bitwise_equal(a.grads, b.grads), r
        assert bitwise_equal(a.params, b.params), r
    say("deferred bias gradients", net.name, "workspaces:", len(a.bias_ws))
