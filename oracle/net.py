"""Oracle composition of one synchronous SGD step of a convnet replica (fp64, CPU).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The step follows the paper's synchronous-replica semantics (Section 4.4): every
gradient is computed from the same pre-update parameters, and only after the
whole backward pass is every variable updated with W' = W - alpha * dL/dW
(Section 4.1).  Backward visits the ops in reverse order and sums the partial
gradients that reach a tensor along different paths (Section 4.1); no
gradient is formed for the step input unless the workload asks for it.

The surrogate loss is L = <g, out>, so the upstream gradient of the net's
output tensor is the given ``g``.  A classifier net (``net.loss ==
"softmax_xent"``) instead ends in logits and its loss is the batch mean of the
softmax cross-entropy against ``labels``; the upstream gradient of the logits
is then (softmax - onehot) / N.

``net`` is a plain description: ``net.ops`` in forward order, each op carrying
``name, src, dst, dst_c0, kh, kw, sh, sw, pads`` and, for convolutions,
``cout`` and ``relu``; ``net.tensors`` maps names to NHWC shapes; ``net.output``
names the output tensor.  Every convolution is followed by bias-add and, unless
its ``relu`` is false (a classifier's logits), ReLU.
"""
from __future__ import annotations

import numpy as np

from . import (apply_sgd, bias_relu_bwd, bias_relu_fwd, conv2d_bwd_filter, conv2d_bwd_input,
               conv2d_fwd, maxpool_bwd, maxpool_fwd, softmax_xent)


def _is_conv(op):
    return hasattr(op, "cout")


def forward(net, x, weights, biases):
    """Runs the forward pass; returns (activations by tensor name, argmax by pool name)."""
    acts = {"x": np.asarray(x, dtype=np.float64)}
    for name, shape in net.tensors.items():
        if name != "x":
            acts[name] = np.zeros(shape)
    argmax = {}
    for op in net.ops:
        src = acts[op.src]
        if _is_conv(op):
            pre = conv2d_fwd(src, weights[op.name], (op.sh, op.sw), op.pads)
            if getattr(op, "relu", True):
                out = bias_relu_fwd(pre, biases[op.name])
            else:
                out = pre + np.asarray(biases[op.name], dtype=np.float64)
        else:
            out, am = maxpool_fwd(src, (op.kh, op.kw), (op.sh, op.sw), op.pads)
            argmax[op.name] = am
        acts[op.dst][..., op.dst_c0:op.dst_c0 + out.shape[-1]] = out
    return acts, argmax


def backward(net, acts, argmax, weights, g):
    """Reverse pass from dL/d(out) = g; returns (grads by tensor, dW, db)."""
    grads = {net.output: np.asarray(g, dtype=np.float64)}
    dW, db = {}, {}

    def accumulate(name, d):
        if name in grads:
            grads[name] = grads[name] + d
        else:
            grads[name] = d

    for op in reversed(net.ops):
        if op.dst not in grads:
            continue
        width = op.cout if _is_conv(op) else net.tensors[op.src][3]
        dy = grads[op.dst][..., op.dst_c0:op.dst_c0 + width]
        src = acts[op.src]
        if _is_conv(op):
            y = acts[op.dst][..., op.dst_c0:op.dst_c0 + width]
            if getattr(op, "relu", True):
                dpre, db[op.name] = bias_relu_bwd(y, dy)
            else:
                dpre, db[op.name] = dy, dy.sum(axis=(0, 1, 2))
            dW[op.name] = conv2d_bwd_filter(src, dpre, (op.kh, op.kw), (op.sh, op.sw), op.pads)
            if op.src != "x" or net.input_grad:
                dx = conv2d_bwd_input(dpre, weights[op.name], src.shape, (op.sh, op.sw), op.pads)
                accumulate(op.src, dx)
        else:
            dx = maxpool_bwd(dy, argmax[op.name], src.shape)
            if op.src != "x" or net.input_grad:
                accumulate(op.src, dx)
    return grads, dW, db


def classifier_loss(net, acts, labels):
    """Batch-mean softmax cross-entropy of the logits and its gradient (N, 1, 1, C)."""
    out = acts[net.output]
    n = out.shape[0]
    rows, dz = softmax_xent(out.reshape(n, -1), labels, 1.0 / n)
    return float(np.mean(rows)), dz.reshape(out.shape)


def step(net, x, weights, biases, g, lr=None, labels=None):
    """One SGD step.  Returns a dict with acts, argmax, grads, dW, db, new_weights, new_biases
    (and, for a classifier, loss)."""
    # The learning rate is an fp32 attribute of the update op: use its fp32 value.
    lr = float(np.float32(net.lr if lr is None else lr))
    acts, argmax = forward(net, x, weights, biases)
    value = None
    if net.loss == "softmax_xent":
        value, g = classifier_loss(net, acts, labels)
    grads, dW, db = backward(net, acts, argmax, weights, g)
    new_w = {k: apply_sgd(weights[k], dW[k], lr) for k in dW}
    new_b = {k: apply_sgd(biases[k], db[k], lr) for k in db}
    return dict(acts=acts, argmax=argmax, grads=grads, dW=dW, db=db,
                new_weights=new_w, new_biases=new_b, loss=value)


def loss(net, x, weights, biases, g, labels=None):
    """The loss of the forward pass: <g, out>, or a classifier's mean cross-entropy."""
    acts, _ = forward(net, x, weights, biases)
    if net.loss == "softmax_xent":
        return classifier_loss(net, acts, labels)[0]
    return float(np.sum(np.asarray(g, dtype=np.float64) * acts[net.output]))
