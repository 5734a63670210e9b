"""Sampled-softmax classifier head: one training step over a large class set (Section 4.2's sampled
softmax, evaluated on a language model in Section 6.4).

The head multiplies its input h (n x d) only by the weight rows of the candidates: the shared
sample of m classes (drawn on the host from a proposal Q, with the log of each class's expected
count) and the examples' true classes.  Every step of the computation runs in the library's
kernels; the host only lists the distinct candidates (sample first) and each example's candidate
column, and uploads them with the draws.
"""
from __future__ import annotations

import numpy as np
import torch

from . import ops


def _round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


class SampledSoftmaxHead:
    """Variables W (vocab x d, fp32 master + bf16 shadow) and b (vocab, fp32) of a softmax
    classifier, trained by the sampled softmax with SGD on the candidate rows only."""

    def __init__(self, W: np.ndarray, b: np.ndarray, lr: float, device="cuda"):
        dev = torch.device(device)
        self.vocab, self.d = W.shape
        self.lr = float(np.float32(lr))
        # master weights start at their bf16 values (the values the GEMMs read)
        self.W = torch.from_numpy(np.asarray(W, np.float32)).to(torch.bfloat16).to(torch.float32).to(dev)
        self.W_lp = self.W.to(torch.bfloat16)
        self.b = torch.from_numpy(np.asarray(b, np.float32)).to(dev)
        self.device = dev

    @staticmethod
    def candidates(labels: np.ndarray, sampled: np.ndarray):
        """Distinct candidate classes (the sample first, then true classes outside it, in order of
        first appearance) and the candidate column of each example's true class."""
        pos = {int(c): j for j, c in enumerate(sampled)}
        cand = [int(c) for c in sampled]
        for t in labels:
            if int(t) not in pos:
                pos[int(t)] = len(cand)
                cand.append(int(t))
        true_pos = np.array([pos[int(t)] for t in labels], np.int32)
        return np.asarray(cand, np.int32), true_pos

    def prepare(self, labels: np.ndarray, sampled: np.ndarray, lq_true: np.ndarray, lq_sampled: np.ndarray):
        """Host side of a step: the candidate list and columns, uploaded with the draws."""
        dev = self.device
        cand, true_pos = self.candidates(labels, sampled)
        up = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(dev)
        return dict(n=labels.size, u=cand.size, m=sampled.size, u_pad=_round_up(cand.size, 64),
                    cand=up(cand, np.int32), true_pos=up(true_pos, np.int32), lq_true=up(lq_true, np.float32),
                    lq_sampled=up(lq_sampled, np.float32))

    def run(self, h: torch.Tensor, bt: dict, stream=None):
        """Device side of a step on h (n x d, bf16): returns (loss per row, dh).  W and b are
        updated in place on the candidate rows."""
        n, d = h.shape
        u, m, u_pad, cand = bt["u"], bt["m"], bt["u_pad"], bt["cand"]
        # candidate weights as a d x u_pad filter, candidate biases
        wc = ops.gather_rows_t(self.W_lp, cand, u_pad, stream=stream)
        bc = ops.gather_rows_t(self.b.view(-1, 1), cand, u_pad, stream=stream).view(-1)
        h4 = h.view(n, 1, 1, d)
        w4 = wc.view(1, 1, d, u_pad)
        z = ops.conv2d_fwd(h4, w4, 1, (0, 0, 0, 0), stream=stream)
        loss, dz = ops.sampled_softmax_xent(z, u, m, bt["true_pos"], bt["lq_true"], bt["lq_sampled"], 1.0 / n,
                                            bias_c=bc, stream=stream)
        _, dbc = ops.bias_relu_bwd(None, dz, dpre=dz, stream=stream)
        dwc = ops._empty(stream, (1, 1, d, u_pad), dtype=torch.float32, device=h.device)
        ops.conv2d_bwd_filter(h4, dz, (1, 1), 1, (0, 0, 0, 0), dw=dwc, stream=stream)
        dh = ops._empty_like(stream, h4)
        ops.conv2d_bwd_input(dz, w4, dh, 1, (0, 0, 0, 0), stream=stream)
        ops.scatter_apply_sgd(self.W, cand, dwc.view(d, u_pad), self.lr, shadow=self.W_lp, stream=stream)
        ops.scatter_apply_sgd(self.b, cand, dbc.view(1, u_pad), self.lr, stream=stream)
        return loss, dh.view(n, d)

    def step(self, h: torch.Tensor, labels: np.ndarray, sampled: np.ndarray, lq_true: np.ndarray,
             lq_sampled: np.ndarray, stream=None):
        """One step: prepare() then run()."""
        return self.run(h, self.prepare(labels, sampled, lq_true, lq_sampled), stream)


class FullSoftmaxHead:
    """The same classifier trained with the full softmax, for comparison: W stored d x vocab (the
    filter of a 1 x 1 convolution), logits over every class, dense SGD."""

    def __init__(self, W: np.ndarray, b: np.ndarray, lr: float, device="cuda"):
        dev = torch.device(device)
        self.vocab, self.d = W.shape
        self.lr = float(np.float32(lr))
        Wt = np.ascontiguousarray(np.asarray(W, np.float32).T)
        self.W = torch.from_numpy(Wt).to(torch.bfloat16).to(torch.float32).to(dev)
        self.W_lp = self.W.to(torch.bfloat16)
        self.b = torch.from_numpy(np.asarray(b, np.float32)).to(dev)

    def run(self, h: torch.Tensor, labels: torch.Tensor, stream=None):
        n, d = h.shape
        h4 = h.view(n, 1, 1, d)
        w4 = self.W_lp.view(1, 1, d, self.vocab)
        z = ops.conv2d_fwd(h4, w4, 1, (0, 0, 0, 0), stream=stream)
        loss, dz = ops.softmax_xent(z, labels, 1.0 / n, bias=self.b, dlogits=z, stream=stream)
        _, db = ops.bias_relu_bwd(None, dz, dpre=dz, stream=stream)
        dw = ops._empty(stream, (1, 1, d, self.vocab), dtype=torch.float32, device=h.device)
        ops.conv2d_bwd_filter(h4, dz, (1, 1), 1, (0, 0, 0, 0), dw=dw, stream=stream)
        dh = ops._empty_like(stream, h4)
        ops.conv2d_bwd_input(dz, w4, dh, 1, (0, 0, 0, 0), stream=stream)
        ops.apply_sgd(self.W.view(-1), dw.view(-1), self.lr, shadow=self.W_lp.view(-1), stream=stream)
        ops.apply_sgd(self.b, db, self.lr, stream=stream)
        return loss, dh.view(n, d)
