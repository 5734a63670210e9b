"""Sampled softmax on the GPU against the CPU oracle: the candidate gather, the candidate
cross-entropy, the sparse row update, and a whole head step at a small and at a language-model
size."""
import numpy as np
import pytest
import torch

import oracle
from paper_1605_08695_amd import ops
from paper_1605_08695_amd import workloads as W
from paper_1605_08695_amd.sampled import SampledSoftmaxHead
from tests.gpu_parity import assert_close, err, f64, rel_l2, say, ulp_diff_f32

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_gather_rows_t_exact(dt):
    rng = np.random.default_rng(90)
    table = torch.from_numpy(rng.standard_normal((300, 24))).to(dt).to(DEV)
    idx_np = rng.permutation(300)[:37].astype(np.int32)
    idx_np[5] = 300                                            # out of range: a zero column
    out = ops.gather_rows_t(table, torch.from_numpy(idx_np).to(DEV), 64)
    torch.cuda.synchronize()
    ref = np.zeros((24, 64))
    t = f64(table)
    for j, r in enumerate(idx_np):
        if 0 <= r < 300:
            ref[:, j] = t[r]
    assert np.array_equal(f64(out), ref)


def _candidate_case(rng, n, m, extra, dt):
    """Candidate logits z (n x u) with the sample in the first m columns and `extra` more true
    classes; labels drawn over all candidates (accidental hits included)."""
    u = m + extra
    cls = rng.permutation(5 * u)[:u].astype(np.int32)        # class ids of the candidates
    true_pos = rng.integers(0, u, size=n).astype(np.int32)
    true_pos[:extra] = m + np.arange(extra)                    # every extra column is somebody's class
    z = rng.standard_normal((n, u)) * 2
    bc = rng.standard_normal(u) * 0.1
    lq = rng.standard_normal(u) * 0.5 - 3                      # log expected count per candidate
    return u, cls, true_pos, z, bc, lq


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("n,m,extra", [(1, 1, 0), (37, 20, 9), (256, 512, 130)], ids=["tiny", "ragged", "lm"])
def test_sampled_softmax_xent(n, m, extra, dt):
    """Against the oracle's sampled softmax with W[cls[j]] = e_j and h = z: the candidate logits
    are then exactly z, and the oracle's dh is the gradient of the logits in candidate order."""
    say("sampled xent", n, m, extra, dt)
    rng = np.random.default_rng(91 + n)
    u, cls, true_pos, z, bc, lq = _candidate_case(rng, n, m, extra, dt)
    u_pad = (u + 63) // 64 * 64
    zt = torch.zeros(n, u_pad, dtype=dt)
    zt[:, :u] = torch.from_numpy(z).to(dt)
    zq = f64(zt)[:, :u]                                         # the values the kernel reads
    bct = torch.zeros(u_pad, dtype=torch.float32)
    bct[:u] = torch.from_numpy(bc).float()
    lq32 = lq.astype(np.float32)
    loss, dz = ops.sampled_softmax_xent(zt.to(DEV), u, m, torch.from_numpy(true_pos).to(DEV),
                                        torch.from_numpy(lq32[true_pos]).to(DEV), torch.from_numpy(lq32[:m]).to(DEV),
                                        1.0 / n, bias_c=bct.to(DEV))
    torch.cuda.synchronize()
    V = 5 * u
    Wv = np.zeros((V, u))
    Wv[cls, np.arange(u)] = 1.0
    bv = np.zeros(V)
    bv[cls] = f64(bct)[:u]
    r_loss, r_dh, _, _ = oracle.sampled_softmax(zq, Wv, bv, cls[true_pos], cls[:m], lq32[true_pos].astype(np.float64),
                                                lq32[:m].astype(np.float64), 1.0 / n)
    assert_close(f64(loss), r_loss, torch.float32, label="loss")
    assert_close(f64(dz)[:, :u], r_dh, dt, torch.float32, label="dz")
    assert np.all(f64(dz)[:, u:] == 0)


def test_scatter_apply_sgd_rows():
    rng = np.random.default_rng(92)
    var = torch.from_numpy(rng.standard_normal((500, 48)).astype(np.float32)).to(DEV)
    v0 = var.clone()
    sh = var.to(torch.bfloat16)
    idx_np = rng.permutation(500)[:70].astype(np.int32)
    g = torch.from_numpy(rng.standard_normal((48, 80)).astype(np.float32)).to(DEV)    # ld 80 > u
    ops.scatter_apply_sgd(var, torch.from_numpy(idx_np).to(DEV), g, 0.05, shadow=sh)
    torch.cuda.synchronize()
    ref = f64(v0)
    gg = f64(g)
    lr = float(np.float32(0.05))
    for j, r in enumerate(idx_np):
        ref[r] = oracle.apply_sgd(ref[r], gg[:, j], lr)
    assert ulp_diff_f32(var.cpu().numpy(), ref) <= 1
    touched = np.zeros(500, bool)
    touched[idx_np] = True
    assert torch.equal(var[torch.from_numpy(~touched).to(DEV)], v0[torch.from_numpy(~touched).to(DEV)])
    assert torch.equal(sh[torch.from_numpy(touched).to(DEV)], var[torch.from_numpy(touched).to(DEV)].to(torch.bfloat16))


@pytest.mark.parametrize("n,d,vocab,m", [(48, 64, 700, 60), (512, 512, 40000, 512)], ids=["small", "lm"])
def test_sampled_softmax_head_step(n, d, vocab, m):
    """A whole head step (gather, candidate GEMM, cross-entropy, gradients, sparse update) against
    the oracle on the same bf16-rounded inputs.  The candidate logits are stored in bf16, so the
    loss and gradients carry bf16-level error: rel_l2 and err bars of the bf16 path."""
    say("sampled head step", n, d, vocab, m)
    inp = W.make_sampled_inputs(n, d, vocab, m, seed=5)
    head = SampledSoftmaxHead(inp.W, inp.b, lr=0.1)
    h = torch.from_numpy(inp.h).to(torch.bfloat16).to(DEV)
    W0 = f64(head.W)
    b0 = f64(head.b)
    loss, dh = head.step(h, inp.labels, inp.sampled, inp.lq_true, inp.lq_sampled)
    torch.cuda.synchronize()
    lq_t = inp.lq_true.astype(np.float32).astype(np.float64)
    lq_s = inp.lq_sampled.astype(np.float32).astype(np.float64)
    r_loss, r_dh, r_dW, r_db = oracle.sampled_softmax(f64(h), W0, b0, inp.labels, inp.sampled, lq_t, lq_s, 1.0 / n)
    e = {"loss": err(f64(loss), r_loss), "dh_rel_l2": rel_l2(f64(dh), r_dh),
         "dW_rel_l2": rel_l2(W0 - f64(head.W), head.lr * r_dW), "db_rel_l2": rel_l2(b0 - f64(head.b), head.lr * r_db)}
    say("  ", {k: "%.2e" % v for k, v in e.items()})
    assert e["loss"] <= 2e-2 and all(v <= 2e-2 for k, v in e.items() if k != "loss"), e
    # rows outside the candidates are untouched, bit for bit
    cand, _ = SampledSoftmaxHead.candidates(inp.labels, inp.sampled)
    other = np.ones(vocab, bool)
    other[cand] = False
    assert np.array_equal(f64(head.W)[other], W0[other]) and np.array_equal(f64(head.b)[other], b0[other])
    assert torch.equal(head.W_lp, head.W.to(torch.bfloat16))
