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


U_BF16 = 2.0 ** -8          # unit roundoff of bf16 (round to nearest even, 8-bit significand)
U_F32 = 2.0 ** -24


def _head_error_bounds(h, Wc, bc, lq_true, lq_sampled, true_pos, m, scale):
    """Per-element bounds of what the head's bf16 storage of the candidate logits and of their
    gradient allows, given exact (fp64) arithmetic elsewhere and fp32 sums.

    With logits z_i stored in bf16, each moves by at most E_i = u max_j |z_ij| (u = 2^-8), so the
    softmax p_ij moves by at most p_ij (exp(2 E_i) - 1) and the loss by at most 2 E_i (the
    log-sum-exp is 1-Lipschitz in the max norm).  The stored gradient dz_ij = scale (p_ij -
    [j = true]) then errs by at most e_ij = scale p_ij k_i + u (|dz_ij| + scale p_ij k_i), k_i =
    exp(2 E_i) - 1.  Returns (e, k-independent loss bound, |dz|)."""
    n, u = h.shape[0], Wc.shape[0]
    z = h @ Wc.T + bc[None, :]
    lq = np.broadcast_to(np.concatenate([lq_sampled, np.zeros(u - m)])[None, :], (n, u)).copy()
    rows = np.arange(n)
    lq[rows, true_pos] = lq_true
    z = z - lq
    keep = np.zeros((n, u), bool)
    keep[:, :m] = True
    keep[rows, true_pos] = True          # the true column (an accidental hit is this same column)
    z = np.where(keep, z, -np.inf)
    mx = z.max(axis=1, keepdims=True)
    p = np.exp(z - mx)
    p /= p.sum(axis=1, keepdims=True)
    # + the fp32 sums of the candidate GEMM and of the bias and log-count terms
    gemm = h.shape[1] * U_F32 * np.max(np.abs(h) @ np.abs(Wc).T, axis=1)
    E = (U_BF16 * np.max(np.where(keep, np.abs(z), 0.0), axis=1) + gemm
         + 4 * U_F32 * (np.max(np.where(keep, np.abs(z), 0.0), axis=1) + np.max(np.abs(lq), axis=1) + 1))
    k = np.expm1(2 * E)[:, None]
    dz = scale * (p - (np.arange(u)[None, :] == true_pos[:, None]))
    e = scale * p * k + U_BF16 * (np.abs(dz) + scale * p * k)
    return e, 2 * E, np.abs(dz)


def _assert_within(name, a, r, tol):
    excess = np.abs(a - r) - tol
    worst = float(np.max(excess / np.maximum(tol, 1e-300))) if a.size else 0.0
    say("  %-10s max|a-r| %.3e  max tol %.3e  worst (|a-r|-tol)/tol %.3f" % (name, float(np.max(np.abs(a - r))),
                                                                          float(np.max(tol)), worst))
    assert np.all(excess <= 0), (name, int(np.sum(excess > 0)))


@pytest.mark.parametrize("n,d,vocab,m", [(48, 64, 700, 60), (512, 512, 40000, 512)], ids=["small", "lm"])
def test_sampled_softmax_head_step(n, d, vocab, m):
    """A whole head step (gather, candidate GEMM, cross-entropy, gradients, sparse update) against
    the oracle on the same bf16-rounded inputs, element by element.  The head stores the candidate
    logits and their gradient in bf16, so every element of the loss, dh and the two updates is
    held to the bound that this storage allows (_head_error_bounds), plus the fp32 rounding of
    the sums and of the update."""
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
    scale = 1.0 / n
    r_loss, r_dh, r_dW, r_db = oracle.sampled_softmax(f64(h), W0, b0, inp.labels, inp.sampled, lq_t, lq_s, scale)
    e = {"loss": err(f64(loss), r_loss), "dh_rel_l2": rel_l2(f64(dh), r_dh),
         "dW_rel_l2": rel_l2(W0 - f64(head.W), head.lr * r_dW), "db_rel_l2": rel_l2(b0 - f64(head.b), head.lr * r_db)}
    say("  ", {k: "%.2e" % v for k, v in e.items()})
    assert e["loss"] <= 2e-2 and all(v <= 2e-2 for k, v in e.items() if k != "loss"), e
    # element by element, against the bounds of the bf16 storage of the logits and their gradient
    cand, true_pos = SampledSoftmaxHead.candidates(inp.labels, inp.sampled)
    hh, Wc, bc = f64(h), W0[cand], b0[cand]
    lr = head.lr
    eb, loss_tol, adz = _head_error_bounds(hh, Wc, bc, lq_t, lq_s, true_pos, m, scale)
    u = cand.size
    _assert_within("loss", f64(loss), r_loss, loss_tol + 8 * U_F32 * (np.abs(r_loss) + u))
    dh_err = eb @ np.abs(Wc) + u * U_F32 * (adz @ np.abs(Wc))
    _assert_within("dh", f64(dh), r_dh, dh_err + U_BF16 * (np.abs(r_dh) + dh_err))
    # candidate rows of the updated variables: W0 - W1 = lr dW up to the fp32 rounding of W1
    W1, b1 = f64(head.W)[cand], f64(head.b)[cand]
    dW_err = eb.T @ np.abs(hh) + n * U_F32 * (adz.T @ np.abs(hh))
    _assert_within("dW", Wc - W1, lr * r_dW[cand], lr * dW_err + U_F32 * (np.abs(W1) + np.abs(Wc)))
    db_err = eb.sum(axis=0) + n * U_F32 * adz.sum(axis=0)
    _assert_within("db", bc - b1, lr * r_db[cand], lr * db_err + U_F32 * (np.abs(b1) + np.abs(bc)))
    # rows outside the candidates are untouched, bit for bit
    other = np.ones(vocab, bool)
    other[cand] = False
    assert np.array_equal(f64(head.W)[other], W0[other]) and np.array_equal(f64(head.b)[other], b0[other])
    assert torch.equal(head.W_lp, head.W.to(torch.bfloat16))
