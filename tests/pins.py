"""Independent checks that pin the CPU oracle to the mathematics.

Each ``check_*`` returns an error figure (0 for a perfect match).  The pin
tests assert it is tiny; the mutation tests build the oracle with a planted
mistake and assert the same check then fails.  None of these re-types the
oracle's loop nests: they use a library convolution, matmul, finite
differences of a scalar loss, adjoint identities, closed forms or brute-force
numpy window scans.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F

import oracle
from oracle import net as onet


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    s = max(np.max(np.abs(b)), 1e-300)
    return float(np.max(np.abs(a - b)) / s)


def torch_conv(x, w, stride, pads):
    """Library reference: torch float64 CPU conv2d (cross-correlation) with explicit pads."""
    pt, pb, pl, pr = pads
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2)))
    xt = F.pad(xt, (pl, pr, pt, pb))
    wt = torch.from_numpy(np.ascontiguousarray(w.transpose(3, 2, 0, 1)))
    y = F.conv2d(xt, wt, stride=stride)
    return y.numpy().transpose(0, 2, 3, 1)


def random_conv_case(rng, max_hw=9):
    N = int(rng.integers(1, 3))
    C = int(rng.integers(1, 5))
    K = int(rng.integers(1, 5))
    KH = int(rng.integers(1, 6))
    KW = int(rng.integers(1, 6))
    s = (int(rng.integers(1, 4)), int(rng.integers(1, 4)))
    pads = (int(rng.integers(0, KH)), int(rng.integers(0, KH)),
            int(rng.integers(0, KW)), int(rng.integers(0, KW)))
    H = int(rng.integers(max(1, KH - pads[0] - pads[1]), max_hw + 1))
    W = int(rng.integers(max(1, KW - pads[2] - pads[3]), max_hw + 1))
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((KH, KW, C, K))
    return x, w, s, pads


# ----------------------------------------------------------------------------- conv
def check_conv_vs_torch(seed=0, cases=40):
    rng = np.random.default_rng(seed)
    worst = 0.0
    for _ in range(cases):
        x, w, s, pads = random_conv_case(rng)
        worst = max(worst, rel(oracle.conv2d_fwd(x, w, s, pads), torch_conv(x, w, s, pads)))
    return worst


def check_shifted_delta(p=1):
    """A single 1 at tap (0,0) with pad p copies x shifted by p: y[oh,ow] = x[oh-p, ow-p]."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 6, 7, 3))
    w = np.zeros((3, 3, 3, 3))
    for c in range(3):
        w[0, 0, c, c] = 1.0
    y = oracle.conv2d_fwd(x, w, 1, (p, p, p, p))
    OH, OW = y.shape[1:3]
    ref = np.zeros_like(y)
    for oh in range(OH):
        for ow in range(OW):
            ih, iw = oh - p, ow - p
            if 0 <= ih < x.shape[1] and 0 <= iw < x.shape[2]:
                ref[:, oh, ow, :] = x[:, ih, iw, :]
    return rel(y, ref)


def check_delta_identity(k=3):
    """Centre-tap identity kernel with SAME padding: y == x and bwd_input(g) == g exactly."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 5, 6, 4))
    w = np.zeros((k, k, 4, 4))
    for c in range(4):
        w[k // 2, k // 2, c, c] = 1.0
    p = k // 2
    y = oracle.conv2d_fwd(x, w, 1, (p, p, p, p))
    g = rng.standard_normal(y.shape)
    dx = oracle.conv2d_bwd_input(g, w, x.shape, 1, (p, p, p, p))
    return max(float(np.max(np.abs(y - x))), float(np.max(np.abs(dx - g))))


def check_one_by_one_is_matmul():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 5, 4, 7))
    w = rng.standard_normal((1, 1, 7, 6))
    y = oracle.conv2d_fwd(x, w, 1, (0, 0, 0, 0))
    ref = np.matmul(x.reshape(-1, 7), w.reshape(7, 6)).reshape(2, 5, 4, 6)
    return rel(y, ref)


def check_full_window_is_fc():
    """A VALID conv whose window is the whole image is a fully connected layer (matmul),
    and its filter gradient is the outer product x_flat^T @ dy."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 4, 5, 2))
    w = rng.standard_normal((4, 5, 2, 6))
    y = oracle.conv2d_fwd(x, w, 1, (0, 0, 0, 0))
    e1 = rel(y.reshape(3, 6), x.reshape(3, -1) @ w.reshape(-1, 6))
    dy = rng.standard_normal((3, 1, 1, 6))
    dw = oracle.conv2d_bwd_filter(x, dy, (4, 5), 1, (0, 0, 0, 0))
    e2 = rel(dw.reshape(-1, 6), x.reshape(3, -1).T @ dy.reshape(3, 6))
    dx = oracle.conv2d_bwd_input(dy, w, x.shape, 1, (0, 0, 0, 0))
    e3 = rel(dx.reshape(3, -1), dy.reshape(3, 6) @ w.reshape(-1, 6).T)
    return max(e1, e2, e3)


def check_all_ones_closed_form():
    """x = 1, w = 1: y[oh,ow] = Cin * (in-bounds rows of the window) * (in-bounds cols)."""
    worst = 0.0
    for (H, W, KH, KW, s, pads) in [(7, 6, 3, 3, 1, (1, 1, 1, 1)), (8, 9, 4, 2, 2, (3, 0, 1, 1)),
                                    (5, 5, 5, 5, 3, (2, 2, 4, 1))]:
        C = 3
        x = np.ones((1, H, W, C))
        w = np.ones((KH, KW, C, 2))
        y = oracle.conv2d_fwd(x, w, s, pads)
        OH, OW = y.shape[1:3]
        ref = np.zeros((OH, OW))
        for oh in range(OH):
            r0 = oh * s - pads[0]
            rows = min(H, r0 + KH) - max(0, r0)
            for ow in range(OW):
                c0 = ow * s - pads[2]
                cols = min(W, c0 + KW) - max(0, c0)
                ref[oh, ow] = C * max(rows, 0) * max(cols, 0)
        worst = max(worst, float(np.max(np.abs(y[0, :, :, 0] - ref))),
                    float(np.max(np.abs(y[0, :, :, 1] - ref))))
    return worst


def check_adjoints(seed=5, cases=40):
    """<conv(x,w), g> = <x, bwd_input(g,w)> = <w, bwd_filter(x,g)>, strides 1-4, any pad split."""
    rng = np.random.default_rng(seed)
    worst = 0.0
    for i in range(cases):
        x, w, _, pads = random_conv_case(rng)
        s = (1 + i % 4, 1 + (i // 4) % 4)
        H, W = x.shape[1:3]
        if oracle.out_len(H, w.shape[0], s[0], pads[0], pads[1]) < 1 or \
           oracle.out_len(W, w.shape[1], s[1], pads[2], pads[3]) < 1:
            continue
        y = oracle.conv2d_fwd(x, w, s, pads)
        g = rng.standard_normal(y.shape)
        lhs = float(np.sum(y * g))
        dx = oracle.conv2d_bwd_input(g, w, x.shape, s, pads)
        dw = oracle.conv2d_bwd_filter(x, g, w.shape[:2], s, pads)
        scale = float(np.sum(np.abs(y * g))) + 1e-300
        worst = max(worst, abs(lhs - float(np.sum(x * dx))) / scale,
                    abs(lhs - float(np.sum(w * dw))) / scale)
    return worst


def check_unused_rows_get_zero():
    """VALID 3x3/2 on H = 8: windows cover rows 0-6, so dx row 7 (and column 7) is 0."""
    rng = np.random.default_rng(6)
    x_shape = (1, 8, 8, 2)
    w = rng.standard_normal((3, 3, 2, 3))
    g = rng.standard_normal((1, 3, 3, 3))
    dx = oracle.conv2d_bwd_input(g, w, x_shape, 2, (0, 0, 0, 0))
    return float(np.max(np.abs(dx[0, 7]))) + float(np.max(np.abs(dx[0, :, 7])))


def check_conv_fd(seed=7, samples=12):
    """Central differences of L = <g, conv(x,w)>: L is linear in x and in w, so the
    difference quotient has no truncation error; returns the worst relative error."""
    rng = np.random.default_rng(seed)
    worst = 0.0
    for case in range(6):
        x, w, s, pads = random_conv_case(rng, max_hw=7)
        y = oracle.conv2d_fwd(x, w, s, pads)
        g = rng.standard_normal(y.shape)
        dx = oracle.conv2d_bwd_input(g, w, x.shape, s, pads)
        dw = oracle.conv2d_bwd_filter(x, g, w.shape[:2], s, pads)

        def L(xx, ww):
            return float(np.sum(g * torch_conv(xx, ww, s, pads)))
        gscale = max(np.max(np.abs(dx)), np.max(np.abs(dw)), 1e-3)
        for _ in range(samples):
            h = 1e-3
            i = tuple(int(rng.integers(0, d)) for d in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[i] += h
            xm[i] -= h
            fd = (L(xp, w) - L(xm, w)) / (2 * h)
            worst = max(worst, abs(fd - dx[i]) / gscale)
            j = tuple(int(rng.integers(0, d)) for d in w.shape)
            wp, wm = w.copy(), w.copy()
            wp[j] += h
            wm[j] -= h
            fd = (L(x, wp) - L(x, wm)) / (2 * h)
            worst = max(worst, abs(fd - dw[j]) / gscale)
    return worst


def check_conv_bwd_vs_autograd(seed=15, cases=25):
    """Library pin: torch float64 autograd of conv2d gives dX and dW of <g, conv(x, w)>;
    also checks the sampled filter-gradient entry point at random entries."""
    rng = np.random.default_rng(seed)
    worst = 0.0
    for _ in range(cases):
        x, w, s, pads = random_conv_case(rng)
        y = torch_conv(x, w, s, pads)
        g = rng.standard_normal(y.shape)
        pt, pb, pl, pr = pads
        xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2))).requires_grad_(True)
        wt = torch.from_numpy(np.ascontiguousarray(w.transpose(3, 2, 0, 1))).requires_grad_(True)
        yt = F.conv2d(F.pad(xt, (pl, pr, pt, pb)), wt, stride=s)
        (yt * torch.from_numpy(np.ascontiguousarray(g.transpose(0, 3, 1, 2)))).sum().backward()
        dx_ref = xt.grad.numpy().transpose(0, 2, 3, 1)
        dw_ref = wt.grad.numpy().transpose(2, 3, 1, 0)
        dx = oracle.conv2d_bwd_input(g, w, x.shape, s, pads)
        dw = oracle.conv2d_bwd_filter(x, g, w.shape[:2], s, pads)
        idx = rng.integers(0, w.size, size=8)
        dw_at = oracle.conv2d_bwd_filter_at(x, g, w.shape[:2], s, pads, idx)
        worst = max(worst, rel(dx, dx_ref), rel(dw, dw_ref), rel(dw_at, dw_ref.ravel()[idx]))
    return worst


# ----------------------------------------------------------------------------- pool
def windows(x_shape, kh, kw, s, pads):
    """Brute-force window enumeration: for each output position, the in-bounds taps in
    (kh outer, kw inner) order as (h, w) pairs."""
    N, H, W, C = x_shape
    sh, sw = (s, s) if np.isscalar(s) else s
    OH = (H + pads[0] + pads[1] - kh) // sh + 1
    OW = (W + pads[2] + pads[3] - kw) // sw + 1
    out = {}
    for oh in range(OH):
        for ow in range(OW):
            taps = []
            for a in range(kh):
                for b in range(kw):
                    h, w = oh * sh + a - pads[0], ow * sw + b - pads[2]
                    if 0 <= h < H and 0 <= w < W:
                        taps.append((h, w))
            out[(oh, ow)] = taps
    return OH, OW, out


def brute_pool(x, kh, kw, s, pads):
    N, H, W, C = x.shape
    OH, OW, win = windows(x.shape, kh, kw, s, pads)
    y = np.zeros((N, OH, OW, C))
    am = np.zeros((N, OH, OW, C), dtype=np.int64)
    for (oh, ow), taps in win.items():
        vals = np.stack([x[:, h, w, :] for (h, w) in taps], axis=0)   # [T, N, C]
        k = np.argmax(vals, axis=0)                                   # first maximum
        y[:, oh, ow, :] = np.max(vals, axis=0)
        hs = np.array([t[0] for t in taps])[k]
        ws = np.array([t[1] for t in taps])[k]
        n_idx = np.arange(N)[:, None]
        c_idx = np.arange(C)[None, :]
        am[:, oh, ow, :] = ((n_idx * H + hs) * W + ws) * C + c_idx
    return y, am


def check_pool_bruteforce(seed=8):
    rng = np.random.default_rng(seed)
    worst = 0.0
    for (H, W, k, s, pads) in [(7, 7, 3, 2, (0, 0, 0, 0)), (6, 5, 3, 1, (1, 1, 1, 1)),
                               (8, 8, 2, 2, (0, 0, 0, 0)), (7, 9, 3, 2, (0, 1, 0, 1)),
                               (5, 6, 3, 3, (1, 2, 2, 1))]:
        for mode in ("normal", "ties"):
            x = rng.standard_normal((2, H, W, 3))
            if mode == "ties":
                x = np.round(x)            # many repeated values and exact zeros
                x[0] = 0.0                 # whole all-zero image: every window ties
            y, am = oracle.maxpool_fwd(x, (k, k), s, pads)
            yb, amb = brute_pool(x, k, k, s, pads)
            worst = max(worst, float(np.max(np.abs(y - yb))), float(np.sum(am != amb)))
    return worst


def check_pool_reshape_max():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 8, 6, 5))
    y, _ = oracle.maxpool_fwd(x, (2, 2), 2, (0, 0, 0, 0))
    ref = x.reshape(2, 4, 2, 3, 2, 5).max(axis=(2, 4))
    return rel(y, ref)


def check_pool_bwd(seed=10):
    """Mass conservation, support on argmax positions, and exact finite differences of
    <g, pool(x)> at tie-free points (max-pool is piecewise linear)."""
    rng = np.random.default_rng(seed)
    worst = 0.0
    for (H, W, k, s, pads) in [(7, 7, 3, 2, (0, 0, 0, 0)), (6, 5, 3, 1, (1, 1, 1, 1))]:
        x = rng.standard_normal((2, H, W, 3))
        y, am = oracle.maxpool_fwd(x, (k, k), s, pads)
        g = rng.standard_normal(y.shape)
        dx = oracle.maxpool_bwd(g, am, x.shape)
        worst = max(worst, abs(float(np.sum(dx)) - float(np.sum(g))) / float(np.sum(np.abs(g))))
        mask = np.zeros(x.size, dtype=bool)
        mask[am.ravel()] = True
        worst = max(worst, float(np.max(np.abs(dx.ravel()[~mask]), initial=0.0)))
        h = 1e-6
        for _ in range(10):
            i = tuple(int(rng.integers(0, d)) for d in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[i] += h
            xm[i] -= h
            fd = (float(np.sum(g * brute_pool(xp, k, k, s, pads)[0])) -
                  float(np.sum(g * brute_pool(xm, k, k, s, pads)[0]))) / (2 * h)
            worst = max(worst, abs(fd - dx[i]) / max(1.0, abs(dx[i])))
    return worst


def check_pool_bwd_beta():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((1, 5, 5, 2))
    y, am = oracle.maxpool_fwd(x, (3, 3), 2, (0, 0, 0, 0))
    g = rng.standard_normal(y.shape)
    base = rng.standard_normal(x.shape)
    d0 = oracle.maxpool_bwd(g, am, x.shape)
    d1 = oracle.maxpool_bwd(g, am, x.shape, dx=base, beta=1)
    return rel(d1, base + d0)


# ----------------------------------------------------------------------------- bias + relu
def check_bias_relu(seed=12):
    """FD of <g, relu(pre + b)> in pre and b away from the kink; db = numpy column sums;
    outputs at the kink are +0.0; the mask comes from the stored output."""
    rng = np.random.default_rng(seed)
    pre = rng.standard_normal((2, 3, 4, 5))
    b = rng.standard_normal(5)
    y = oracle.bias_relu_fwd(pre, b)
    worst = float(np.sum(np.signbit(y)))      # no -0.0 and no negatives
    g = rng.standard_normal(y.shape)
    dpre, db = oracle.bias_relu_bwd(y, g)
    worst = max(worst, rel(db, np.sum(dpre, axis=(0, 1, 2))))
    h = 1e-7

    def L(pp, bb):
        z = pp + bb
        return float(np.sum(g * np.where(z > 0, z, 0.0)))
    for _ in range(10):
        i = tuple(int(rng.integers(0, d)) for d in pre.shape)
        if abs(pre[i] + b[i[-1]]) < 1e-3:
            continue
        pp, pm = pre.copy(), pre.copy()
        pp[i] += h
        pm[i] -= h
        worst = max(worst, abs((L(pp, b) - L(pm, b)) / (2 * h) - dpre[i]))
    for c in range(5):
        if np.min(np.abs(pre[..., c] + b[c])) < 1e-3:
            continue
        bp, bm = b.copy(), b.copy()
        bp[c] += h
        bm[c] -= h
        worst = max(worst, abs((L(pre, bp) - L(pre, bm)) / (2 * h) - db[c]) / max(1, abs(db[c])))
    # exact zeros: y == 0 must give zero gradient, y > 0 must pass dy through
    z = np.array([[[[0.0, 1e-30, -0.0, 2.0]]]])
    dz, _ = oracle.bias_relu_bwd(z, np.ones_like(z))
    worst = max(worst, float(np.max(np.abs(dz - np.array([[[[0.0, 1.0, 0.0, 1.0]]]])))))
    return worst


# ----------------------------------------------------------------------------- sgd
def check_sgd_decrease(seed=13):
    """For a linear loss L(W) = <c, W> the gradient is c and one SGD step lowers L by
    exactly lr * ||c||^2 (up to rounding)."""
    rng = np.random.default_rng(seed)
    W = rng.standard_normal(1000)
    c = rng.standard_normal(1000)
    lr = float(np.float32(0.01))
    W2 = oracle.apply_sgd(W, c, lr)
    dl = float(np.dot(c, W2) - np.dot(c, W))
    return abs(dl + lr * float(np.dot(c, c))) / (lr * float(np.dot(c, c)))


# ----------------------------------------------------------------------------- momentum, adam
def _relerr(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(1.0, np.abs(b))))


def check_momentum_closed_form(nesterov=False, seed=16, T=7):
    """A constant gradient g from a zero velocity: after t steps the velocity is the geometric
    series g (1 - m^t) / (1 - m), so the parameter moves by lr g times the summed series (classical)
    or by lr g times (T + m times the summed series) (look-ahead form).  Also momentum 0 is SGD."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal(257)
    var0 = rng.standard_normal(257)
    lr, m = 0.05, 0.9
    var, acc = var0.copy(), np.zeros_like(g)
    for _ in range(T):
        var, acc = oracle.apply_momentum(var, acc, g, lr, m, nesterov)
    series = sum((1 - m ** t) / (1 - m) for t in range(1, T + 1))
    moved = T + m * series if nesterov else series
    worst = _relerr(acc, g * (1 - m ** T) / (1 - m))
    worst = max(worst, _relerr(var, var0 - lr * g * moved))
    v1, a1 = oracle.apply_momentum(var0, rng.standard_normal(257), g, lr, 0.0, nesterov)
    worst = max(worst, _relerr(v1, var0 - lr * g), _relerr(a1, g))
    return worst


def check_momentum_geometric_sum(nesterov=False, seed=17, T=6):
    """With any gradient sequence g_1..g_T and a zero start the velocity is sum_k m^(T-k) g_k, and
    the last parameter move is lr times it (classical) or lr (g_T + m times it) (look-ahead form)."""
    rng = np.random.default_rng(seed)
    gs = rng.standard_normal((T, 129))
    lr, m = 0.03, 0.75
    var, acc = rng.standard_normal(129), np.zeros(129)
    prev = var
    for g in gs:
        prev = var
        var, acc = oracle.apply_momentum(var, acc, g, lr, m, nesterov)
    vel = sum(m ** (T - 1 - k) * gs[k] for k in range(T))
    step = gs[-1] + m * vel if nesterov else vel
    return max(_relerr(acc, vel), _relerr(var, prev - lr * step))


def check_nesterov_closed_form():
    return check_momentum_closed_form(nesterov=True)


def check_adam_closed_form(seed=18, T=5):
    """A constant gradient g from zero moments: the moments are g (1 - b1^t) and g^2 (1 - b2^t), so
    the bias-corrected ones are exactly g and g^2 and every step moves the parameter by
    lr g / (|g| + eps).  eps is of the order of |g| so that where it enters shows."""
    rng = np.random.default_rng(seed)
    g = rng.uniform(-2.0, 2.0, 301)
    var0 = rng.standard_normal(301)
    lr, b1, b2, eps = 0.01, 0.9, 0.999, 0.3
    var, mm, vv = var0.copy(), np.zeros_like(g), np.zeros_like(g)
    for t in range(1, T + 1):
        var, mm, vv = oracle.apply_adam(var, mm, vv, g, lr, b1, b2, eps, t)
    worst = _relerr(mm, g * (1 - b1 ** T))
    worst = max(worst, _relerr(vv, g * g * (1 - b2 ** T)))
    worst = max(worst, _relerr(var, var0 - T * lr * g / (np.abs(g) + eps)))
    return worst


def check_adam_weighted_sums(seed=19, T=6):
    """With any gradient sequence and zero start, the moments are the exponentially weighted sums
    (1 - b1) sum_k b1^(T-k) g_k and (1 - b2) sum_k b2^(T-k) g_k^2.  With b1 = b2 = 0 a step is
    lr g / (|g| + eps) at every t."""
    rng = np.random.default_rng(seed)
    gs = rng.standard_normal((T, 131))
    lr, b1, b2, eps = 0.002, 0.8, 0.95, 1e-3
    var, mm, vv = rng.standard_normal(131), np.zeros(131), np.zeros(131)
    for t, g in enumerate(gs, start=1):
        var, mm, vv = oracle.apply_adam(var, mm, vv, g, lr, b1, b2, eps, t)
    m_ref = (1 - b1) * sum(b1 ** (T - 1 - k) * gs[k] for k in range(T))
    v_ref = (1 - b2) * sum(b2 ** (T - 1 - k) * gs[k] ** 2 for k in range(T))
    worst = max(_relerr(mm, m_ref), _relerr(vv, v_ref))
    var0 = rng.standard_normal(131)
    v3, _, _ = oracle.apply_adam(var0, rng.standard_normal(131), np.abs(rng.standard_normal(131)), gs[0],
                                 lr, 0.0, 0.0, eps, 3)
    worst = max(worst, _relerr(v3, var0 - lr * gs[0] / (np.abs(gs[0]) + eps)))
    return worst


# ----------------------------------------------------------------------------- softmax cross-entropy
def check_softmax_xent_vs_torch(seed=20, n=7, c=13):
    """Against the library: torch float64 cross_entropy per row, and the autograd gradient of the
    batch-mean loss (scale 1/n), with a bias added to the logits."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((n, c)) * 3
    b = rng.standard_normal(c)
    lab = rng.integers(0, c, size=n).astype(np.int32)
    rows, dz = oracle.softmax_xent(z, lab, 1.0 / n, bias=b)
    zt = torch.tensor(z + b, dtype=torch.float64, requires_grad=True)
    ref_rows = F.cross_entropy(zt, torch.tensor(lab, dtype=torch.int64), reduction="none")
    ref_rows.mean().backward()
    return max(rel(rows, ref_rows.detach().numpy()), rel(dz, zt.grad.numpy()))


def check_softmax_xent_closed_forms(seed=21, n=5, c=11):
    """Equal logits give loss log(c) and gradient scale (1/c - onehot); a shift of every logit of a
    row by +-1000 changes nothing (the max is taken out before exp); gradient rows sum to zero; a
    label outside [0, c) gives a NaN row."""
    rng = np.random.default_rng(seed)
    lab = rng.integers(0, c, size=n).astype(np.int32)
    rows, dz = oracle.softmax_xent(np.full((n, c), 0.7), lab, 0.25)
    onehot = np.eye(c)[lab]
    worst = max(float(np.max(np.abs(rows - np.log(c)))), float(np.max(np.abs(dz - 0.25 * (1.0 / c - onehot)))))
    z = rng.standard_normal((n, c))
    r0, d0 = oracle.softmax_xent(z, lab, 1.0)
    for shift in (1000.0, -1000.0):
        r1, d1 = oracle.softmax_xent(z + shift, lab, 1.0)
        worst = max(worst, float(np.max(np.abs(r1 - r0))) if np.all(np.isfinite(r1)) else np.inf,
                    float(np.max(np.abs(d1 - d0))) if np.all(np.isfinite(d1)) else np.inf)
    worst = max(worst, float(np.max(np.abs(d0.sum(axis=1)))))
    bad = lab.copy()
    bad[1], bad[3] = -1, c
    rb, db = oracle.softmax_xent(z, bad, 1.0)
    ok = (np.isnan(rb[1]) and np.isnan(rb[3]) and np.all(np.isnan(db[[1, 3]]))
          and np.array_equal(rb[[0, 2, 4]], r0[[0, 2, 4]]))
    return worst if ok else np.inf


def check_classifier_step_fd(net, inputs, samples=12, seed=22):
    """Finite differences of the batch-mean cross-entropy of a classifier net in the filters and
    biases of every layer and in x.  The loss is smooth apart from ReLU and max-pool kinks; entries
    whose steps h and h/2 disagree crossed one and are skipped."""
    rng = np.random.default_rng(seed)
    res = onet.step(net, inputs.x, inputs.weights, inputs.biases, None, labels=inputs.labels)
    lab = inputs.labels

    def L(ws, bs, xx):
        return onet.loss(net, xx, ws, bs, None, labels=lab)

    def fd(f, arr, idx, h):
        ap, am = arr.copy(), arr.copy()
        ap[idx] += h
        am[idx] -= h
        return (f(ap) - f(am)) / (2 * h)
    worst, checked = 0.0, 0
    targets = []
    for c in net.convs:
        targets.append(("W", c.name, inputs.weights[c.name], res["dW"][c.name]))
        targets.append(("b", c.name, inputs.biases[c.name], res["db"][c.name]))
    targets.append(("x", "x", inputs.x, res["grads"]["x"]))
    for kind, name, arr, ref in targets:
        gscale = max(float(np.max(np.abs(ref))), 1e-12)

        def f(a, kind=kind, name=name):
            ws, bs, xx = dict(inputs.weights), dict(inputs.biases), inputs.x
            if kind == "W":
                ws[name] = a
            elif kind == "b":
                bs[name] = a
            else:
                xx = a
            return L(ws, bs, xx)
        h = 1e-5 * float(np.sqrt(np.mean(arr ** 2)) or 1.0)
        for _ in range(samples):
            idx = tuple(int(rng.integers(0, d)) for d in arr.shape)
            d1, d2 = fd(f, arr, idx, h), fd(f, arr, idx, h / 2)
            if abs(d1 - d2) > 1e-6 * gscale:
                continue
            checked += 1
            worst = max(worst, abs(d2 - ref[idx]) / gscale)
    assert checked >= samples * len(targets) // 2, checked
    return worst


# ----------------------------------------------------------------------------- sampled softmax
def _sampled_case(rng, n=6, d=5, v=9):
    h = rng.standard_normal((n, d))
    W = rng.standard_normal((v, d))
    b = rng.standard_normal(v)
    lab = rng.integers(0, v, size=n).astype(np.int32)
    lq = rng.standard_normal(v)                    # log expected count of each class
    return h, W, b, lab, lq


def check_sampled_softmax_full_sample(seed=23):
    """Every class sampled once: with the true class removed from each row as an accidental hit,
    the candidates are the whole vocabulary, so the loss is the full softmax cross-entropy of the
    logits h W^T + b - log q, and dh, dW, db follow from its gradient by the chain rule."""
    rng = np.random.default_rng(seed)
    h, W, b, lab, lq = _sampled_case(rng)
    n = h.shape[0]
    smp = rng.permutation(W.shape[0]).astype(np.int32)
    loss, dh, dW, db = oracle.sampled_softmax(h, W, b, lab, smp, lq[lab], lq[smp], 1.0 / n)
    z = h @ W.T + b - lq
    rows, dz = oracle.softmax_xent(z, lab, 1.0 / n)
    return max(rel(loss, rows), rel(dh, dz @ W), rel(dW, dz.T @ h), rel(db, dz.sum(axis=0)))


def check_sampled_softmax_shift_and_fd(seed=24):
    """A constant added to every log q changes nothing; central differences of the summed loss in
    h, W and b (smooth in all of them) match the gradients."""
    rng = np.random.default_rng(seed)
    h, W, b, lab, lq = _sampled_case(rng)
    smp = np.array([1, 4, 7, 2], dtype=np.int32)
    args = lambda lqx: (lqx[lab], lqx[smp])
    loss, dh, dW, db = oracle.sampled_softmax(h, W, b, lab, smp, *args(lq), 1.0)
    l2 = oracle.sampled_softmax(h, W, b, lab, smp, *args(lq + 3.0), 1.0)[0]
    worst = rel(l2, loss)
    L = lambda hh, WW, bb: float(np.sum(oracle.sampled_softmax(hh, WW, bb, lab, smp, *args(lq), 1.0)[0]))
    eps = 1e-6
    for name, arr, grad in (("h", h, dh), ("W", W, dW), ("b", b, db)):
        for idx in [tuple(int(rng.integers(0, s)) for s in arr.shape) for _ in range(6)]:
            ap, am = arr.copy(), arr.copy()
            ap[idx] += eps
            am[idx] -= eps
            f = {"h": lambda a: L(a, W, b), "W": lambda a: L(h, a, b), "b": lambda a: L(h, W, a)}[name]
            fd = (f(ap) - f(am)) / (2 * eps)
            worst = max(worst, abs(fd - grad[idx]) / max(1.0, float(np.max(np.abs(grad)))))
    return worst


# ----------------------------------------------------------------------------- whole step
def check_step_fd(net, inputs, samples=24, seed=14):
    """Finite differences of the whole single-step surrogate loss L(W, b, x) = <g, out>.

    The net is piecewise linear, so a central difference that crosses no kink is exact;
    entries whose steps h and h/2 disagree crossed one and are skipped."""
    rng = np.random.default_rng(seed)
    res = onet.step(net, inputs.x, inputs.weights, inputs.biases, inputs.g)
    conv = net.convs[0]
    W, b, x, g = inputs.weights[conv.name], inputs.biases[conv.name], inputs.x, inputs.g

    def L(WW, bb, xx):
        return onet.loss(net, xx, {conv.name: WW}, {conv.name: bb}, g)
    worst = 0.0
    checked = 0
    gscale = max(np.max(np.abs(res["dW"][conv.name])), 1e-12)

    def fd(f, arr, idx, h):
        ap, am = arr.copy(), arr.copy()
        ap[idx] += h
        am[idx] -= h
        return (f(ap) - f(am)) / (2 * h)
    for kind in ("W", "b", "x"):
        arr = {"W": W, "b": b, "x": x}[kind]
        ref = {"W": res["dW"][conv.name], "b": res["db"][conv.name], "x": res["grads"].get("x")}[kind]
        if ref is None:
            continue
        f = {"W": lambda a: L(a, b, x), "b": lambda a: L(W, a, x), "x": lambda a: L(W, b, a)}[kind]
        h = 1e-6 * float(np.sqrt(np.mean(arr ** 2)) or 1.0)
        for _ in range(samples):
            idx = tuple(int(rng.integers(0, d)) for d in arr.shape)
            d1, d2 = fd(f, arr, idx, h), fd(f, arr, idx, h / 2)
            if abs(d1 - d2) > 1e-6 * gscale:
                continue
            checked += 1
            worst = max(worst, abs(d1 - ref[idx]) / gscale)
    assert checked >= samples, checked
    return worst


def check_step_decrease(net, inputs):
    """Piecewise-linear net: with a tiny lr no kink or argmax switch is crossed, and one SGD
    step lowers L by exactly lr * (||dW||^2 + ||db||^2)."""
    lr = 1e-9
    res = onet.step(net, inputs.x, inputs.weights, inputs.biases, inputs.g, lr=lr)
    lr = float(np.float32(lr))
    L0 = onet.loss(net, inputs.x, inputs.weights, inputs.biases, inputs.g)
    L1 = onet.loss(net, inputs.x, res["new_weights"], res["new_biases"], inputs.g)
    pred = -lr * sum(float(np.sum(v ** 2)) for v in list(res["dW"].values()) + list(res["db"].values()))
    return abs((L1 - L0) - pred) / abs(pred)
