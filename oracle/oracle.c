/*
 * CPU oracle for one synchronous SGD step of a convnet replica.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * reference that the HIP kernels are checked against.  Only the tests, the
 * smoke check and the bench's CPU-baseline leg may load it; the product path
 * never does.  It shares no code, header or constant with the HIP library.
 *
 * Every array is dense and float64.  Activations are NHWC row-major
 * (x[n][h][w][c]); filters are HWIO row-major (w[kh][kw][ci][co]); pool argmax
 * is int32.  Every sum runs in a fixed order inside one output element, and
 * OpenMP only splits *independent* output elements across threads, so results
 * are bitwise identical for any thread count.
 *
 * The paper (Section 3.1) treats a mini-batch 2-D convolution as an operation
 * from two 4-D tensors to a 4-D tensor, and (Section 6.1) puts convolution and
 * pooling on the critical path of training; it does not spell out their
 * arithmetic.  The definitions below use the conventions of the paper's
 * system: cross-correlation (no filter flip), explicit padding, max-pooling
 * over in-bounds taps only, gradient = sum of the partial gradients of every
 * path (Section 4.1), and the update W' = W - alpha * dL/dW (Section 4.1).
 *
 * Parity pins (what fixes each function independently of this file) live in
 * the CPU tests: brute-force finite differences, adjoint identities, delta
 * kernels, library convolution and matmul, closed forms and brute-force
 * window scans.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef int64_t i64;

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Number of windows along one axis with explicit padding: floor((n+p0+p1-k)/s)+1. */
int orc_out_len(int n, int k, int s, int p0, int p1) {
    int span = n + p0 + p1 - k;
    if (span < 0 || s <= 0) return 0;
    return span / s + 1;
}

/*
 * Conv2D forward (cross-correlation):
 *   y[n,oh,ow,co] = sum_{kh,kw,ci} X[n, oh*sh+kh-pt, ow*sw+kw-pl, ci] * w[kh,kw,ci,co]
 * with X = 0 outside [0,H) x [0,W).  Sum order: kh, kw, ci.
 */
void orc_conv2d_fwd(const double *x, int N, int H, int W, int C,
                    const double *w, int KH, int KW, int K,
                    int sh, int sw, int pt, int pl,
                    double *y, int OH, int OW) {
    i64 npix = (i64)N * OH * OW;
#pragma omp parallel for schedule(static)
    for (i64 p = 0; p < npix; ++p) {
        int n = (int)(p / ((i64)OH * OW));
        int oh = (int)((p / OW) % OH);
        int ow = (int)(p % OW);
        double *out = y + p * K;
        for (int co = 0; co < K; ++co) out[co] = 0.0;
        for (int kh = 0; kh < KH; ++kh) {
            int ih = oh * sh + kh - pt;
            if (ih < 0 || ih >= H) continue;
            for (int kw = 0; kw < KW; ++kw) {
                int iw = ow * sw + kw - pl;
                if (iw < 0 || iw >= W) continue;
                const double *xin = x + (((i64)n * H + ih) * W + iw) * C;
                for (int ci = 0; ci < C; ++ci) {
                    const double xv = xin[ci];
                    const double *wr = w + (((i64)kh * KW + kw) * C + ci) * K;
                    for (int co = 0; co < K; ++co) out[co] += xv * wr[co];
                }
            }
        }
    }
}

/*
 * Conv2DBackpropInput: the adjoint of the forward map in x.
 *   dx[n,h,w,ci] = sum over (kh,kw,co) and the unique (oh,ow) with
 *                  oh*sh + kh - pt = h and ow*sw + kw - pl = w
 *                  (0 <= oh < OH, 0 <= ow < OW) of dy[n,oh,ow,co] * w[kh,kw,ci,co].
 * Written as a gather per dx element; input positions no window reaches get 0.
 * beta == 0: dx is overwritten; beta == 1: the sum is added to dx.
 * Sum order: kh, kw, co (after the old value when beta == 1).
 */
void orc_conv2d_bwd_input(const double *dy, int N, int OH, int OW, int K,
                          const double *w, int KH, int KW,
                          int sh, int sw, int pt, int pl,
                          double *dx, int H, int W, int C, int beta) {
    i64 npix = (i64)N * H * W;
#pragma omp parallel for schedule(static)
    for (i64 p = 0; p < npix; ++p) {
        int n = (int)(p / ((i64)H * W));
        int h = (int)((p / W) % H);
        int wi = (int)(p % W);
        for (int ci = 0; ci < C; ++ci) {
            double acc = beta ? dx[p * C + ci] : 0.0;
            for (int kh = 0; kh < KH; ++kh) {
                int th = h + pt - kh;            /* = oh*sh */
                if (th < 0 || th % sh != 0) continue;
                int oh = th / sh;
                if (oh >= OH) continue;
                for (int kw = 0; kw < KW; ++kw) {
                    int tw = wi + pl - kw;       /* = ow*sw */
                    if (tw < 0 || tw % sw != 0) continue;
                    int ow = tw / sw;
                    if (ow >= OW) continue;
                    const double *g = dy + (((i64)n * OH + oh) * OW + ow) * K;
                    const double *wr = w + (((i64)kh * KW + kw) * C + ci) * K;
                    for (int co = 0; co < K; ++co) acc += g[co] * wr[co];
                }
            }
            dx[p * C + ci] = acc;
        }
    }
}

/*
 * Conv2DBackpropFilter: the adjoint of the forward map in w.
 *   dw[kh,kw,ci,co] = sum_{n,oh,ow} X[n, oh*sh+kh-pt, ow*sw+kw-pl, ci] * dy[n,oh,ow,co]
 * (padding contributes nothing).  dw is overwritten.  Sum order: n, oh, ow.
 */
void orc_conv2d_bwd_filter(const double *x, int N, int H, int W, int C,
                           const double *dy, int OH, int OW, int K,
                           int KH, int KW, int sh, int sw, int pt, int pl,
                           double *dw) {
    i64 rows = (i64)KH * KW * C;
#pragma omp parallel for schedule(dynamic, 1)
    for (i64 r = 0; r < rows; ++r) {
        int kh = (int)(r / ((i64)KW * C));
        int kw = (int)((r / C) % KW);
        int ci = (int)(r % C);
        double *out = dw + r * K;
        for (int co = 0; co < K; ++co) out[co] = 0.0;
        for (int n = 0; n < N; ++n)
            for (int oh = 0; oh < OH; ++oh) {
                int ih = oh * sh + kh - pt;
                if (ih < 0 || ih >= H) continue;
                for (int ow = 0; ow < OW; ++ow) {
                    int iw = ow * sw + kw - pl;
                    if (iw < 0 || iw >= W) continue;
                    const double xv = x[(((i64)n * H + ih) * W + iw) * C + ci];
                    const double *g = dy + (((i64)n * OH + oh) * OW + ow) * K;
                    for (int co = 0; co < K; ++co) out[co] += xv * g[co];
                }
            }
    }
}

/*
 * Selected elements of Conv2DBackpropFilter (same definition and sum order as
 * above): out[i] = dw[idx[i]] for flat HWIO indices idx[i].  Lets a check
 * evaluate a handful of filter-gradient entries of a full-size problem.
 */
void orc_conv2d_bwd_filter_at(const double *x, int N, int H, int W, int C,
                              const double *dy, int OH, int OW, int K,
                              int KH, int KW, int sh, int sw, int pt, int pl,
                              const int64_t *idx, i64 count, double *out) {
#pragma omp parallel for schedule(dynamic, 1)
    for (i64 i = 0; i < count; ++i) {
        i64 f = idx[i];
        int co = (int)(f % K);
        int ci = (int)((f / K) % C);
        int kw = (int)((f / ((i64)K * C)) % KW);
        int kh = (int)(f / ((i64)K * C * KW));
        double s = 0.0;
        for (int n = 0; n < N; ++n)
            for (int oh = 0; oh < OH; ++oh) {
                int ih = oh * sh + kh - pt;
                if (ih < 0 || ih >= H) continue;
                for (int ow = 0; ow < OW; ++ow) {
                    int iw = ow * sw + kw - pl;
                    if (iw < 0 || iw >= W) continue;
                    s += x[(((i64)n * H + ih) * W + iw) * C + ci] *
                         dy[(((i64)n * OH + oh) * OW + ow) * K + co];
                }
            }
        out[i] = s;
    }
}

/*
 * Fused BiasAdd + ReLU forward over P pixels of C channels:
 *   y = pre + b[c];  y = (y > 0) ? y : +0.0
 * (the paper's hand-fused ReLU kernels, Section 5).  y may equal pre.
 */
void orc_bias_relu_fwd(const double *pre, const double *b, i64 P, int C, double *y) {
#pragma omp parallel for schedule(static)
    for (i64 p = 0; p < P; ++p)
        for (int c = 0; c < C; ++c) {
            double v = pre[p * C + c] + b[c];
            y[p * C + c] = v > 0.0 ? v : 0.0;
        }
}

/*
 * ReLU backward + bias gradient:
 *   dpre = (y > 0) ? dy : 0            (mask from the stored output y)
 *   db[c] = sum_p dpre[p, c]           (ascending p)
 * dpre may equal dy.
 */
void orc_bias_relu_bwd(const double *y, const double *dy, i64 P, int C,
                       double *dpre, double *db) {
#pragma omp parallel for schedule(static)
    for (i64 p = 0; p < P; ++p)
        for (int c = 0; c < C; ++c)
            dpre[p * C + c] = y[p * C + c] > 0.0 ? dy[p * C + c] : 0.0;
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; ++c) {
        double s = 0.0;
        for (i64 p = 0; p < P; ++p) s += dpre[p * C + c];
        db[c] = s;
    }
}

/*
 * MaxPool forward with argmax.  For each output (n,oh,ow,c) the window taps
 * are scanned kh outer, kw inner, skipping taps outside [0,H) x [0,W).  The
 * first in-bounds tap seeds the maximum; a later tap replaces it only if
 * strictly greater, so the first maximum in scan order wins.  argmax is the
 * flat dense NHWC index ((n*H + h)*W + w)*C + c into x.  A window with no
 * in-bounds tap yields y = 0 and argmax = -1 (the HIP library rejects such
 * windows before launching).
 */
void orc_maxpool_fwd(const double *x, int N, int H, int W, int C,
                     int KH, int KW, int sh, int sw, int pt, int pl,
                     double *y, int32_t *argmax, int OH, int OW) {
    i64 total = (i64)N * OH * OW * C;
#pragma omp parallel for schedule(static)
    for (i64 o = 0; o < total; ++o) {
        int c = (int)(o % C);
        i64 pix = o / C;
        int ow = (int)(pix % OW);
        int oh = (int)((pix / OW) % OH);
        int n = (int)(pix / ((i64)OW * OH));
        int have = 0;
        double best = 0.0;
        i64 besti = -1;
        for (int kh = 0; kh < KH; ++kh) {
            int ih = oh * sh + kh - pt;
            if (ih < 0 || ih >= H) continue;
            for (int kw = 0; kw < KW; ++kw) {
                int iw = ow * sw + kw - pl;
                if (iw < 0 || iw >= W) continue;
                i64 idx = (((i64)n * H + ih) * W + iw) * C + c;
                double v = x[idx];
                if (!have || v > best) {
                    best = v;
                    besti = idx;
                    have = 1;
                }
            }
        }
        y[o] = best;
        argmax[o] = (int32_t)besti;
    }
}

/*
 * MaxPool backward: dx[i] = (beta ? dx[i] : 0) + sum_{o : argmax[o] == i} dy[o],
 * the routed contributions added in ascending o.  nx = number of x elements,
 * ny = number of pooled elements.  Indices outside [0, nx) are ignored.
 */
void orc_maxpool_bwd(const double *dy, const int32_t *argmax, i64 ny,
                     double *dx, i64 nx, int beta) {
    if (!beta) memset(dx, 0, sizeof(double) * (size_t)nx);
    for (i64 o = 0; o < ny; ++o) {
        i64 i = argmax[o];
        if (i >= 0 && i < nx) dx[i] += dy[o];
    }
}

/* ApplyGradientDescent, in place: var <- var - lr * grad (Section 4.1). */
void orc_apply_sgd(double *var, const double *grad, i64 n, double lr) {
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i) var[i] = var[i] - lr * grad[i];
}

/* Momentum (Section 4.1 names it: a per-parameter velocity accumulated from the gradients,
 * from which the update is computed), in the velocity form of Sutskever et al. (2013):
 *   accum <- momentum * accum + grad
 *   var   <- var - lr * accum                         (classical)
 *   var   <- var - lr * (grad + momentum * accum)     (nesterov: the look-ahead form)
 * with accum already updated in the nesterov line. */
void orc_apply_momentum(double *var, double *accum, const double *grad, i64 n, double lr, double momentum,
                        int nesterov) {
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i) {
        accum[i] = momentum * accum[i] + grad[i];
        if (nesterov)
            var[i] = var[i] - lr * (grad[i] + momentum * accum[i]);
        else
            var[i] = var[i] - lr * accum[i];
    }
}

/* Adam (named in Section 4.1), Algorithm 1 of Kingma & Ba (2015), step t >= 1:
 *   m    <- beta1 * m + (1 - beta1) * grad
 *   v    <- beta2 * v + (1 - beta2) * grad^2
 *   mhat  = m / (1 - beta1^t),  vhat = v / (1 - beta2^t)
 *   var  <- var - lr * mhat / (sqrt(vhat) + epsilon) */
void orc_apply_adam(double *var, double *m, double *v, const double *grad, i64 n, double lr, double beta1,
                    double beta2, double epsilon, int t) {
    const double c1 = 1.0 - pow(beta1, (double)t), c2 = 1.0 - pow(beta2, (double)t);
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i) {
        m[i] = beta1 * m[i] + (1.0 - beta1) * grad[i];
        v[i] = beta2 * v[i] + (1.0 - beta2) * grad[i] * grad[i];
        const double mhat = m[i] / c1, vhat = v[i] / c2;
        var[i] = var[i] - lr * mhat / (sqrt(vhat) + epsilon);
    }
}

/* Softmax cross-entropy of a classifier's logits against integer labels (the paper's image
 * models end in a softmax classifier trained by the gradient of its loss, Section 4.1).
 * Row i of z = logits + bias (bias may be NULL), n rows of c classes:
 *   loss[i]  = log(sum_j exp(z_ij)) - z_i,label      evaluated as m + log(sum_j exp(z_ij - m)),
 *                                                     m = max_j z_ij, so no exp overflows
 *   dz[i][j] = scale * (exp(z_ij - m) / sum_k exp(z_ik - m) - [j == label])
 * A label outside [0, c) gives a NaN loss and a NaN gradient row. */
void orc_softmax_xent(const double *logits, const double *bias, const int32_t *labels, i64 n, int c,
                      double scale, double *loss, double *dz) {
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i) {
        const double *zr = logits + i * c;
        double *dr = dz + i * c;
        const int lab = labels[i];
        if (lab < 0 || lab >= c) {
            loss[i] = NAN;
            for (int j = 0; j < c; ++j) dr[j] = NAN;
            continue;
        }
        double m = -INFINITY;
        for (int j = 0; j < c; ++j) {
            const double z = zr[j] + (bias ? bias[j] : 0.0);
            if (z > m) m = z;
        }
        double sum = 0.0;
        for (int j = 0; j < c; ++j) sum += exp(zr[j] + (bias ? bias[j] : 0.0) - m);
        loss[i] = m + log(sum) - (zr[lab] + (bias ? bias[lab] : 0.0));
        for (int j = 0; j < c; ++j) {
            const double p = exp(zr[j] + (bias ? bias[j] : 0.0) - m) / sum;
            dr[j] = scale * (p - (j == lab ? 1.0 : 0.0));
        }
    }
}

/* Sampled softmax (Section 4.2, large classifiers; evaluated in Section 6.4; Jean et al. 2015):
 * the classifier's output h (n x d) meets only the weight rows of each example's true class
 * and of one shared sample of classes, drawn from a proposal Q by the caller.  For row i the
 * candidate logits are
 *   true:     h_i . W[t_i] + b[t_i] - lq_true[i]
 *   sampled:  h_i . W[s_j] + b[s_j] - lq_sampled[j]    (j < m; lq = log expected count under Q)
 * and a sampled class equal to t_i (an accidental hit) is left out of row i.  The loss is the
 * cross-entropy with the true class at position 0:
 *   loss[i] = log(sum over candidates of exp(logit)) - true logit
 * Gradients (scale = 1/n for the batch mean), accumulated over every use of a class:
 *   dh[i] = scale * sum_c (p_c - [c true]) W[c],   dW[c] += scale * (p_c - [c true]) h_i,
 *   db[c] += scale * (p_c - [c true]).
 * dW (v x d) and db (v) are dense and overwritten. */
void orc_sampled_softmax(const double *h, const double *W, const double *b, const int32_t *labels,
                         const int32_t *sampled, const double *lq_true, const double *lq_sampled, i64 n, int d,
                         int v, int m, double scale, double *loss, double *dh, double *dW, double *db) {
    memset(dW, 0, sizeof(double) * (size_t)v * d);
    memset(db, 0, sizeof(double) * (size_t)v);
    double *z = (double *)malloc(sizeof(double) * (size_t)(m + 1));
    for (i64 i = 0; i < n; ++i) {          /* rows in order: the dW, db accumulation order is fixed */
        const double *hi = h + i * d;
        const int t = labels[i];
        double zt = b[t] - lq_true[i];
        for (int k = 0; k < d; ++k) zt += hi[k] * W[(i64)t * d + k];
        z[0] = zt;
        double mx = zt;
        for (int j = 0; j < m; ++j) {
            const int c = sampled[j];
            if (c == t) { z[j + 1] = -INFINITY; continue; }
            double zz = b[c] - lq_sampled[j];
            for (int k = 0; k < d; ++k) zz += hi[k] * W[(i64)c * d + k];
            z[j + 1] = zz;
            if (zz > mx) mx = zz;
        }
        double sum = 0.0;
        for (int j = 0; j <= m; ++j) sum += exp(z[j] - mx);
        loss[i] = mx + log(sum) - zt;
        double *dhi = dh + i * d;
        for (int k = 0; k < d; ++k) dhi[k] = 0.0;
        for (int j = 0; j <= m; ++j) {
            const int c = j == 0 ? t : sampled[j - 1];
            const double g = scale * (exp(z[j] - mx) / sum - (j == 0 ? 1.0 : 0.0));
            if (j > 0 && c == t) continue;
            for (int k = 0; k < d; ++k) {
                dhi[k] += g * W[(i64)c * d + k];
                dW[(i64)c * d + k] += g * hi[k];
            }
            db[c] += g;
        }
    }
    free(z);
}
