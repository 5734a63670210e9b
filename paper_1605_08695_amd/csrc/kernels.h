// Internal interface between the C ABI (api.cpp) and the gfx950 kernels.
// Everything here is validated by the caller before it is reached.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace tfk {

// Geometry of one forward convolution (input N,H,W,C; output OH,OW,K).
struct ConvShape {
    int N, H, W, C;
    int OH, OW, K;
    int KH, KW, sh, sw, pt, pl;
};

struct PoolGeom {
    int N, H, W, C;      // input
    int OH, OW;          // output
    int KH, KW, sh, sw, pt, pl;
    int64_t xs, ys;      // pixel strides of x (dx) and y (dy)
};

// Scalars of the Momentum and Adam updates, rounded to fp32 on the host.  Adam's bias
// corrections are folded in: lr = lr / (1 - b1^t), rc2 = 1 / (1 - b2^t).
struct OptParams {
    float lr, mom, b1, omb1, b2, omb2, rc2, eps;
};

constexpr int kSgdBatch = 16;
struct SgdBatch {
    int count;
    float *var[kSgdBatch];
    const float *grad[kSgdBatch];
    uint16_t *shadow[kSgdBatch];
    int64_t n[kSgdBatch];
    int64_t blk_start[kSgdBatch + 1];   // prefix sums of ceil(n / 1024)
};

// dt: 0 = fp32, 1 = bf16
// bias (may be null): fused y = max(conv + bias, +0).
hipError_t launch_conv_fwd(int dt, const void *x, int64_t xs, const void *w, void *y, int64_t ys,
                           const ConvShape &s, const float *bias, void *ws, hipStream_t st);
// The forward convolution with bias + ReLU and a VALID max-pool of its output (g: the pool over
// y) fused in one kernel, when its row bands cover whole pool windows (bf16, the implicit-GEMM
// path): writes y, the pooled py (pixel stride pys) and the uint8 window taps.  Returns false,
// launching nothing, when the fused kernel does not apply.
bool conv_fwd_pool_fused(const void *x, int64_t xs, const void *w, void *y, int64_t ys, const ConvShape &s,
                         const float *bias, const PoolGeom &g, void *py, int64_t pys, uint8_t *taps,
                         hipStream_t st, hipError_t *err);
hipError_t launch_conv_bwd_data(int dt, const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs,
                                float beta, const ConvShape &s, float *ws, hipStream_t st);
// Workspace of the split-K forward / input gradient (0: no split for this shape).
size_t conv_fwd_split_ws_bytes(int dt, const ConvShape &s);
size_t conv_bwd_data_ws_bytes(int dt, const ConvShape &s);
// Where a bias-gradient producer given a BiasPartials* left its per-channel partial sums instead of
// reducing them: channel c's rows values at part[c * rows .. c * rows + rows - 1] (inside its ws).
struct BiasPartials {
    const float *part;
    int rows;
};
// Input gradient fused with the ReLU backward + bias gradient of the layer that produced x:
// dpre = y > 0 ? bwd_input(dy, w) : +0 (dx's view), db = column sums of dpre; ws: partials.
// defer: if not NULL, db is not written and the partials are left where *defer says.
hipError_t launch_conv_bwd_data_relu(int dt, const void *dy, int64_t dys, const void *w, void *dpre, int64_t dxs,
                                     const void *y, float beta, float *db, float *ws, const ConvShape &s,
                                     hipStream_t st, BiasPartials *defer = nullptr);
size_t conv_bwd_data_relu_ws_bytes(int dt, const ConvShape &s, int64_t dxs);
// Per-channel sums of partial[c][G] (G values per channel, summed in order) into out[C].
hipError_t launch_sum_partials(const float *partial, int G, int C, float *out, hipStream_t st);
// The same sums for several tensors in one launch per kPartialsBatch of them (job i: channels[i]
// channels of rows[i] partials at part[i], into out[i]), each channel summed in the same order.
constexpr int kPartialsBatch = 32;
struct PartialsBatch {
    int count;
    int chan0[kPartialsBatch + 1];                 // first block of each job; chan0[count] = total
    const float *part[kPartialsBatch];
    int rows[kPartialsBatch];
    float *out[kPartialsBatch];
};
hipError_t launch_sum_partials_multi(int count, const float *const *part, const int *rows, const int *channels,
                                     float *const *out, hipStream_t st);
hipError_t launch_conv_bwd_filter(int dt, const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                  const ConvShape &s, void *ws, hipStream_t st);
// Split-K plan of bwd-filter: number of splits and reduction elements per split.
void conv_bwd_filter_plan(int dt, const ConvShape &s, int *splits, int *k_split);
size_t conv_bwd_filter_ws_bytes(int dt, const ConvShape &s);
// The library's own device scratch (noalloc.hip): its size, and its address on the current
// device, which must be the device of `stream`.
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void **ptr, hipStream_t stream);
// bf16 convolutions with C % 8 != 0 run as an equivalent 8-channel convolution (conv_fold.hip).
bool conv_fold_applies(int dt, const ConvShape &s);
size_t conv_fold_ws_bytes(int op, const ConvShape &s);
hipError_t launch_conv_fwd_folded(const void *x, int64_t xs, const void *w, void *y, int64_t ys, const ConvShape &s,
                                  const float *bias, void *ws, hipStream_t st);
hipError_t launch_conv_bwd_filter_folded(const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                         const ConvShape &s, void *ws, hipStream_t st);

// First layers with at most 4 input channels as band kernels (conv_band.hip): the input is read
// as 4-channel pixels (an RGBx view in place, or a padded copy made by rgbx_input in xp).
const uint16_t *rgbx_input(const void *x, int64_t npix, int C, int64_t xs, uint16_t *xp, hipStream_t st);
bool conv_band_fwd_applies(const ConvShape &s);
bool conv_band_bwf_applies(const ConvShape &s);
size_t conv_band_bwf_partial_bytes(const ConvShape &s);
hipError_t launch_conv_fwd_band(const uint16_t *x4, const void *w, void *y, int64_t ys, const ConvShape &s,
                                const float *bias, hipStream_t st);
hipError_t launch_conv_bwd_filter_band(const uint16_t *x4, const void *dy, int64_t dys, float *dw, const ConvShape &s,
                                       float *part, hipStream_t st);

hipError_t launch_bias_relu_fwd(int dt, void *y, int64_t P, int C, int64_t ys, const float *bias, hipStream_t st);
void relu_bwd_plan(int dt, int64_t P, int C, int64_t ys, int *G, int64_t *ppb);
void relu_bwd_only_plan(int dt, int64_t P, int C, int64_t ys, int *G, int64_t *ppb);
hipError_t launch_bias_relu_bwd(int dt, const void *y, const void *dy, void *dpre, int64_t P, int C,
                                int64_t ys, float *db, float *ws, hipStream_t st, BiasPartials *defer = nullptr);
// am: int32 dense-index argmax, or with taps the uint8 window tap kh * KW + kw.
hipError_t launch_maxpool_fwd(int dt, const void *x, const PoolGeom &g, void *y, void *am, bool taps, hipStream_t st);
hipError_t launch_maxpool_bwd(int dt, const void *dy, const void *am, bool taps, const PoolGeom &g, float beta,
                              void *dx, hipStream_t st);
// Fused max-pool backward + ReLU backward + bias gradient over the pool input y (pixel stride g.xs);
// ws holds the bias-gradient partials of relu_bwd_plan.  py (beta = 0 only; else NULL): the pool's
// output (pixel stride pys), whose windows give the ReLU mask in place of y, which is then not read.
hipError_t launch_maxpool_relu_bwd(int dt, const void *dy, const void *am, bool taps, const PoolGeom &g,
                                   const void *y, const void *py, int64_t pys, void *dpre, float beta, float *db,
                                   float *ws, hipStream_t st, BiasPartials *defer = nullptr);
hipError_t launch_sgd(float *var, const float *grad, int64_t n, float lr, uint16_t *sh, hipStream_t st);
hipError_t launch_sgd_multi(const SgdBatch &b, float lr, hipStream_t st);
// Epilogue of a split-K forward or input-gradient GEMM: out[j][i] = f(sum over splits, in split
// order, of part[s][j][i]) stored as bf16 at out + j * ostride + i, with f adding bias then ReLU
// (forward, bias set), beta * old out (input gradient), or the ReLU backward mask y > 0 of the
// producing layer (relu_y set; the stored values also go to db_part[i][j], the rows of the
// bias gradient's partial sums).
struct SplitEpi {
    const float *part;
    int splits, rows, ni;
    int64_t split_stride, ostride;
    void *out;
    const float *bias;
    float beta;
    const void *relu_y;
    float *db_part;
};
hipError_t launch_split_epilogue(const SplitEpi &e, hipStream_t st);
// Sampled softmax: candidate-row gather (as the columns of a d x u_pad filter), the
// candidate cross-entropy, and the sparse SGD of the candidate rows.
hipError_t launch_gather_rows_t(int dt, const void *table, int64_t rows, int d, const int32_t *idx, int u,
                                int u_pad, void *out_t, hipStream_t st);
hipError_t launch_sampled_xent(int dt, const void *z, int64_t n, int u, int u_pad, int m, const float *bc,
                               const int32_t *tp, const float *lq_true, const float *lq_sampled, float scale,
                               float *loss, void *dz, hipStream_t st);
hipError_t launch_scatter_sgd(float *var, uint16_t *sh, int64_t rows, int d, const int32_t *idx, int u,
                              const float *grad_t, int64_t ld, float lr, hipStream_t st);
// Softmax cross-entropy of n x c logits (+ bias) against labels: per-row loss and
// dz = scale * (softmax - onehot); dz may be z.
hipError_t launch_softmax_xent(int dt, const void *z, const float *bias, const int32_t *labels, int64_t n, int c,
                               float scale, float *loss, void *dz, hipStream_t st);
// Momentum (kind 0, 1 = look-ahead form) and Adam (kind 2) in place over n fp32 elements.
hipError_t launch_opt(int kind, float *var, float *s1, float *s2, const float *grad, int64_t n, const OptParams &p,
                      uint16_t *sh, hipStream_t st);
// Sums split-K partials part[splits][mn] into out; part (workspace) is overwritten.
hipError_t launch_sum_splits(float *part, int splits, int64_t mn, float *out, hipStream_t st);
hipError_t launch_fill_zero(float *out, int64_t n, hipStream_t st);

}  // namespace tfk
