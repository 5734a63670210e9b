// Conv2DBackpropInput on gfx950 MFMA, one stride phase per blockIdx.z:
// Out[p'][ci] = sum over the phase's taps (kh, kw) and co of dy[...][co] * w[kh][kw][ci][co].
#include "igemm_launch.h"

namespace tfk {

// The forward pass's tile rule.  (64 x 192 tiles for 33-64 input channels over many pixels copy
// 48 flop per byte against 64 x 128's 43 and ran AlexNet conv2's input gradient faster alone,
// 74.8 -> 71.3 us back to back, but the sustained two-stream step slower, 0.694 -> 0.705 ms, where
// the filter gradient of the other stream shares the GPU with it; GoogLeNet and Inception-v3
// steps are the same either way.)
static Igemm2Tile bwd_data_tiles(int ni, int mj, int zdim) {
    return igemm2_tiles_narrow(ni, mj, zdim);
}

// Rows of bias-gradient partials of the fused ReLU-backward epilogue: one per block and wave
// column of the pipelined kernel's grid.
static int relu_partial_rows(const ConvShape &s) {
    const int mj = s.N * ((s.H + s.sh - 1) / s.sh) * ((s.W + s.sw - 1) / s.sw);
    const int z = s.sh * s.sw;
    const Igemm2Tile t = bwd_data_tiles(s.C, mj, z);
    return z * ((mj + t.bj - 1) / t.bj) * (t.nw / 2);
}

// Split-K at stride 1 (one phase) with few output tiles (fully connected layers and small late-
// stage images at small batch): fp32 partials in the workspace, then one epilogue pass (beta,
// or the fused ReLU backward with the bias-gradient rows after the partials).
static int bwd_data_splits(const ConvShape &s, int *k_split) {
    *k_split = 0;
    if (s.sh != 1 || s.sw != 1) return 1;
    return gemm_split_plan(s.C, s.N * s.H * s.W, (int64_t)s.KH * s.KW * s.K, k_split);
}

static size_t split_ws_bytes(int dt, const ConvShape &s, bool relu) {
    int ks;
    const int sp = bwd_data_splits(s, &ks);
    if (dt != 1 || sp <= 1) return 0;
    const int64_t mj = (int64_t)s.N * s.H * s.W;
    return (size_t)((sp + (relu ? 1 : 0)) * mj) * s.C * sizeof(float);
}

size_t conv_bwd_data_ws_bytes(int dt, const ConvShape &s) { return split_ws_bytes(dt, s, false); }

// ws: workspace (split-K partials; with relu_y also the bias-gradient partials).
// relu_y: the fused ReLU backward (of beta dx + the gradient); *db_parts / *db_at receive the number and place of
// the bias-gradient partial rows, or 0 when the fused kernels do not apply (nothing is launched
// then).
template <typename T>
static hipError_t conv_bwd_data_t(const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs, float beta,
                                  const ConvShape &s, hipStream_t st, float *ws, const void *relu_y = nullptr,
                                  int *db_parts = nullptr, float **db_at = nullptr) {
    constexpr int EPC = Elem<T>::kPerChunk;
    IgArgs a;
    fill_geom(a, s);
    a.src_i = w;
    a.src_j = dy;
    a.out = dx;
    a.xs = dxs;
    a.ys = dys;
    a.beta = beta;
    a.NI = s.C;
    const bool vi = s.K % EPC == 0 && aligned16p(w);
    const bool vj = s.K % EPC == 0 && dys % EPC == 0 && aligned16p(dy);
    // largest phase: ceil(H / sh) x ceil(W / sw) pixels per image
    const int mj = s.N * ((s.H + s.sh - 1) / s.sh) * ((s.W + s.sw - 1) / s.sw);
    if constexpr (sizeof(T) == 2) {
        const int64_t wb = (int64_t)s.KH * s.KW * s.C * s.K * 2;
        if (vi && vj && s.C % 8 == 0 && dxs % 8 == 0 && aligned16p(dx) &&
            igemm2_fits(a, wb, span_bytes((int64_t)s.N * s.OH * s.OW, dys, s.K))) {
            const int z = s.sh * s.sw;
            int ks;
            const int sp = ws != nullptr && aligned16p(ws) ? bwd_data_splits(s, &ks) : 1;
            if (sp > 1) {
                a.k_split = ks;
                a.split_stride = (int64_t)mj * a.NI;
                a.out = ws;
                if (!igemm2_launch<DIR_BWD_DATA>(a, mj, sp, bwd_data_tiles(a.NI, mj, sp), st))
                    return hipErrorInvalidValue;
                const hipError_t e = hipGetLastError();
                if (e != hipSuccess) return e;
                SplitEpi ep{};
                ep.part = ws;
                ep.splits = sp;
                ep.rows = mj;
                ep.ni = a.NI;
                ep.split_stride = a.split_stride;
                ep.ostride = dxs;
                ep.out = dx;
                ep.beta = beta;
                ep.relu_y = relu_y;
                if (relu_y != nullptr) {                 // one partial row per output row
                    ep.db_part = ws + (int64_t)sp * mj * a.NI;
                    *db_parts = mj;
                    *db_at = ep.db_part;
                }
                return launch_split_epilogue(ep, st);
            }
            if (relu_y != nullptr) {
                a.relu_y = relu_y;
                a.db_part = ws;
                a.db_rows = relu_partial_rows(s);
                *db_parts = a.db_rows;
                *db_at = ws;
            }
            if (!igemm2_launch<DIR_BWD_DATA>(a, mj, z, bwd_data_tiles(a.NI, mj, z), st)) return hipErrorInvalidValue;
            return hipGetLastError();
        }
    }
    if (relu_y != nullptr) return hipSuccess;
    return igemm_launch<T, DIR_BWD_DATA>(a, mj, s.sh * s.sw, vi, vj, st);
}

size_t conv_bwd_data_relu_ws_bytes(int dt, const ConvShape &s, int64_t dxs) {
    int G;
    int64_t ppb;
    relu_bwd_plan(dt, (int64_t)s.N * s.H * s.W, s.C, dxs, &G, &ppb);
    const size_t fallback = (size_t)G * s.C * sizeof(float);
    if (dt != 1) return fallback;
    return std::max({fallback, (size_t)relu_partial_rows(s) * s.C * sizeof(float), split_ws_bytes(dt, s, true)});
}

hipError_t launch_conv_bwd_data_relu(int dt, const void *dy, int64_t dys, const void *w, void *dpre, int64_t dxs,
                                     const void *y, float beta, float *db, float *ws, const ConvShape &s,
                                     hipStream_t st, BiasPartials *defer) {
    int parts = 0;
    float *db_at = nullptr;
    if (dt == 1 && ((uintptr_t)y & 7) == 0) {
        const hipError_t e = conv_bwd_data_t<bf16_t>(dy, dys, w, dpre, dxs, beta, s, st, ws, y, &parts, &db_at);
        if (e != hipSuccess) return e;
        if (parts > 0) {
            if (defer != nullptr) {
                defer->part = db_at;
                defer->rows = parts;
                return hipSuccess;
            }
            return launch_sum_partials(db_at, parts, s.C, db, st);
        }
    }
    // otherwise the two ops in sequence: the input gradient, then the ReLU backward in place
    const hipError_t e = launch_conv_bwd_data(dt, dy, dys, w, dpre, dxs, beta, s, nullptr, st);
    if (e != hipSuccess) return e;
    return launch_bias_relu_bwd(dt, y, dpre, dpre, (int64_t)s.N * s.H * s.W, s.C, dxs, db, ws, st, defer);
}

hipError_t launch_conv_bwd_data(int dt, const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs,
                                float beta, const ConvShape &s, float *ws, hipStream_t st) {
    return dt == 0 ? conv_bwd_data_t<float>(dy, dys, w, dx, dxs, beta, s, st, ws)
                   : conv_bwd_data_t<bf16_t>(dy, dys, w, dx, dxs, beta, s, st, ws);
}

}  // namespace tfk
