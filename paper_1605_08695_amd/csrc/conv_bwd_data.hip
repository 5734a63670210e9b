// Conv2DBackpropInput on gfx950 MFMA, one stride phase per blockIdx.z:
// Out[p'][ci] = sum over the phase's taps (kh, kw) and co of dy[...][co] * w[kh][kw][ci][co].
#include "igemm_launch.h"

namespace tfk {

// Rows of bias-gradient partials of the fused ReLU-backward epilogue: one per block and wave
// column of the pipelined kernel's grid.
static int relu_partial_rows(const ConvShape &s) {
    const int mj = s.N * ((s.H + s.sh - 1) / s.sh) * ((s.W + s.sw - 1) / s.sw);
    const int z = s.sh * s.sw;
    const Igemm2Tile t = igemm2_tiles(s.C, mj, z);
    return z * ((mj + t.bj - 1) / t.bj) * (t.nw / 2);
}

// relu_y / db_part: the fused ReLU backward of the pipelined kernel (beta 0; false is returned
// when that kernel does not run, and nothing is launched then).
template <typename T>
static hipError_t conv_bwd_data_t(const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs, float beta,
                                  const ConvShape &s, hipStream_t st, const void *relu_y = nullptr,
                                  float *db_part = nullptr, bool *fused = nullptr) {
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
            if (relu_y != nullptr) {
                a.relu_y = relu_y;
                a.db_part = db_part;
                a.db_rows = relu_partial_rows(s);
                *fused = true;
            }
            if (!igemm2_launch<DIR_BWD_DATA>(a, mj, z, igemm2_tiles(a.NI, mj, z), st)) return hipErrorInvalidValue;
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
    return std::max(fallback, (size_t)relu_partial_rows(s) * s.C * sizeof(float));
}

hipError_t launch_conv_bwd_data_relu(int dt, const void *dy, int64_t dys, const void *w, void *dpre, int64_t dxs,
                                     const void *y, float *db, float *ws, const ConvShape &s, hipStream_t st) {
    bool fused = false;
    if (dt == 1 && ((uintptr_t)y & 7) == 0) {
        const hipError_t e = conv_bwd_data_t<bf16_t>(dy, dys, w, dpre, dxs, 0.f, s, st, y, ws, &fused);
        if (e != hipSuccess) return e;
        if (fused) return launch_sum_partials(ws, relu_partial_rows(s), s.C, db, st);
    }
    // otherwise the two ops in sequence: the input gradient, then the ReLU backward in place
    const hipError_t e = launch_conv_bwd_data(dt, dy, dys, w, dpre, dxs, 0.f, s, st);
    if (e != hipSuccess) return e;
    return launch_bias_relu_bwd(dt, y, dpre, dpre, (int64_t)s.N * s.H * s.W, s.C, dxs, db, ws, st);
}

hipError_t launch_conv_bwd_data(int dt, const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs,
                                float beta, const ConvShape &s, hipStream_t st) {
    return dt == 0 ? conv_bwd_data_t<float>(dy, dys, w, dx, dxs, beta, s, st)
                   : conv_bwd_data_t<bf16_t>(dy, dys, w, dx, dxs, beta, s, st);
}

}  // namespace tfk
