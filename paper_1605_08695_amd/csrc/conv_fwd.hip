// Conv2D forward on gfx950 MFMA: Out[p][co] = sum_k im2col(x)[p][k] * w[k][co].
#include "igemm_launch.h"

namespace tfk {

// Split-K (fp32 partials in the workspace, then one epilogue pass) for convolutions with few
// output tiles: the fully connected layers (flattened to 1 x 1 convolutions) and the small
// images of late stages at small batch.
static int fwd_splits(const ConvShape &s, int *k_split) {
    return gemm_split_plan(s.K, s.N * s.OH * s.OW, (int64_t)s.KH * s.KW * s.C, k_split);
}

size_t conv_fwd_split_ws_bytes(int dt, const ConvShape &s) {
    int ks;
    const int sp = fwd_splits(s, &ks);
    if (dt != 1 || sp <= 1) return 0;
    return (size_t)sp * s.N * s.OH * s.OW * s.K * sizeof(float);
}

template <typename T>
static hipError_t conv_fwd_t(const void *x, int64_t xs, const void *w, void *y, int64_t ys, const ConvShape &s,
                             const float *bias, void *ws, hipStream_t st) {
    constexpr int EPC = Elem<T>::kPerChunk;
    IgArgs a;
    fill_geom(a, s);
    a.src_i = w;
    a.src_j = x;
    a.out = y;
    a.xs = xs;
    a.ys = ys;
    a.NI = s.K;
    a.bias = bias;
    const bool vi = s.K % EPC == 0 && aligned16p(w);
    const bool vj = s.C % EPC == 0 && xs % EPC == 0 && aligned16p(x);
    const int mj = s.N * s.OH * s.OW;
    if constexpr (sizeof(T) == 2) {
        const int64_t wb = (int64_t)s.KH * s.KW * s.C * s.K * 2;
        if (vi && vj && ys % 8 == 0 && aligned16p(y) &&
            igemm2_fits(a, wb, span_bytes((int64_t)s.N * s.H * s.W, xs, s.C))) {
            int ks;
            const int sp = ws != nullptr && aligned16p(ws) ? fwd_splits(s, &ks) : 1;
            if (sp > 1) {
                a.k_split = ks;
                a.split_stride = (int64_t)mj * a.NI;
                a.out = ws;
                if (!igemm2_launch<DIR_FWD>(a, mj, sp, igemm2_tiles(a.NI, mj, sp), st)) return hipErrorInvalidValue;
                const hipError_t e = hipGetLastError();
                if (e != hipSuccess) return e;
                SplitEpi ep{};
                ep.part = reinterpret_cast<const float *>(ws);
                ep.splits = sp;
                ep.rows = mj;
                ep.ni = a.NI;
                ep.split_stride = a.split_stride;
                ep.ostride = ys;
                ep.out = y;
                ep.bias = bias;
                return launch_split_epilogue(ep, st);
            }
            if (!igemm2_launch<DIR_FWD>(a, mj, 1, igemm2_tiles(a.NI, mj, 1), st)) return hipErrorInvalidValue;
            return hipGetLastError();
        }
    }
    return igemm_launch<T, DIR_FWD>(a, mj, 1, vi, vj, st);
}

hipError_t launch_conv_fwd(int dt, const void *x, int64_t xs, const void *w, void *y, int64_t ys,
                           const ConvShape &s, const float *bias, void *ws, hipStream_t st) {
    if (dt == 1 && ws != nullptr && conv_band_fwd_applies(s) && aligned16p(w) && ((uintptr_t)y & 7) == 0 &&
        ys % 4 == 0) {
        const bf16_t *x4 = rgbx_input(x, (int64_t)s.N * s.H * s.W, s.C, xs, reinterpret_cast<bf16_t *>(ws), st);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        return launch_conv_fwd_band(x4, w, y, ys, s, bias, st);
    }
    if (ws != nullptr && conv_fold_applies(dt, s) && ((uintptr_t)y & 15) == 0 && ys % 8 == 0)
        return launch_conv_fwd_folded(x, xs, w, y, ys, s, bias, ws, st);
    return dt == 0 ? conv_fwd_t<float>(x, xs, w, y, ys, s, bias, ws, st)
                   : conv_fwd_t<bf16_t>(x, xs, w, y, ys, s, bias, ws, st);
}

}  // namespace tfk
