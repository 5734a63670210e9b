// Conv2D forward on gfx950 MFMA: Out[p][co] = sum_k im2col(x)[p][k] * w[k][co].
#include "igemm_launch.h"

namespace tfk {

template <typename T>
static hipError_t conv_fwd_t(const void *x, int64_t xs, const void *w, void *y, int64_t ys, const ConvShape &s,
                             const float *bias, hipStream_t st) {
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
    return dt == 0 ? conv_fwd_t<float>(x, xs, w, y, ys, s, bias, st)
                   : conv_fwd_t<bf16_t>(x, xs, w, y, ys, s, bias, st);
}

}  // namespace tfk
