// Conv2DBackpropInput on gfx950 MFMA, one stride phase per blockIdx.z:
// Out[p'][ci] = sum over the phase's taps (kh, kw) and co of dy[...][co] * w[kh][kw][ci][co].
#include "igemm_launch.h"

namespace tfk {

template <typename T>
static hipError_t conv_bwd_data_t(const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs, float beta,
                                  const ConvShape &s, hipStream_t st) {
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
            if (!igemm2_launch<DIR_BWD_DATA>(a, mj, z, igemm2_tiles(a.NI, mj, z), st)) return hipErrorInvalidValue;
            return hipGetLastError();
        }
    }
    return igemm_launch<T, DIR_BWD_DATA>(a, mj, s.sh * s.sw, vi, vj, st);
}

hipError_t launch_conv_bwd_data(int dt, const void *dy, int64_t dys, const void *w, void *dx, int64_t dxs,
                                float beta, const ConvShape &s, hipStream_t st) {
    return dt == 0 ? conv_bwd_data_t<float>(dy, dys, w, dx, dxs, beta, s, st)
                   : conv_bwd_data_t<bf16_t>(dy, dys, w, dx, dxs, beta, s, st);
}

}  // namespace tfk
