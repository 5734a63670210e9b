// Conv2DBackpropFilter on gfx950 MFMA: Out[(kh,kw,ci)][co] = sum_p x-gather[p][(kh,kw,ci)] * dy[p][co],
// the reduction over p = (n, oh, ow) split across blockIdx.z and summed in split order.
#include "igemm_launch.h"

namespace tfk {

void conv_bwd_filter_plan(int dt, const ConvShape &s, int *splits, int *k_split) {
    const int bk = dt == 0 ? 32 : 64;
    const int m = s.KH * s.KW * s.C;
    const int bi = igemm_bi(s.K);
    const int tiles = ((s.K + bi - 1) / bi) * ((m + 127) / 128);
    const int64_t ktot = (int64_t)s.N * s.OH * s.OW;
    const int64_t ktiles = (ktot + bk - 1) / bk;
    int64_t sp = (512 + tiles - 1) / tiles;            // about two blocks per CU
    const int64_t max_sp = std::max<int64_t>(1, ktiles / 8);   // at least 8 K tiles per split
    sp = std::max<int64_t>(1, std::min<int64_t>(sp, max_sp));
    sp = std::min<int64_t>(sp, 4096);
    int64_t per = (ktiles + sp - 1) / sp;              // K tiles per split
    *k_split = (int)(per * bk);
    *splits = (int)((ktiles + per - 1) / per);
}

size_t conv_bwd_filter_ws_bytes(int dt, const ConvShape &s) {
    int splits, k_split;
    conv_bwd_filter_plan(dt, s, &splits, &k_split);
    if (splits <= 1) return 0;
    return (size_t)splits * (size_t)s.KH * s.KW * s.C * s.K * sizeof(float);
}

template <typename T>
static hipError_t conv_bwd_filter_t(const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                    const ConvShape &s, void *ws, hipStream_t st) {
    constexpr int EPC = Elem<T>::kPerChunk;
    IgArgs a;
    fill_geom(a, s);
    int splits, k_split;
    conv_bwd_filter_plan(sizeof(T) == 4 ? 0 : 1, s, &splits, &k_split);
    const int64_t mn = (int64_t)s.KH * s.KW * s.C * s.K;
    a.src_i = dy;
    a.src_j = x;
    a.out = splits > 1 ? ws : (void *)dw;
    a.xs = xs;
    a.ys = dys;
    a.NI = s.K;
    a.k_split = k_split;
    a.split_stride = mn;
    const bool vi = s.K % EPC == 0 && dys % EPC == 0 && aligned16p(dy);
    const bool vj = s.C % EPC == 0 && xs % EPC == 0 && aligned16p(x);
    hipError_t e = igemm_launch<T, DIR_BWD_FILTER>(a, s.KH * s.KW * s.C, splits, vi, vj, st);
    if (e != hipSuccess || splits <= 1) return e;
    return launch_sum_splits(reinterpret_cast<const float *>(ws), splits, mn, dw, st);
}

hipError_t launch_conv_bwd_filter(int dt, const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                  const ConvShape &s, void *ws, hipStream_t st) {
    return dt == 0 ? conv_bwd_filter_t<float>(x, xs, dy, dys, dw, s, ws, st)
                   : conv_bwd_filter_t<bf16_t>(x, xs, dy, dys, dw, s, ws, st);
}

}  // namespace tfk
