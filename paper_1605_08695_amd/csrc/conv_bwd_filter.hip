// Conv2DBackpropFilter on gfx950 MFMA: Out[(kh,kw,ci)][co] = sum_p x-gather[p][(kh,kw,ci)] * dy[p][co],
// the reduction over p = (n, oh, ow) split across blockIdx.z and summed in split order.
#include "igemm_launch.h"

namespace tfk {

namespace {

struct BwfPlan {
    int bi, bj, splits, k_split;
    Igemm2Tile t;      // configuration of the pipelined bf16 kernel
};

// Tiles and split-K of one bwd-filter launch, chosen from sweeps over the AlexNet/VGG
// shapes: 128 x 128 tiles (even for 192 output channels, where the second channel tile
// is half empty) and the pixel reduction split into as many parts as keep the blocks within
// one full round of two blocks per CU (512 blocks): a last round with only a few blocks
// costs a whole block time, and more splits only add partial-sum traffic (AlexNet conv2-5:
// 357 us with four-block rounds, 297 us with this rule; the sustained two-stream AlexNet step
// 0.686 ms, against 0.694 with 384 blocks for the short launches).
// 64-channel layers take 64 x 128
// tiles, layers of at most 32 output channels 32 x 128, multiples of 64 that are not of 128 64 x 128.  (192-channel tiles, which pay in the
// forward pass, need more registers here than two waves per SIMD have and spill.)
BwfPlan bwf_plan(int dt, const ConvShape &s, bool v2) {
    BwfPlan p;
    const int bk = dt == 0 ? 32 : 64;
    const int m = s.KH * s.KW * s.C;
    // output channels a multiple of 64 but not of 128 (AlexNet conv2's 192): 64-channel tiles leave
    // none empty (128-channel ones would compute a quarter of the rows for nothing), and three of
    // their 48 KiB blocks fit a CU, so the splits fill one round of three (conv2: 95 -> 90 us)
    const bool by64 = v2 && s.K > 64 && s.K % 128 != 0 && s.K % 64 == 0;
    if (v2) {
        p.t = s.K > 64 && !by64 ? Igemm2Tile{128, 128, 4, 2}
                                : (s.K > 32 ? Igemm2Tile{64, 128, 4, 2} : Igemm2Tile{32, 128, 4, 2});
        p.bi = p.t.bi;
        p.bj = p.t.bj;
    } else {
        p.bi = igemm_bi(s.K);
        p.bj = 128;
    }
    const int tiles = ((s.K + p.bi - 1) / p.bi) * ((m + p.bj - 1) / p.bj);
    const int64_t ktot = (int64_t)s.N * s.OH * s.OW;
    const int64_t ktiles = (ktot + bk - 1) / bk;
    const int target = by64 ? 768 : 512;
    int64_t sp = target / tiles;
    const int64_t max_sp = std::max<int64_t>(1, ktiles / 8);   // at least 8 K tiles per split
    sp = std::max<int64_t>(1, std::min<int64_t>(sp, max_sp));
    sp = std::min<int64_t>(sp, 4096);
    const int64_t per = (ktiles + sp - 1) / sp;                 // K tiles per split
    p.k_split = (int)(per * bk);
    p.splits = (int)((ktiles + per - 1) / per);
    return p;
}

size_t plan_ws(const ConvShape &s, const BwfPlan &p) {
    if (p.splits <= 1) return 0;
    return (size_t)p.splits * (size_t)s.KH * s.KW * s.C * s.K * sizeof(float);
}

// Workspace bytes ahead of the band kernel's partials: room for a 4-channel copy of x.
size_t band_x_bytes(const ConvShape &s) { return ((size_t)s.N * s.H * s.W * 8 + 255) & ~(size_t)255; }

}  // namespace

void conv_bwd_filter_plan(int dt, const ConvShape &s, int *splits, int *k_split) {
    const BwfPlan p = bwf_plan(dt, s, false);
    *splits = p.splits;
    *k_split = p.k_split;
}

size_t conv_bwd_filter_ws_bytes(int dt, const ConvShape &s) {
    size_t need = plan_ws(s, bwf_plan(dt, s, false));
    if (dt == 1) need = std::max(need, plan_ws(s, bwf_plan(dt, s, true)));
    if (conv_fold_applies(dt, s)) need = std::max(need, conv_fold_ws_bytes(2, s));
    if (dt == 1 && conv_band_bwf_applies(s)) need = std::max(need, band_x_bytes(s) + conv_band_bwf_partial_bytes(s));
    return need;
}

template <typename T>
static hipError_t conv_bwd_filter_t(const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                    const ConvShape &s, void *ws, hipStream_t st) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const int dti = sizeof(T) == 4 ? 0 : 1;
    IgArgs a;
    fill_geom(a, s);
    const int64_t mn = (int64_t)s.KH * s.KW * s.C * s.K;
    const int m = s.KH * s.KW * s.C;
    a.src_i = dy;
    a.src_j = x;
    a.xs = xs;
    a.ys = dys;
    a.NI = s.K;
    a.split_stride = mn;
    const bool vi = s.K % EPC == 0 && dys % EPC == 0 && aligned16p(dy);
    const bool vj = s.C % EPC == 0 && xs % EPC == 0 && aligned16p(x);
    hipError_t e;
    BwfPlan p;
    bool v2 = false;
    if constexpr (sizeof(T) == 2) {
        if (vi && vj && igemm2_fits(a, span_bytes((int64_t)s.N * s.OH * s.OW, dys, s.K),
                                    span_bytes((int64_t)s.N * s.H * s.W, xs, s.C))) {
            p = bwf_plan(dti, s, true);
            v2 = p.splits > 1 || aligned16p(dw);
        }
    }
    if (v2) {
        a.out = p.splits > 1 ? ws : (void *)dw;
        a.k_split = p.k_split;
        // (each XCD runs a contiguous range of a split's tiles: they read the same pixel range of
        // x and dy, from one L2; AlexNet conv2-5: 232 -> 228 us)
        a.xcd_order = 1;
        e = igemm2_launch<DIR_BWD_FILTER>(a, m, p.splits, p.t, st) ? hipGetLastError() : hipErrorInvalidValue;
    } else {
        p = bwf_plan(dti, s, false);
        a.out = p.splits > 1 ? ws : (void *)dw;
        a.k_split = p.k_split;
        e = igemm_launch<T, DIR_BWD_FILTER>(a, m, p.splits, vi, vj, st);
    }
    if (e != hipSuccess || p.splits <= 1) return e;
    return launch_sum_splits(reinterpret_cast<float *>(ws), p.splits, mn, dw, st);
}

hipError_t launch_conv_bwd_filter(int dt, const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                  const ConvShape &s, void *ws, hipStream_t st) {
    if (dt == 1 && conv_band_bwf_applies(s) && dys % 8 == 0 && aligned16p(dy) && aligned16p(ws)) {
        const int64_t npix = (int64_t)s.N * s.H * s.W;
        unsigned char *base = reinterpret_cast<unsigned char *>(ws);
        const bf16_t *x4 = rgbx_input(x, npix, s.C, xs, reinterpret_cast<bf16_t *>(base), st);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        float *part = reinterpret_cast<float *>(base + band_x_bytes(s));
        return launch_conv_bwd_filter_band(x4, dy, dys, dw, s, part, st);
    }
    if (conv_fold_applies(dt, s) && dys % 8 == 0 && ((uintptr_t)dy & 15) == 0 && ((uintptr_t)ws & 15) == 0)
        return launch_conv_bwd_filter_folded(x, xs, dy, dys, dw, s, ws, st);
    return dt == 0 ? conv_bwd_filter_t<float>(x, xs, dy, dys, dw, s, ws, st)
                   : conv_bwd_filter_t<bf16_t>(x, xs, dy, dys, dw, s, ws, st);
}

}  // namespace tfk
