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
                if (!igemm2_launch<DIR_FWD>(a, mj, sp, igemm2_tiles_narrow(a.NI, mj, sp), st)) return hipErrorInvalidValue;
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
            if (!igemm2_launch<DIR_FWD>(a, mj, 1, igemm2_tiles_narrow(a.NI, mj, 1), st)) return hipErrorInvalidValue;
            return hipGetLastError();
        }
    }
    return igemm_launch<T, DIR_FWD>(a, mj, 1, vi, vj, st);
}

// Row bands of a forward convolution whose J tiles each hold whole windows of a VALID max-pool
// of its output: q pool rows per band need rows = (q - 1) * psh + pkh output rows of OW
// pixels (at most bj), consecutive bands start step = q * psh rows apart (sharing the rows
// their windows overlap on), and enough bands run to cover every pool row and every output row.
namespace {
constexpr int64_t kFusedPoolCUs = 256;  // MI355X compute units

struct BandPlan {
    int bj, q, rows, step, bands;
};

bool band_plan(const ConvShape &s, const PoolGeom &g, int bj, BandPlan &b) {
    int q = 0;
    while (q < g.OH && (q * g.sh + g.KH) * s.OW <= bj) ++q;
    if (q < 1) return false;
    b.bj = bj;
    b.q = q;
    b.rows = (q - 1) * g.sh + g.KH;
    b.step = q * g.sh;
    const int by_pool = (g.OH + q - 1) / q;
    const int by_rows = s.OH > b.rows ? (s.OH - b.rows + b.step - 1) / b.step + 1 : 1;
    b.bands = by_pool > by_rows ? by_pool : by_rows;
    return true;
}
}  // namespace

bool conv_fwd_pool_fused(const void *x, int64_t xs, const void *w, void *y, int64_t ys, const ConvShape &s,
                         const float *bias, const PoolGeom &g, void *py, int64_t pys, uint8_t *taps,
                         hipStream_t st, hipError_t *err) {
    *err = hipSuccess;
    // the pool reads exactly y (VALID, no padding), and the convolution takes the pipelined
    // bf16 path without a split
    if (g.pt != 0 || g.pl != 0 || g.N != s.N || g.H != s.OH || g.W != s.OW || g.C != s.K || g.xs != ys) return false;
    if (g.KH * g.KW > 256 || g.KH > s.OH || g.KW > s.OW) return false;
    // (no padding at the bottom or right either: every window lies inside y)
    if (g.OH != (s.OH - g.KH) / g.sh + 1 || g.OW != (s.OW - g.KW) / g.sw + 1) return false;
    if (conv_band_fwd_applies(s) || conv_fold_applies(1, s)) return false;
    if (s.K % 8 != 0 || s.C % 8 != 0 || xs % 8 != 0 || ys % 8 != 0 || pys % 2 != 0) return false;
    if (!aligned16p(w) || !aligned16p(x) || !aligned16p(y) || ((uintptr_t)py & 3) || ((uintptr_t)taps & 1))
        return false;
    int ks;
    if (fwd_splits(s, &ks) > 1) return false;
    BandPlan best{}, b{};
    bool have = false;
    for (int bj : {128, 192}) {
        if (band_plan(s, g, bj, b) && (!have || (int64_t)b.bands * b.bj < (int64_t)best.bands * best.bj)) {
            best = b;
            have = true;
        }
    }
    if (!have) return false;
    // Bands cost recomputed rows (windows that overlap across bands) and tile rows past the band's
    // pixels; fused only when that adds at most 15 % to the output rows (measured on AlexNet:
    // conv5 + pool5, 13 x 13, one band of 169 of 192 rows: 42.6 -> 41.3 us; conv2 + pool2, 27 x 27,
    // 5 bands of 189 of 192 rows with a shared row between bands, 32 % more rows: 84 -> 118 us).
    if ((int64_t)best.bands * best.bj * 100 > (int64_t)s.OH * s.OW * 115) return false;
    // and only when the unfused convolution runs as one round of two blocks per CU, whose last
    // blocks set its time and absorb the extra rows: over several rounds they add their share to
    // every round and cost more than the separate pool pass (VGG-16 b64, conv7 + pool3, 56 x 56 x
    // 256, and conv10 + pool4, 28 x 28 x 512, each 14 % more rows: 298 -> 364 and 287 -> 341 us
    // fused with 64-channel tiles, 322 and 292 us with 128-channel tiles)
    {
        const int mj_plain = s.N * s.OH * s.OW;
        const Igemm2Tile pt = igemm2_tiles_narrow(s.K, mj_plain, 1);
        const int64_t blocks = (int64_t)((s.K + pt.bi - 1) / pt.bi) * ((mj_plain + pt.bj - 1) / pt.bj);
        if (blocks > 2 * kFusedPoolCUs) return false;
    }
    IgArgs a;
    fill_geom(a, s);
    a.src_i = w;
    a.src_j = x;
    a.out = y;
    a.xs = xs;
    a.ys = ys;
    a.NI = s.K;
    a.bias = bias;
    const int64_t wb = (int64_t)s.KH * s.KW * s.C * s.K * 2;
    if (!igemm2_fits(a, wb, span_bytes((int64_t)s.N * s.H * s.W, xs, s.C))) return false;
    a.band_rows = best.rows;
    a.band_step = best.step;
    a.bands_per_img = best.bands;
    a.pool_y = py;
    a.pool_taps = taps;
    a.pkh = g.KH;
    a.pkw = g.KW;
    a.psh = g.sh;
    a.psw = g.sw;
    a.pOH = g.OH;
    a.pOW = g.OW;
    a.pool_rows = best.q;
    a.pool_ys = pys;
    const int bi = 64;       // 64-channel tiles: two blocks per CU (fastest of 64/128/192 on the cases above)
    const int mj = s.N * best.bands * best.bj;      // one J tile per (image, band)
    if (!igemm2_launch<DIR_FWD>(a, mj, 1, Igemm2Tile{bi, best.bj, 4, 2}, st)) return false;
    *err = hipGetLastError();
    return true;
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
