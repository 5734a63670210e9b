// Host-side launch of the implicit-GEMM kernel: tile choice, vector-path
// selection and grid shape.
#pragma once
#include "igemm.h"
#include "igemm2.h"
#include "kernels.h"

namespace tfk {

static inline bool aligned16p(const void *p) { return ((uintptr_t)p & 15) == 0; }

template <typename T, int DIR, int BI>
static void igemm_dispatch(const IgArgs &a, dim3 grid, bool vi, bool vj, hipStream_t st) {
    if (vi && vj)
        hipLaunchKernelGGL((igemm_kernel<T, DIR, BI, 128, true, true>), grid, dim3(256), 0, st, a);
    else if (vi)
        hipLaunchKernelGGL((igemm_kernel<T, DIR, BI, 128, true, false>), grid, dim3(256), 0, st, a);
    else if (vj)
        hipLaunchKernelGGL((igemm_kernel<T, DIR, BI, 128, false, true>), grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL((igemm_kernel<T, DIR, BI, 128, false, false>), grid, dim3(256), 0, st, a);
}

// I tile: 64 output channels when the direction has at most 64, else 128.
static inline int igemm_bi(int ni) { return ni <= 64 ? 64 : 128; }

template <typename T, int DIR>
static hipError_t igemm_launch(IgArgs &a, int mj, int zdim, bool vi, bool vj, hipStream_t st) {
    const int bi = igemm_bi(a.NI);
    a.tiles_i = (a.NI + bi - 1) / bi;
    const int tiles_j = (mj + 127) / 128;
    const dim3 grid((unsigned)(a.tiles_i * tiles_j), 1, (unsigned)zdim);
    if (bi == 64)
        igemm_dispatch<T, DIR, 64>(a, grid, vi, vj, st);
    else
        igemm_dispatch<T, DIR, 128>(a, grid, vi, vj, st);
    return hipGetLastError();
}

// Tile configuration of the pipelined bf16 kernel: BI x BJ output tile, waves per block,
// LDS stages.
struct Igemm2Tile {
    int bi, bj, nw, ns;
};

// Chosen from sweeps over the AlexNet/VGG layer shapes on MI355X.  Two 4-wave blocks
// share each CU (two LDS stages each; the 64-channel kernel fits three).  128-channel tiles
// pay when the channel count is a multiple of 128 and they give at least one block per CU
// (AlexNet conv4/conv5 forward: 57 -> 54 and 38 -> 36 us against 64-channel tiles), and
// 192-channel tiles likewise for multiples of 192 (AlexNet conv2 forward: 76 -> 64 us),
// otherwise 64-channel tiles.
static inline Igemm2Tile igemm2_tiles(int ni, int mj, int zdim) {
    const int64_t blocks_j = (int64_t)((mj + 127) / 128) * zdim;
    if (ni % 128 == 0 && (ni / 128) * blocks_j >= 256) {
        // 128-row tiles that leave most CUs with one block (AlexNet conv4/conv5: 338 blocks)
        // spread better as 96-row tiles, still within one round of two blocks per CU
        const int64_t b128 = (ni / 128) * blocks_j, b96 = (ni / 128) * (int64_t)((mj + 95) / 96) * zdim;
        // (not for a single row of tiles: 96-row tiles would leave most of the second row empty)
        if (b128 < 448 && b96 <= 512 && mj > 128) return {128, 96, 4, 2};
        return {128, 128, 4, 2};
    }
    if (ni % 192 == 0 && (ni / 192) * blocks_j >= 256) {
        // 96-row J tiles when they fill the last round of two blocks per CU better: the same
        // operand reuse per byte (192 x 96 tiles read 64 flop per copied byte, 96 x 48 wave
        // tiles 32 per LDS byte, as 128 x 128 tiles do) in more, smaller blocks (AlexNet conv2
        // forward, 93312 pixels: 729 blocks of 128 rows fill 71 % of two rounds, 972 of 96
        // rows 95 %; 73.4 -> 71.9 us back to back)
        const int64_t b128 = (ni / 192) * blocks_j, b96 = (ni / 192) * (int64_t)((mj + 95) / 96) * zdim;
        auto fill = [](int64_t b) { return (double)b / (double)(((b + 511) / 512) * 512); };
        if (zdim == 1 && fill(b96) > fill(b128) + 0.05) return {192, 96, 4, 2};
        return {192, 128, 4, 2};
    }
    return {64, 128, 4, 2};
}

// At most 32 output rows (channels) on the I side: 32-row tiles, which keep every MFMA row in use
// (a 64-row tile would compute half or more of its rows for nothing).
static inline Igemm2Tile igemm2_tiles_narrow(int ni, int mj, int zdim) {
    if (ni <= 32) return {32, 128, 4, 2};
    return igemm2_tiles(ni, mj, zdim);
}

template <int DIR, int BI, int BJ, int NW, int NS>
static void igemm2_go(const IgArgs &a, dim3 grid, hipStream_t st) {
    hipLaunchKernelGGL((igemm2_kernel<DIR, BI, BJ, NW, NS>), grid, dim3(NW * 64), 0, st, a);
}

// Launches one of the compiled configurations; false if t is not one of them.
template <int DIR>
static bool igemm2_launch(IgArgs &a, int mj, int zdim, const Igemm2Tile &t, hipStream_t st) {
    a.tiles_i = (a.NI + t.bi - 1) / t.bi;
    const int tiles_j = (mj + t.bj - 1) / t.bj;
    const dim3 grid((unsigned)(a.tiles_i * tiles_j), 1, (unsigned)zdim);
    const int key = ((t.bi / 64) << 12) | ((t.bj / 64) << 8) | (t.nw << 4) | t.ns;
    if (t.bi == 32 && t.bj == 128 && t.nw == 4 && t.ns == 2) {
        igemm2_go<DIR, 32, 128, 4, 2>(a, grid, st);
        return true;
    }
    if (t.bi == 128 && t.bj == 96 && t.nw == 4 && t.ns == 2) {
        // (96-row k-major tiles are not laid out: forward and bwd-input only)
        if constexpr (DIR == DIR_BWD_FILTER) return false;
        else { igemm2_go<DIR, 128, 96, 4, 2>(a, grid, st); return true; }
    }
    if (t.bj == 192 && t.nw == 4 && t.ns == 2) {
        // (192-row J tiles: the forward row bands of a fused max-pool and 64-channel forward
        // tiles; 192-row k-major tiles are not laid out)
        if constexpr (DIR == DIR_BWD_FILTER) return false;
        else {
            if (t.bi == 64) { igemm2_go<DIR, 64, 192, 4, 2>(a, grid, st); return true; }
            if (t.bi == 128) { igemm2_go<DIR, 128, 192, 4, 2>(a, grid, st); return true; }
            if (t.bi == 192) { igemm2_go<DIR, 192, 192, 4, 2>(a, grid, st); return true; }
            return false;
        }
    }
    if (t.bi == 192 && t.bj == 96 && t.nw == 4 && t.ns == 2) {
        if constexpr (DIR == DIR_BWD_FILTER) return false;
        else { igemm2_go<DIR, 192, 96, 4, 2>(a, grid, st); return true; }
    }
    if (t.bi == 192 && t.bj == 128 && t.nw == 4 && t.ns == 2) {
        // (the filter-gradient direction does not fit these tiles in its registers)
        if constexpr (DIR == DIR_BWD_FILTER) return false;
        else { igemm2_go<DIR, 192, 128, 4, 2>(a, grid, st); return true; }
    }
    switch (key) {
    case (1 << 12) | (2 << 8) | (8 << 4) | 3: igemm2_go<DIR, 64, 128, 8, 3>(a, grid, st); return true;
    case (1 << 12) | (4 << 8) | (8 << 4) | 3: igemm2_go<DIR, 64, 256, 8, 3>(a, grid, st); return true;
    case (2 << 12) | (2 << 8) | (8 << 4) | 3: igemm2_go<DIR, 128, 128, 8, 3>(a, grid, st); return true;
    case (2 << 12) | (4 << 8) | (8 << 4) | 3: igemm2_go<DIR, 128, 256, 8, 3>(a, grid, st); return true;
    case (2 << 12) | (2 << 8) | (4 << 4) | 2: igemm2_go<DIR, 128, 128, 4, 2>(a, grid, st); return true;
    case (1 << 12) | (2 << 8) | (4 << 4) | 3: igemm2_go<DIR, 64, 128, 4, 3>(a, grid, st); return true;
    case (1 << 12) | (2 << 8) | (4 << 4) | 2: igemm2_go<DIR, 64, 128, 4, 2>(a, grid, st); return true;
    case (1 << 12) | (4 << 8) | (4 << 4) | 2: igemm2_go<DIR, 64, 256, 4, 2>(a, grid, st); return true;
    default: return false;
    }
}

// Split-K for GEMMs with few output tiles (fully connected layers at small batch): the
// reduction is cut into ranges of whole 64-wide K tiles, one per blockIdx.z, so that about 256
// blocks run, each range keeping at least 8 K tiles.  Returns the number of ranges (1: no split)
// and sets k_split to the range length in reduction elements.
static inline int gemm_split_plan(int ni, int mj, int64_t kred, int *k_split) {
    const int64_t blocks = (int64_t)((ni + 127) / 128) * ((mj + 127) / 128);
    const int64_t ktiles = (kred + 63) / 64;
    const int64_t sp = std::min<int64_t>((256 + blocks - 1) / blocks, ktiles / 8);
    *k_split = 0;
    if (blocks >= 128 || sp < 2) return 1;
    const int64_t per = (ktiles + sp - 1) / sp;
    *k_split = (int)(per * 64);
    return (int)((ktiles + per - 1) / per);
}

// Bytes from the first element of a pixel-major bf16 operand to the end of its last
// pixel's channels.
static inline int64_t span_bytes(int64_t pixels, int64_t stride, int64_t ch) {
    return pixels > 0 ? ((pixels - 1) * stride + ch) * 2 : 0;
}

// The pipelined kernel addresses each operand with 32-bit byte offsets (offsets from 2^31
// up read as zeros) and keeps masks of a filter's valid rows and columns in 31 bits.
// Records the spans when they fit.
static inline bool igemm2_fits(IgArgs &a, int64_t span_i, int64_t span_j) {
    constexpr int64_t kLim = int64_t(1) << 31;
    if (span_i >= kLim || span_j >= kLim || a.KH > 31 || a.KW > 31) return false;
    a.bytes_i = (uint32_t)span_i;
    a.bytes_j = (uint32_t)span_j;
    return true;
}

static inline void fill_geom(IgArgs &a, const ConvShape &s) {
    a.N = s.N; a.H = s.H; a.W = s.W; a.C = s.C;
    a.OH = s.OH; a.OW = s.OW; a.K = s.K;
    a.KH = s.KH; a.KW = s.KW; a.sh = s.sh; a.sw = s.sw; a.pt = s.pt; a.pl = s.pl;
    a.dC.init((uint32_t)s.C);
    a.dKW.init((uint32_t)s.KW);
    a.dOW.init((uint32_t)s.OW);
    a.dOH.init((uint32_t)s.OH);
    a.dK.init((uint32_t)s.K);
    a.beta = 0.f;
    a.bias = nullptr;
    a.xcd_order = 1;
    a.k_split = 0;
    a.split_stride = 0;
    a.bytes_i = a.bytes_j = 0;
    a.relu_y = nullptr;
    a.db_part = nullptr;
    a.db_rows = 0;
    a.band_rows = a.band_step = a.bands_per_img = 0;
    a.pool_y = nullptr;
    a.pool_taps = nullptr;
    a.pkh = a.pkw = a.psh = a.psw = a.pOH = a.pOW = a.pool_rows = 0;
    a.pool_ys = 0;
}

}  // namespace tfk
