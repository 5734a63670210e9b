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

// Tiles of the pipelined bf16 kernel (one block per CU), chosen from a sweep over the
// AlexNet/VGG layer shapes on MI355X: 128-channel I tiles when the channel count is a
// multiple of 128 (else 64, so 192 channels waste nothing), paired with 256-row J tiles;
// 64-channel tiles take 256 rows only when that fits one round of blocks on the 256 CUs.
static inline void igemm2_tiles(int ni, int mj, int zdim, int *bi, int *bj) {
    *bi = (ni % 128 == 0) ? 128 : 64;
    if (*bi == 128) {
        *bj = 256;
        return;
    }
    const int ti = (ni + 63) / 64;
    const int64_t blocks256 = (int64_t)ti * ((mj + 255) / 256) * zdim;
    *bj = blocks256 <= 256 ? 256 : 128;
}

template <int DIR>
static hipError_t igemm2_launch(IgArgs &a, int mj, int zdim, int bi, int bj, hipStream_t st) {
    a.tiles_i = (a.NI + bi - 1) / bi;
    const int tiles_j = (mj + bj - 1) / bj;
    const dim3 grid((unsigned)(a.tiles_i * tiles_j), 1, (unsigned)zdim);
    if (bi == 64 && bj == 128)
        hipLaunchKernelGGL((igemm2_kernel<DIR, 64, 128>), grid, dim3(512), 0, st, a);
    else if (bi == 64)
        hipLaunchKernelGGL((igemm2_kernel<DIR, 64, 256>), grid, dim3(512), 0, st, a);
    else if (bj == 128)
        hipLaunchKernelGGL((igemm2_kernel<DIR, 128, 128>), grid, dim3(512), 0, st, a);
    else
        hipLaunchKernelGGL((igemm2_kernel<DIR, 128, 256>), grid, dim3(512), 0, st, a);
    return hipGetLastError();
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
    a.k_split = 0;
    a.split_stride = 0;
}

}  // namespace tfk
