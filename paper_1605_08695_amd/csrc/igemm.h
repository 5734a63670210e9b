// Implicit-GEMM convolution on gfx950 matrix cores (MFMA), all three directions.
//
// Each direction of the cross-correlation y = x (*) w is a matrix product with
// the operands gathered on the fly from the NHWC / HWIO tensors (no im2col
// buffer in memory):
//
//   forward      Out[p][co]    = sum_k Xg[p][k]  * Wt[co][k]     p = (n,oh,ow), k = (kh,kw,ci)
//   bwd-input    Out[p'][ci]   = sum_k DYg[p'][k] * Wg[ci][k]    p' = dx pixel, k = (kh,kw,co)
//   bwd-filter   Out[r][co]    = sum_k Xg[k][r]  * DY[k][co]     r = (kh,kw,ci), k = (n,oh,ow)
//
// In the kernel the "I" side is the output-channel axis (contiguous in memory
// in every output) and the "J" side is the row axis (pixels, or filter taps).
// Both MFMA operands want eight (bf16) or four (fp32) consecutive k values of
// one row per lane, i.e. a 16-byte k-chunk.  Tiles are therefore kept in LDS
// as [row][k-chunk] with 8 chunks (128 bytes) per row; the chunk index is
// XOR-swizzled with (row & 7) so that the 16-byte MFMA fragment reads of 8
// consecutive rows and the staging writes are free of bank conflicts.
//
// Operands whose memory layout is already k-contiguous (the im2col rows of x in
// the forward pass, the dy gather and the filter in bwd-input) are copied as
// 16-byte chunks.  Operands that are contiguous along the row axis instead (the
// filter in the forward pass, both operands of bwd-filter) are transposed in
// registers: each thread loads an EPC x EPC block (EPC k-rows of EPC
// elements), transposes it and writes EPC chunks.
//
// Strided bwd-input uses a stride-phase decomposition: the dx pixels with the
// same (h + pad_top) mod s_h and (w + pad_left) mod s_w receive exactly the
// taps kh = r_h + s_h * j_h (and likewise for kw); blockIdx.z selects the
// phase, so no MFMA work is spent on the zeros of a dilated dy.
//
// bwd-filter splits its long reduction (N*OH*OW) over blockIdx.z; each split
// writes an fp32 partial product that a second kernel sums in split order.
//
// Pipelining: two LDS stages; the global loads of K-tile t+1 are in flight
// while the MFMAs of tile t run, then the staged registers go to the other LDS
// stage and one barrier closes the iteration.
#pragma once
#include "common.h"

namespace tfk {

enum ConvDir { DIR_FWD = 0, DIR_BWD_DATA = 1, DIR_BWD_FILTER = 2 };

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;

struct IgArgs {
    const void *src_i;   // FWD: w (HWIO)   BWD_DATA: w (HWIO)   BWD_FILTER: dy
    const void *src_j;   // FWD: x          BWD_DATA: dy         BWD_FILTER: x
    void *out;           // FWD: y          BWD_DATA: dx         BWD_FILTER: fp32 dw / partials
    float beta;          // BWD_DATA: 0 overwrite, 1 accumulate
    const float *bias;   // FWD: when set, y = max(conv + bias[co], +0) (bias + ReLU fused)
    int xcd_order;       // pipelined kernel: 1 = give each XCD a contiguous range of logical blocks
    // forward-convolution geometry
    int N, H, W, C;      // input extents
    int OH, OW, K;       // output extents, K = output channels
    int KH, KW, sh, sw, pt, pl;
    int64_t xs;          // pixel stride (elements) of x (FWD, BWD_FILTER) or dx (BWD_DATA)
    int64_t ys;          // pixel stride of y (FWD) or dy (BWD_DATA, BWD_FILTER)
    // GEMM view
    int NI;              // I extent (output channels of this direction)
    int tiles_i;         // number of I tiles (blockIdx.x = tj * tiles_i + ti)
    int k_split;         // BWD_FILTER: reduction elements per split (multiple of the K tile)
    int64_t split_stride;// BWD_FILTER: floats between consecutive partial outputs
    FastDiv dC, dKW, dOW, dOH, dK;
    uint32_t bytes_i, bytes_j;   // pipelined kernel: byte spans of src_i / src_j (each < 2^31)
    // pipelined BWD_DATA with beta 0: when relu_y is set, the ReLU backward of the layer that produced
    // x is applied (out = relu_y > 0 ? dx : +0, relu_y with dx's layout) and per-channel sums of
    // the stored values go to db_part[c * db_rows + row] (row: block and wave column)
    const void *relu_y;
    float *db_part;
    int db_rows;
    // pipelined FWD, row bands (band_rows > 0): J tile tj covers output rows r0 .. r0 + band_rows - 1
    // (clipped to OH, r0 = (tj % bands_per_img) * band_step) of image tj / bands_per_img, all columns;
    // consecutive bands may share rows (each computes and stores them, the same values)
    int band_rows, band_step, bands_per_img;
    // with row bands, a VALID max-pool of the band's ReLU output (pool_y set): pool rows
    // q0 .. q0 + pool_rows - 1 of the band (q0 = band * pool_rows) are written to pool_y (pixel
    // stride pool_ys, same element type) with the selected window tap kh * pkw + kw in pool_taps
    // (dense uint8 [N][pOH][pOW][K]); the first maximum in (kh, kw) order wins
    void *pool_y;
    unsigned char *pool_taps;
    int pkh, pkw, psh, psw, pOH, pOW, pool_rows;
    int64_t pool_ys;
};

template <typename T> struct Mfma;
template <> struct Mfma<bf16_t> {
    __device__ __forceinline__ static void run(f32x4_t &acc, const U4 &a, const U4 &b) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                      __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
    }
};
template <> struct Mfma<float> {
    // One 16-byte chunk holds four k values: four 16x16x4 products, one per k.
    __device__ __forceinline__ static void run(f32x4_t &acc, const U4 &a, const U4 &b) {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    }
};

__device__ __forceinline__ U4 zero4() { U4 z; z.x = z.y = z.z = z.w = 0u; return z; }

__device__ __forceinline__ U4 ld16(const void *p) { return *reinterpret_cast<const U4 *>(p); }

// One element's bits (bf16 in the low half, or the fp32 word).
template <typename T>
__device__ __forceinline__ uint32_t ld_elem(const T *p) { return Elem<T>::bits(p); }

// Set element e of a 16-byte chunk from raw element bits.
template <typename T>
__device__ __forceinline__ void chunk_set(U4 &v, int e, uint32_t bits) {
    uint32_t *w = reinterpret_cast<uint32_t *>(&v);
    if constexpr (sizeof(T) == 4) {
        w[e] = bits;
    } else {
        const int s = (e & 1) * 16;
        w[e >> 1] = (w[e >> 1] & ~(0xffffu << s)) | (bits << s);
    }
}

// Transpose an EPC x EPC block: in[e] holds EPC row values at k = e;
// out[r] receives the EPC k values of row r.
template <typename T>
__device__ __forceinline__ void transpose_block(const U4 *in, U4 *out) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t *a0 = reinterpret_cast<const uint32_t *>(&in[0]);
            const uint32_t *a1 = reinterpret_cast<const uint32_t *>(&in[1]);
            const uint32_t *a2 = reinterpret_cast<const uint32_t *>(&in[2]);
            const uint32_t *a3 = reinterpret_cast<const uint32_t *>(&in[3]);
            out[r].x = a0[r]; out[r].y = a1[r]; out[r].z = a2[r]; out[r].w = a3[r];
        }
    } else {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            uint32_t o[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t lo = reinterpret_cast<const uint32_t *>(&in[2 * j])[r >> 1];
                const uint32_t hi = reinterpret_cast<const uint32_t *>(&in[2 * j + 1])[r >> 1];
                o[j] = (r & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
            }
            out[r].x = o[0]; out[r].y = o[1]; out[r].z = o[2]; out[r].w = o[3];
        }
    }
}

__device__ __forceinline__ int lds_off(int row, int chunk) {
    return row * 128 + ((chunk ^ (row & 7)) << 4);
}

template <typename T, int DIR, int BI, int BJ, bool VI, bool VJ>
__global__ __launch_bounds__(256) void igemm_kernel(const IgArgs a) {
    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int BKC = 8;                 // K tile, in 16-byte chunks
    constexpr int BK = BKC * EPC;          // K tile, in elements
    constexpr int NT = 256;
    constexpr int WAVES_I = (BI >= 64) ? 2 : 1;
    constexpr int WAVES_J = 4 / WAVES_I;
    constexpr int WI = BI / WAVES_I, WJ = BJ / WAVES_J;
    constexpr int MI = WI / 16, MJ = WJ / 16;
    constexpr int TI_BYTES = BI * BKC * 16, TJ_BYTES = BJ * BKC * 16;
    constexpr int STAGE = TI_BYTES + TJ_BYTES;

    // operand loader shapes
    constexpr bool TRANS_I = (DIR == DIR_FWD) || (DIR == DIR_BWD_FILTER);
    constexpr bool TRANS_J = (DIR == DIR_BWD_FILTER);
    constexpr int DR_I = BI * BKC / NT;                    // direct: chunks per thread
    constexpr int DR_J = BJ * BKC / NT;
    constexpr int TU_I = (BI / EPC) * BKC;                 // transposed: units in the tile
    constexpr int TU_J = (BJ / EPC) * BKC;
    constexpr int TN_I = (TU_I + NT - 1) / NT;             // transposed: units per thread
    constexpr int TN_J = (TU_J + NT - 1) / NT;
    constexpr int SI = TRANS_I ? TN_I * EPC : DR_I;        // staged chunks per thread
    constexpr int SJ = TRANS_J ? TN_J * EPC : DR_J;
    static_assert(DR_I * NT == BI * BKC && DR_J * NT == BJ * BKC, "tile/thread mismatch");

    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int ti = blockIdx.x % a.tiles_i;
    const int tj = blockIdx.x / a.tiles_i;
    const int i0 = ti * BI;
    const int j0 = tj * BJ;
    const int cc = tid & 7;                // chunk column of the direct loaders

    const T *__restrict__ srcI = reinterpret_cast<const T *>(a.src_i);
    const T *__restrict__ srcJ = reinterpret_cast<const T *>(a.src_j);

    // ------------------------------------------------------------ direction set-up
    int MJ_ext;                  // J extent of this block's problem
    int k_beg = 0, k_end;        // reduction range
    // BWD_DATA phase geometry
    int rh = 0, rw = 0, h0 = 0, w0 = 0, Hp = 1, Wp = 1, offh = 0, offw = 0, KHp = 1, KWp = 1;
    if constexpr (DIR == DIR_FWD) {
        MJ_ext = a.N * a.OH * a.OW;
        k_end = a.KH * a.KW * a.C;
    } else if constexpr (DIR == DIR_BWD_DATA) {
        const int z = blockIdx.z;
        rh = z / a.sw;
        rw = z - rh * a.sw;
        h0 = ((rh - a.pt) % a.sh + a.sh) % a.sh;
        w0 = ((rw - a.pl) % a.sw + a.sw) % a.sw;
        Hp = h0 < a.H ? (a.H - h0 + a.sh - 1) / a.sh : 0;
        Wp = w0 < a.W ? (a.W - w0 + a.sw - 1) / a.sw : 0;
        offh = (h0 + a.pt - rh) / a.sh;
        offw = (w0 + a.pl - rw) / a.sw;
        KHp = rh < a.KH ? (a.KH - rh + a.sh - 1) / a.sh : 0;
        KWp = rw < a.KW ? (a.KW - rw + a.sw - 1) / a.sw : 0;
        MJ_ext = a.N * Hp * Wp;
        k_end = KHp * KWp * a.K;
    } else {
        MJ_ext = a.KH * a.KW * a.C;
        const int ktot = a.N * a.OH * a.OW;
        k_beg = blockIdx.z * a.k_split;
        k_end = min(ktot, k_beg + a.k_split);
    }
    if (j0 >= MJ_ext) return;
    const int nk = k_end > k_beg ? (k_end - k_beg + BK - 1) / BK : 0;

    // ------------------------------------------------------------ loader state
    U4 stI[SI], stJ[SJ];

    // Direct loaders: thread rows (tid >> 3) + 32 * r, chunk column cc.
    // FWD J rows = output pixels; BWD_DATA J rows = dx pixels of the phase.
    int64_t jbase[DR_J];
    int jy0[DR_J], jx0[DR_J];
    bool jok[DR_J];
    if constexpr (DIR == DIR_FWD || DIR == DIR_BWD_DATA) {
#pragma unroll
        for (int r = 0; r < DR_J; ++r) {
            const int m = j0 + (tid >> 3) + 32 * r;
            jok[r] = m < MJ_ext;
            const int mm = jok[r] ? m : 0;
            if constexpr (DIR == DIR_FWD) {
                const int ow = mm % a.OW;
                const int t = mm / a.OW;
                const int oh = t % a.OH;
                const int n = t / a.OH;
                jbase[r] = (int64_t)n * a.H * a.W;
                jy0[r] = oh * a.sh - a.pt;
                jx0[r] = ow * a.sw - a.pl;
            } else {
                const int tw = mm % Wp;
                const int t = mm / Wp;
                const int th = t % Hp;
                const int n = t / Hp;
                jbase[r] = (int64_t)n * a.OH * a.OW;
                jy0[r] = th + offh;        // oh = jy0 - jh
                jx0[r] = tw + offw;        // ow = jx0 - jw
            }
        }
    }
    // Incremental decomposition of this thread's chunk-start k (direct loaders).
    // FWD: k = (kh, kw, ci) over (KH, KW, C).  BWD_DATA: k = (jh, jw, co) over (KHp, KWp, K).
    int kq0 = 0, kq1 = 0, kq2 = 0;   // outer, middle, inner
    int kInner = 1, kMid = 1;
    if constexpr (DIR == DIR_FWD) { kInner = a.C; kMid = a.KW; }
    if constexpr (DIR == DIR_BWD_DATA) { kInner = a.K; kMid = KWp; }
    if constexpr (DIR == DIR_FWD || DIR == DIR_BWD_DATA) {
        const int k = cc * EPC;
        kq2 = k % kInner;
        const int t = k / kInner;
        kq1 = kMid > 0 ? t % kMid : 0;
        kq0 = kMid > 0 ? t / kMid : 0;
    }
    auto advance_k = [&]() {
        kq2 += BK;
        while (kq2 >= kInner) {
            kq2 -= kInner;
            if (++kq1 == kMid) { kq1 = 0; ++kq0; }
        }
    };

    // BWD_FILTER J rows (filter taps r = (kh, kw, ci)): per transposed unit.
    int fr_dh[TN_J], fr_dw[TN_J], fr_ci[TN_J];
    bool fr_ok[TN_J];
    if constexpr (DIR == DIR_BWD_FILTER) {
#pragma unroll
        for (int u = 0; u < TN_J; ++u) {
            const int unit = tid + NT * u;
            const int rg = unit >> 3;
            const int r0 = j0 + rg * EPC;
            fr_ok[u] = unit < TU_J && r0 < MJ_ext;
            const int rr = fr_ok[u] ? r0 : 0;
            const int ci = rr % a.C;
            const int t = rr / a.C;
            fr_ci[u] = ci;
            fr_dw[u] = t % a.KW - a.pl;
            fr_dh[u] = t / a.KW - a.pt;
        }
    }

    // ------------------------------------------------------------ fetch (global -> registers)
    auto fetch = [&](int kt) {
        const int kt0 = k_beg + kt * BK;
        // ---------------- I operand
        if constexpr (DIR == DIR_FWD || DIR == DIR_BWD_FILTER) {
            // transposed: source [k][co] with co contiguous (FWD: HWIO filter, BWD_FILTER: dy pixels)
            const int64_t ld = (DIR == DIR_FWD) ? (int64_t)a.K : a.ys;
#pragma unroll
            for (int u = 0; u < TN_I; ++u) {
                const int unit = tid + NT * u;
                const int kg = unit & 7, rg = unit >> 3;
                const int co = i0 + rg * EPC;
                const bool uok = (TU_I >= NT * (u + 1) || unit < TU_I) && co < a.NI;
                U4 v[EPC];
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const int k = kt0 + kg * EPC + e;
                    const bool ok = uok && k < k_end;
                    const T *p = srcI + (int64_t)k * ld + co;
                    if constexpr (VI) {
                        v[e] = ok ? ld16(p) : zero4();
                    } else {
                        v[e] = zero4();
#pragma unroll
                        for (int q = 0; q < EPC; ++q)
                            if (ok && co + q < a.NI) chunk_set<T>(v[e], q, ld_elem<T>(p + q));
                    }
                }
                transpose_block<T>(v, &stI[u * EPC]);
            }
        } else {
            // BWD_DATA: direct, rows = ci, k = (jh, jw, co): w[rh + sh*jh][rw + sw*jw][ci][co..]
#pragma unroll
            for (int r = 0; r < DR_I; ++r) {
                const int ci = i0 + (tid >> 3) + 32 * r;
                const int k = kt0 + cc * EPC;
                const bool ok = ci < a.NI && k < k_end;
                if constexpr (VI) {
                    const int kh = rh + a.sh * kq0, kw = rw + a.sw * kq1;
                    const T *p = srcI + (((int64_t)kh * a.KW + kw) * a.C + ci) * a.K + kq2;
                    stI[r] = ok ? ld16(p) : zero4();
                } else {
                    U4 v = zero4();
                    int q0 = kq0, q1 = kq1, q2 = kq2;
#pragma unroll
                    for (int e = 0; e < EPC; ++e) {
                        if (ok && k + e < k_end) {
                            const int kh = rh + a.sh * q0, kw = rw + a.sw * q1;
                            chunk_set<T>(v, e, ld_elem<T>(srcI + (((int64_t)kh * a.KW + kw) * a.C + ci) * a.K + q2));
                        }
                        if (++q2 == kInner) { q2 = 0; if (++q1 == kMid) { q1 = 0; ++q0; } }
                    }
                    stI[r] = v;
                }
            }
        }
        // ---------------- J operand
        if constexpr (DIR == DIR_FWD || DIR == DIR_BWD_DATA) {
            const int k = kt0 + cc * EPC;
            const int Hlim = (DIR == DIR_FWD) ? a.H : a.OH;
            const int Wlim = (DIR == DIR_FWD) ? a.W : a.OW;
            const int64_t rowlen = (DIR == DIR_FWD) ? a.W : a.OW;
            const int64_t pst = (DIR == DIR_FWD) ? a.xs : a.ys;
#pragma unroll
            for (int r = 0; r < DR_J; ++r) {
                if constexpr (VJ) {
                    int yy, xx;
                    if constexpr (DIR == DIR_FWD) { yy = jy0[r] + kq0; xx = jx0[r] + kq1; }
                    else { yy = jy0[r] - kq0; xx = jx0[r] - kq1; }
                    const bool ok = jok[r] && k < k_end && (unsigned)yy < (unsigned)Hlim &&
                                    (unsigned)xx < (unsigned)Wlim;
                    const T *p = srcJ + (jbase[r] + (int64_t)yy * rowlen + xx) * pst + kq2;
                    stJ[r] = ok ? ld16(p) : zero4();
                } else {
                    U4 v = zero4();
                    int q0 = kq0, q1 = kq1, q2 = kq2;
#pragma unroll
                    for (int e = 0; e < EPC; ++e) {
                        int yy, xx;
                        if constexpr (DIR == DIR_FWD) { yy = jy0[r] + q0; xx = jx0[r] + q1; }
                        else { yy = jy0[r] - q0; xx = jx0[r] - q1; }
                        const bool ok = jok[r] && k + e < k_end && (unsigned)yy < (unsigned)Hlim &&
                                        (unsigned)xx < (unsigned)Wlim;
                        if (ok)
                            chunk_set<T>(v, e, ld_elem<T>(srcJ + (jbase[r] + (int64_t)yy * rowlen + xx) * pst + q2));
                        if (++q2 == kInner) { q2 = 0; if (++q1 == kMid) { q1 = 0; ++q0; } }
                    }
                    stJ[r] = v;
                }
            }
        } else {
            // BWD_FILTER: transposed, rows = taps (kh, kw, ci), k = pixels (n, oh, ow)
#pragma unroll
            for (int u = 0; u < TN_J; ++u) {
                const int unit = tid + NT * u;
                const int kg = unit & 7;
                const int rbase = j0 + (unit >> 3) * EPC;
                U4 v[EPC];
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const int k = kt0 + kg * EPC + e;
                    const bool kok = fr_ok[u] && k < k_end;
                    uint32_t t, ow, n, oh;
                    a.dOW.divmod((uint32_t)(kok ? k : 0), t, ow);
                    a.dOH.divmod(t, n, oh);
                    if constexpr (VJ) {
                        const int ih = (int)oh * a.sh + fr_dh[u];
                        const int iw = (int)ow * a.sw + fr_dw[u];
                        const bool ok = kok && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                        const T *p = srcJ + (((int64_t)n * a.H + ih) * a.W + iw) * a.xs + fr_ci[u];
                        v[e] = ok ? ld16(p) : zero4();
                    } else {
                        v[e] = zero4();
                        // taps of the EPC rows rbase .. rbase + EPC - 1, one element each
#pragma unroll
                        for (int q = 0; q < EPC; ++q) {
                            const int row = rbase + q;
                            if (kok && row < MJ_ext) {
                                uint32_t t2, ci, kh, kw;
                                a.dC.divmod((uint32_t)row, t2, ci);
                                a.dKW.divmod(t2, kh, kw);
                                const int ih = (int)oh * a.sh + (int)kh - a.pt;
                                const int iw = (int)ow * a.sw + (int)kw - a.pl;
                                if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W)
                                    chunk_set<T>(v[e], q, ld_elem<T>(srcJ + (((int64_t)n * a.H + ih) * a.W + iw) * a.xs + ci));
                            }
                        }
                    }
                }
                transpose_block<T>(v, &stJ[u * EPC]);
            }
        }
    };

    // ------------------------------------------------------------ commit (registers -> LDS)
    auto commit = [&](int stage) {
        unsigned char *bI = smem + stage * STAGE;
        unsigned char *bJ = bI + TI_BYTES;
        if constexpr (TRANS_I) {
#pragma unroll
            for (int u = 0; u < TN_I; ++u) {
                const int unit = tid + NT * u;
                if (TU_I >= NT * (u + 1) || unit < TU_I) {
                    const int kg = unit & 7, rg = unit >> 3;
#pragma unroll
                    for (int r = 0; r < EPC; ++r)
                        *reinterpret_cast<U4 *>(bI + lds_off(rg * EPC + r, kg)) = stI[u * EPC + r];
                }
            }
        } else {
#pragma unroll
            for (int r = 0; r < DR_I; ++r)
                *reinterpret_cast<U4 *>(bI + lds_off((tid >> 3) + 32 * r, cc)) = stI[r];
        }
        if constexpr (TRANS_J) {
#pragma unroll
            for (int u = 0; u < TN_J; ++u) {
                const int unit = tid + NT * u;
                if (TU_J >= NT * (u + 1) || unit < TU_J) {
                    const int kg = unit & 7, rg = unit >> 3;
#pragma unroll
                    for (int r = 0; r < EPC; ++r)
                        *reinterpret_cast<U4 *>(bJ + lds_off(rg * EPC + r, kg)) = stJ[u * EPC + r];
                }
            }
        } else {
#pragma unroll
            for (int r = 0; r < DR_J; ++r)
                *reinterpret_cast<U4 *>(bJ + lds_off((tid >> 3) + 32 * r, cc)) = stJ[r];
        }
    };

    // ------------------------------------------------------------ main loop
    const int wi = wave % WAVES_I, wj = wave / WAVES_I;
    f32x4_t acc[MI][MJ];
#pragma unroll
    for (int x = 0; x < MI; ++x)
#pragma unroll
        for (int y = 0; y < MJ; ++y) acc[x][y] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if (nk > 0) {
        fetch(0);
        if constexpr (DIR != DIR_BWD_FILTER) advance_k();
        commit(0);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const bool more = kt + 1 < nk;
            if (more) {
                fetch(kt + 1);
                if constexpr (DIR != DIR_BWD_FILTER) advance_k();
            }
            const unsigned char *bI = smem + (kt & 1) * STAGE;
            const unsigned char *bJ = bI + TI_BYTES;
#pragma unroll
            for (int s = 0; s < BKC / 4; ++s) {
                const int chunk = 4 * s + (lane >> 4);
                U4 fi[MI], fj[MJ];
#pragma unroll
                for (int x = 0; x < MI; ++x)
                    fi[x] = *reinterpret_cast<const U4 *>(bI + lds_off(wi * WI + x * 16 + (lane & 15), chunk));
#pragma unroll
                for (int y = 0; y < MJ; ++y)
                    fj[y] = *reinterpret_cast<const U4 *>(bJ + lds_off(wj * WJ + y * 16 + (lane & 15), chunk));
#pragma unroll
                for (int x = 0; x < MI; ++x)
#pragma unroll
                    for (int y = 0; y < MJ; ++y) Mfma<T>::run(acc[x][y], fi[x], fj[y]);
            }
            if (more) commit((kt + 1) & 1);
            __syncthreads();
        }
    }

    // ------------------------------------------------------------ epilogue
    // acc[x][y] lane l, register q: channel i = i0 + wi*WI + x*16 + 4*(l>>4) + q,
    //                               row     j = j0 + wj*WJ + y*16 + (l & 15).
#pragma unroll
    for (int y = 0; y < MJ; ++y) {
        const int j = j0 + wj * WJ + y * 16 + (lane & 15);
        if (j >= MJ_ext) continue;
        int64_t rowoff;   // element offset of the output row
        if constexpr (DIR == DIR_FWD) {
            rowoff = (int64_t)j * a.ys;
        } else if constexpr (DIR == DIR_BWD_DATA) {
            const int tw = j % Wp;
            const int t = j / Wp;
            const int th = t % Hp;
            const int n = t / Hp;
            const int h = h0 + a.sh * th, w = w0 + a.sw * tw;
            rowoff = (((int64_t)n * a.H + h) * a.W + w) * a.xs;
        } else {
            rowoff = (int64_t)blockIdx.z * a.split_stride + (int64_t)j * a.K;
        }
#pragma unroll
        for (int x = 0; x < MI; ++x) {
            const int i = i0 + wi * WI + x * 16 + 4 * (lane >> 4);
            if (i >= a.NI) continue;
            const f32x4_t v = acc[x][y];
            if constexpr (DIR == DIR_BWD_FILTER) {
                float *o = reinterpret_cast<float *>(a.out) + rowoff + i;
                if (i + 3 < a.NI) {
                    *reinterpret_cast<f32x4_t *>(o) = v;
                } else {
                    for (int q = 0; q < 4 && i + q < a.NI; ++q) o[q] = v[q];
                }
            } else {
                T *o = reinterpret_cast<T *>(a.out) + rowoff + i;
                float r4[4] = {v[0], v[1], v[2], v[3]};
                if constexpr (DIR == DIR_BWD_DATA) {
                    if (a.beta != 0.f) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            if (i + q < a.NI) r4[q] += a.beta * Elem<T>::load(o + q);
                    }
                }
                if constexpr (DIR == DIR_FWD) {
                    if (a.bias != nullptr) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const float v = r4[q] + (i + q < a.NI ? a.bias[i + q] : 0.f);
                            r4[q] = v > 0.f ? v : 0.f;
                        }
                    }
                }
                if (i + 3 < a.NI) {
                    if constexpr (sizeof(T) == 4) {
                        // 16-byte store needs a 16-byte aligned address
                        if (((uintptr_t)o & 15) == 0) {
                            *reinterpret_cast<f32x4_t *>(o) = f32x4_t{r4[0], r4[1], r4[2], r4[3]};
                        } else {
#pragma unroll
                            for (int q = 0; q < 4; ++q) Elem<T>::store(o + q, r4[q]);
                        }
                    } else {
                        if (((uintptr_t)o & 7) == 0) {
                            uint2 pk;
                            pk.x = pack_bf16x2(r4[0], r4[1]);
                            pk.y = pack_bf16x2(r4[2], r4[3]);
                            *reinterpret_cast<uint2 *>(o) = pk;
                        } else {
#pragma unroll
                            for (int q = 0; q < 4; ++q) Elem<T>::store(o + q, r4[q]);
                        }
                    }
                } else {
                    for (int q = 0; q < 4 && i + q < a.NI; ++q) Elem<T>::store(o + q, r4[q]);
                }
            }
        }
    }
}

}  // namespace tfk
