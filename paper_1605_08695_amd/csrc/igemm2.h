// Pipelined bf16 implicit-GEMM convolution for gfx950 (all three directions).
//
// Same GEMM views as igemm.h (I side = output channels, J side = rows), but
// built for latency hiding on CDNA4:
//
//  * Global -> LDS copies use the gfx950 direct-to-LDS load
//    (global_load_lds_dwordx4): no staging registers, no LDS-store
//    instructions.  One wave instruction moves 64 x 16 bytes into a
//    contiguous 1 KiB of LDS (lane l lands at base + 16 l), so each lane is
//    given the global chunk that belongs at its LDS slot; out-of-range chunks
//    are fetched from a 16-byte zero page.
//  * A ring of three LDS stages: the copies of K-tile t+2 are in flight while
//    the MFMAs consume tile t.  Each stage is a separate LDS object and the
//    loop is unrolled by three, so the compiler can see which stage an LDS
//    read touches and only waits for the copies it depends on
//    (s_waitcnt vmcnt(n) with n = the copies of the next tile).
//  * Operands whose memory is k-contiguous (im2col rows of x, the dy gather
//    and the filter in bwd-input) are kept as [row][k] with 16-byte chunks
//    XOR-swizzled by (row & 7) and read with ds_read_b128.  Operands that are
//    contiguous along the row axis (the filter in the forward pass, both
//    operands of bwd-filter) are kept k-major, [k][row], exactly as they sit
//    in memory, with chunks swizzled by k (kmajor_swz); the MFMA fragment (eight
//    consecutive k of one row per lane) is assembled by two ds_read_b64_tr_b16
//    transposing reads.  No operand is transposed in registers.
//
// Requirements (checked by the launcher): bf16, every gathered 16-byte chunk
// is aligned and lies within one pixel's channels (channel counts and pixel
// strides multiples of 8, 16-byte aligned bases).
#pragma once
#include <type_traits>

#include "igemm.h"

namespace tfk {

typedef short __attribute__((ext_vector_type(4))) s16x4_t;

// 16 zero bytes in device memory: the source of every out-of-range chunk.
__device__ __attribute__((aligned(16))) uint32_t g_zero_chunk[4];

// One 16-byte direct-to-LDS copy per lane: lane l's chunk lands at lds_base + 16 l.
// Issued from inline assembly so that the compiler does not track these copies:
// its LDS-DMA alias tracking would otherwise make every LDS read wait for every
// copy in flight.  Completion is ordered explicitly with wait_barrier<N>().
__device__ __forceinline__ void dma16(const void *src, unsigned char *lds_base) {
    const uint32_t lds_addr = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char *)lds_base);
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(lds_addr)
                 : "memory");
}

// Wait until at most N vector-memory operations of this wave are in flight and
// every LDS read of this wave has returned, then synchronise the workgroup.
// After it, tile t has landed for every wave and no wave still reads the stage
// that the next copies overwrite.  One asm statement with a memory clobber, so
// no LDS read is moved above the barrier.
template <int N>
__device__ __forceinline__ void wait_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

__device__ __forceinline__ U4 lds_tr_pair(const unsigned char *p0, const unsigned char *p1) {
    const s16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_t *)(p0));
    const s16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_t *)(p1));
    // Four 16-bit elements already packed in two dwords (element 0 in the low half).
    const uint2 ua = __builtin_bit_cast(uint2, a);
    const uint2 ub = __builtin_bit_cast(uint2, b);
    U4 r;
    r.x = ua.x; r.y = ua.y; r.z = ub.x; r.w = ub.y;
    return r;
}

// Chunk swizzle of k-row k in a k-major tile with R rows.  A transposing read of a
// 16-lane group touches 32 bytes (two chunks) of 4 consecutive k-rows, and two groups
// (k-rows 8g + 0..3 and 8g + 8..11) are served together: 2 (k & 3) spreads the 4 rows
// of a group over distinct chunk pairs and bit 3 of k moves the second group to the
// other half of the banks (for 64-row tiles, whose k-rows are 128 bytes, it moves the
// group to the free chunk pairs instead).
template <int R>
__device__ __forceinline__ int kmajor_swz(int k) {
    if constexpr (R == 64) return ((k & 3) ^ ((k >> 3) & 1)) << 1;
    else return ((k & 3) << 1) ^ (((k >> 3) & 1) << 3);
}

// Byte offset of element (k, row) of a k-major tile with R rows (row a multiple of 4).
template <int R>
__device__ __forceinline__ int kmajor_off(int k, int row) {
    return k * (R * 2) + (((row >> 3) ^ kmajor_swz<R>(k)) << 4) + ((row & 7) << 1);
}

// Workgroups are dealt to the 8 XCDs of the chip round-robin by linear id, and each XCD
// has its own L2.  Renumber them so that XCD x runs one contiguous range of logical
// blocks: neighbouring tiles (which read the same input rows) then share an L2.  Any
// bijection is correct; this one only decides where data is cached.
__device__ __forceinline__ int xcd_order(int linear, int total) {
    constexpr int kXcd = 8;
    const int q = total / kXcd, r = total % kXcd;
    const int x = linear % kXcd;
    return x * q + min(x, r) + linear / kXcd;
}

// BI x BJ output tile, NW waves (a 2 x NW/2 grid of wave tiles), NS LDS stages.  Every
// SIMD runs two waves: one 8-wave block per CU, or two 4-wave blocks per CU when NS
// stages fit twice in the 160 KiB of LDS.  Two independent blocks keep a CU's MFMAs busy
// while the other block waits at its barrier for a slow copy.
template <int DIR, int BI, int BJ, int NW, int NS>
__global__ __launch_bounds__(NW * 64, 2) void igemm2_kernel(const IgArgs a) {
    constexpr int BK = 64;
    constexpr int WGJ = NW / 2;                       // wave grid 2 (I) x NW/2 (J)
    constexpr bool TI = DIR != DIR_BWD_DATA;          // I operand kept k-major
    constexpr bool TJ = DIR == DIR_BWD_FILTER;        // J operand kept k-major
    constexpr int IB = BI * 128, JB = BJ * 128, SB = IB + JB;
    constexpr int NLI = BI / (8 * NW), NLJ = BJ / (8 * NW), NL = NLI + NLJ;   // copies per thread per tile
    constexpr int WI = BI / 2, WJ = BJ / WGJ;
    constexpr int MI = WI / 16, MJ = WJ / 16;
    static_assert(NW == 4 || NW == 8, "waves");
    static_assert(NS == 2 || NS == 3, "stages");
    static_assert(NLI >= 1 && NLJ >= 1 && MI >= 1 && MJ >= 1, "tile");
    static_assert(NS * SB <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) unsigned char lds0[SB];
    __shared__ __attribute__((aligned(1024))) unsigned char lds1[SB];
    __shared__ __attribute__((aligned(1024))) unsigned char lds2[NS == 3 ? SB : 16];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // (the launcher may keep the hardware order: for bwd-filter splits of the AlexNet layers
    // spreading one split's tiles over all XCDs measured faster than concentrating them)
    const int lin_hw = (int)(blockIdx.x + gridDim.x * blockIdx.z);
    const int lin = a.xcd_order ? xcd_order(lin_hw, (int)(gridDim.x * gridDim.z)) : lin_hw;
    const int bx = lin % (int)gridDim.x;
    const int bz = lin / (int)gridDim.x;
    const int ti = bx % a.tiles_i;
    const int tj = bx / a.tiles_i;
    const int i0 = ti * BI;
    const int j0 = tj * BJ;

    const bf16_t *__restrict__ srcI = reinterpret_cast<const bf16_t *>(a.src_i);
    const bf16_t *__restrict__ srcJ = reinterpret_cast<const bf16_t *>(a.src_j);
    const void *zero = (const void *)g_zero_chunk;

    // ------------------------------------------------------------ direction set-up
    int MJ_ext, k_beg = 0, k_end;
    int rh = 0, rw = 0, h0 = 0, w0 = 0, Hp = 1, Wp = 1, offh = 0, offw = 0, KHp = 1, KWp = 1;
    if constexpr (DIR == DIR_FWD) {
        MJ_ext = a.N * a.OH * a.OW;
        k_end = a.KH * a.KW * a.C;
    } else if constexpr (DIR == DIR_BWD_DATA) {
        const int z = bz;
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
        k_beg = bz * a.k_split;
        k_end = min(a.N * a.OH * a.OW, k_beg + a.k_split);
    }
    if (j0 >= MJ_ext) return;
    const int nk = k_end > k_beg ? (k_end - k_beg + BK - 1) / BK : 0;

    // ------------------------------------------------------------ copy plan
    // [row][k] operands: copy r of this thread covers row 8 slot + lane/8, slot = wave*NL_op + r,
    // and the logical chunk (lane & 7) ^ (lane >> 3); it lands at byte 1024 slot of the tile.
    // k-major operands with R rows: copy r covers k-row slot (512/R) + lane / (R/8) and row
    // chunk (lane % (R/8)) ^ kmajor_swz(k-row).  Everything that does not depend on the K tile is
    // computed here once.
    const int dchunk = (lane & 7) ^ (lane >> 3);

    // [row][k] J rows (FWD: output pixels; BWD_DATA: dx pixels of the phase)
    const bf16_t *jptr[NLJ];
    int jy0[NLJ], jx0[NLJ];
    bool jok[NLJ];
    if constexpr (!TJ) {
#pragma unroll
        for (int r = 0; r < NLJ; ++r) {
            const int m = j0 + 8 * (wave * NLJ + r) + (lane >> 3);
            jok[r] = m < MJ_ext;
            const int mm = jok[r] ? m : 0;
            if constexpr (DIR == DIR_FWD) {
                const int ow = mm % a.OW;
                const int t = mm / a.OW;
                const int oh = t % a.OH;
                const int n = t / a.OH;
                jy0[r] = oh * a.sh - a.pt;
                jx0[r] = ow * a.sw - a.pl;
                jptr[r] = srcJ + (((int64_t)n * a.H + jy0[r]) * a.W + jx0[r]) * a.xs;
            } else {
                const int tw = mm % Wp;
                const int t = mm / Wp;
                const int th = t % Hp;
                const int n = t / Hp;
                jy0[r] = th + offh;        // oh = jy0 - jh
                jx0[r] = tw + offw;        // ow = jx0 - jw
                jptr[r] = srcJ + (((int64_t)n * a.OH + jy0[r]) * a.OW + jx0[r]) * a.ys;
            }
        }
    }
    // BWD_DATA I rows (filter rows ci)
    const bf16_t *iptr[NLI];
    bool iok[NLI];
    if constexpr (!TI) {
#pragma unroll
        for (int r = 0; r < NLI; ++r) {
            const int ci = i0 + 8 * (wave * NLI + r) + (lane >> 3);
            iok[r] = ci < a.NI;
            iptr[r] = srcI + (int64_t)(iok[r] ? ci : 0) * a.K;
        }
    }
    // k-major I operand (FWD filter [k][co], BWD_FILTER dy [pixel][co])
    int tik[NLI];
    if constexpr (TI) {
        constexpr int CPR = BI / 8;
        const int64_t ld = (DIR == DIR_FWD) ? (int64_t)a.K : a.ys;
#pragma unroll
        for (int r = 0; r < NLI; ++r) {
            const int krow = (wave * NLI + r) * (512 / BI) + lane / CPR;
            const int co = i0 + ((lane % CPR) ^ kmajor_swz<BI>(krow)) * 8;
            iok[r] = co < a.NI;
            tik[r] = krow;
            iptr[r] = srcI + (int64_t)(k_beg + krow) * ld + (iok[r] ? co : 0);
        }
    }
    // BWD_FILTER J rows (filter taps, k-major): per copy, the 8 taps of its row chunk
    int fr_dh[NLJ], fr_dw[NLJ], fr_ci[NLJ], fr_k[NLJ];
    bool fr_ok[NLJ];
    if constexpr (TJ) {
        constexpr int CPR = BJ / 8;
#pragma unroll
        for (int r = 0; r < NLJ; ++r) {
            const int krow = (wave * NLJ + r) * (512 / BJ) + lane / CPR;
            const int c = (lane % CPR) ^ kmajor_swz<BJ>(krow);
            const int r0 = j0 + c * 8;
            fr_ok[r] = r0 < MJ_ext;
            const int rr = fr_ok[r] ? r0 : 0;
            const int ci = rr % a.C;
            const int t = rr / a.C;
            fr_ci[r] = ci;
            fr_dw[r] = t % a.KW - a.pl;
            fr_dh[r] = t / a.KW - a.pt;
            fr_k[r] = krow;
        }
    }
    // k decomposition of this thread's chunk for [row][k] operands, recomputed per tile
    // with multiply-high division.  FWD J: k = (kh, kw, ci) over (KH, KW, C);
    // BWD_DATA: k = (jh, jw, co) over (KHp, KWp, K).
    FastDiv dInner, dMid;
    if constexpr (DIR == DIR_FWD) { dInner = a.dC; dMid = a.dKW; }
    if constexpr (DIR == DIR_BWD_DATA) { dInner = a.dK; dMid.init((uint32_t)(KWp > 0 ? KWp : 1)); }

    // K-tile order.  With 64 | channels, every 64-wide K-tile lies inside one filter tap,
    // and the tiles are visited channel-chunk outer, tap inner: consecutive tiles then read
    // the same input rows shifted by one tap, which stay in L1/L2.  issue() is called for
    // kt = 0, 1, 2, ... in order, so the (chunk, tap) position advances by one per call.
    int perm_T = 1, perm_CC = 0;
    if constexpr (DIR == DIR_FWD) {
        if (a.C % BK == 0 && a.KH * a.KW > 1) { perm_T = a.KH * a.KW; perm_CC = a.C / BK; }
    } else if constexpr (DIR == DIR_BWD_DATA) {
        if (a.K % BK == 0 && KHp * KWp > 1) { perm_T = KHp * KWp; perm_CC = a.K / BK; }
    }
    int perm_tap = 0, perm_cc = 0;

    // Issue the copies of K-tile kt into LDS stage `st`.
    auto issue = [&](int kt_seq, unsigned char *st) __attribute__((always_inline)) {
        int kt = kt_seq;
        if constexpr (DIR != DIR_BWD_FILTER) {
            if (perm_CC > 0) {
                kt = perm_tap * perm_CC + perm_cc;
                if (++perm_tap == perm_T) { perm_tap = 0; ++perm_cc; }
            }
        }
        const int kt0 = k_beg + kt * BK;
        unsigned char *stI = st;
        unsigned char *stJ = st + IB;
        uint32_t kq0 = 0, kq1 = 0, kq2 = 0;
        if constexpr (DIR != DIR_BWD_FILTER) {
            uint32_t t;
            dInner.divmod((uint32_t)(kt0 + dchunk * 8), t, kq2);
            dMid.divmod(t, kq0, kq1);
        }
        const bool kin = kt0 + dchunk * 8 < k_end;
        // ---------------- I operand
        if constexpr (TI) {
            const int64_t step = (int64_t)(kt * BK) * ((DIR == DIR_FWD) ? (int64_t)a.K : a.ys);
#pragma unroll
            for (int r = 0; r < NLI; ++r) {
                const bool ok = iok[r] && kt0 + tik[r] < k_end;
                dma16(ok ? (const void *)(iptr[r] + step) : zero, stI + (wave * NLI + r) * 1024);
            }
        } else {
            // BWD_DATA filter: w[rh + sh*jh][rw + sw*jw][ci][co..]
            const int64_t koff = ((int64_t)(rh + a.sh * (int)kq0) * a.KW + (rw + a.sw * (int)kq1)) * a.C * a.K + kq2;
#pragma unroll
            for (int r = 0; r < NLI; ++r)
                dma16(iok[r] && kin ? (const void *)(iptr[r] + koff) : zero, stI + (wave * NLI + r) * 1024);
        }
        // ---------------- J operand
        if constexpr (TJ) {
#pragma unroll
            for (int r = 0; r < NLJ; ++r) {
                const int k = kt0 + fr_k[r];
                const bool kok = fr_ok[r] && k < k_end;
                uint32_t t, ow, n, oh;
                a.dOW.divmod((uint32_t)(kok ? k : 0), t, ow);
                a.dOH.divmod(t, n, oh);
                const int ih = (int)oh * a.sh + fr_dh[r];
                const int iw = (int)ow * a.sw + fr_dw[r];
                const bool ok = kok && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                dma16(ok ? (const void *)(srcJ + (((int64_t)n * a.H + ih) * a.W + iw) * a.xs + fr_ci[r]) : zero,
                      stJ + (wave * NLJ + r) * 1024);
            }
        } else {
            int64_t koff;
            int dy, dx;
            if constexpr (DIR == DIR_FWD) {
                dy = (int)kq0; dx = (int)kq1;
                koff = ((int64_t)dy * a.W + dx) * a.xs + kq2;
            } else {
                dy = -(int)kq0; dx = -(int)kq1;
                koff = ((int64_t)dy * a.OW + dx) * a.ys + kq2;
            }
            const int Hlim = (DIR == DIR_FWD) ? a.H : a.OH;
            const int Wlim = (DIR == DIR_FWD) ? a.W : a.OW;
#pragma unroll
            for (int r = 0; r < NLJ; ++r) {
                const bool ok = jok[r] && kin && (unsigned)(jy0[r] + dy) < (unsigned)Hlim &&
                                (unsigned)(jx0[r] + dx) < (unsigned)Wlim;
                dma16(ok ? (const void *)(jptr[r] + koff) : zero, stJ + (wave * NLJ + r) * 1024);
            }
        }
    };

    // ------------------------------------------------------------ MFMA on one stage
    const int wi = wave & 1, wj = wave >> 1;
    f32x4_t acc[MI][MJ];
#pragma unroll
    for (int x = 0; x < MI; ++x)
#pragma unroll
        for (int y = 0; y < MJ; ++y) acc[x][y] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int lg = lane >> 4, ld = lane & 15;
    auto compute = [&](const unsigned char *st) __attribute__((always_inline)) {
        const unsigned char *stI = st;
        const unsigned char *stJ = st + IB;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            U4 fi[MI], fj[MJ];
#pragma unroll
            for (int x = 0; x < MI; ++x) {
                const int rb = wi * WI + x * 16;
                if constexpr (TI) {
                    const int k = 32 * s + 8 * lg + (ld >> 2);
                    const int row = rb + 4 * (ld & 3);
                    fi[x] = lds_tr_pair(stI + kmajor_off<BI>(k, row), stI + kmajor_off<BI>(k + 4, row));
                } else {
                    const int row = rb + ld;
                    fi[x] = *reinterpret_cast<const U4 *>(stI + lds_off(row, 4 * s + lg));
                }
            }
#pragma unroll
            for (int y = 0; y < MJ; ++y) {
                const int rb = wj * WJ + y * 16;
                if constexpr (TJ) {
                    const int k = 32 * s + 8 * lg + (ld >> 2);
                    const int row = rb + 4 * (ld & 3);
                    fj[y] = lds_tr_pair(stJ + kmajor_off<BJ>(k, row), stJ + kmajor_off<BJ>(k + 4, row));
                } else {
                    const int row = rb + ld;
                    fj[y] = *reinterpret_cast<const U4 *>(stJ + lds_off(row, 4 * s + lg));
                }
            }
#pragma unroll
            for (int x = 0; x < MI; ++x)
#pragma unroll
                for (int y = 0; y < MJ; ++y) Mfma<bf16_t>::run(acc[x][y], fi[x], fj[y]);
        }
        // Schedule: the fragment reads of the first sub-step, then the MFMAs of the first
        // sub-step alternating with the reads of the second, then its MFMAs -- so the LDS
        // latency of the second sub-step hides under MFMAs (about 2 % on the AlexNet layers).
        constexpr int RD = (TI ? 2 : 1) * MI + (TJ ? 2 : 1) * MJ;     // LDS reads per sub-step
        __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);             // DS reads
#pragma unroll
        for (int q = 0; q < MI * MJ; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);          // one MFMA
            if (q < RD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, MI * MJ, 0);
    };

    // One pipeline step on stage S = kt % NS: wait for tile kt (the copies of the later
    // tiles already issued may stay in flight), then refill the stage that tile kt - 1 used
    // (every wave has passed the barrier, so none still reads it) with tile kt + NS - 1.
    auto stage = [&](auto S_) __attribute__((always_inline)) -> unsigned char * {
        constexpr int S = decltype(S_)::value % NS;
        return S == 0 ? lds0 : (S == 1 ? lds1 : lds2);
    };
    auto step = [&](auto S_, int kt) __attribute__((always_inline)) {
        constexpr int S = decltype(S_)::value;
        if constexpr (NS == 3) {
            if (kt + 1 < nk) wait_barrier<NL>(); else wait_barrier<0>();
        } else {
            wait_barrier<0>();
        }
        if (kt + NS - 1 < nk) issue(kt + NS - 1, stage(std::integral_constant<int, S + NS - 1>{}));
        compute(stage(S_));
    };

    if (nk > 0) {
        issue(0, lds0);
        if (NS == 3 && nk > 1) issue(1, lds1);
        int kt = 0;
        for (; kt + NS <= nk; kt += NS) {
            step(std::integral_constant<int, 0>{}, kt);
            step(std::integral_constant<int, 1>{}, kt + 1);
            if constexpr (NS == 3) step(std::integral_constant<int, 2>{}, kt + 2);
        }
        if (kt < nk) step(std::integral_constant<int, 0>{}, kt);
        if (NS == 3 && kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
    }

    // ------------------------------------------------------------ epilogue
#pragma unroll
    for (int y = 0; y < MJ; ++y) {
        const int j = j0 + wj * WJ + y * 16 + ld;
        if (j >= MJ_ext) continue;
        int64_t rowoff;
        if constexpr (DIR == DIR_FWD) {
            rowoff = (int64_t)j * a.ys;
        } else if constexpr (DIR == DIR_BWD_DATA) {
            const int tw = j % Wp;
            const int t = j / Wp;
            const int th = t % Hp;
            const int n = t / Hp;
            rowoff = (((int64_t)n * a.H + h0 + a.sh * th) * a.W + w0 + a.sw * tw) * a.xs;
        } else {
            rowoff = (int64_t)bz * a.split_stride + (int64_t)j * a.K;
        }
#pragma unroll
        for (int x = 0; x < MI; ++x) {
            const int i = i0 + wi * WI + x * 16 + 4 * lg;
            if (i >= a.NI) continue;
            const f32x4_t v = acc[x][y];
            if constexpr (DIR == DIR_BWD_FILTER) {
                float *o = reinterpret_cast<float *>(a.out) + rowoff + i;
                *reinterpret_cast<f32x4_t *>(o) = v;          // NI % 8 == 0 and rows 16-byte aligned
            } else {
                bf16_t *o = reinterpret_cast<bf16_t *>(a.out) + rowoff + i;
                float r4[4] = {v[0], v[1], v[2], v[3]};
                if constexpr (DIR == DIR_BWD_DATA) {
                    if (a.beta != 0.f) {
                        const uint2 old = *reinterpret_cast<const uint2 *>(o);
                        r4[0] += a.beta * bf16_to_f32(old.x & 0xffffu);
                        r4[1] += a.beta * bf16_to_f32(old.x >> 16);
                        r4[2] += a.beta * bf16_to_f32(old.y & 0xffffu);
                        r4[3] += a.beta * bf16_to_f32(old.y >> 16);
                    }
                }
                if constexpr (DIR == DIR_FWD) {
                    if (a.bias != nullptr) {      // fused bias + ReLU, rounded once (i + 3 < NI)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const float v = r4[q] + a.bias[i + q];
                            r4[q] = v > 0.f ? v : 0.f;
                        }
                    }
                }
                uint2 pk;
                pk.x = pack_bf16x2(r4[0], r4[1]);
                pk.y = pack_bf16x2(r4[2], r4[3]);
                *reinterpret_cast<uint2 *>(o) = pk;
            }
        }
    }
}

}  // namespace tfk
