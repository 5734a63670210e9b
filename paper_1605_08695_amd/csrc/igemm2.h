// Pipelined bf16 implicit-GEMM convolution for gfx950 (all three directions).
//
// Same GEMM views as igemm.h (I side = output channels, J side = rows), but
// built for latency hiding on CDNA4:
//
//  * Global -> LDS copies use the direct-to-LDS buffer load
//    (buffer_load_dwordx4 ... lds): no staging registers, no LDS-store
//    instructions.  One wave instruction moves 64 x 16 bytes into a
//    contiguous 1 KiB of LDS (lane l lands at base + 16 l), so each lane is
//    given the chunk that belongs at its LDS slot, as a 32-bit byte offset into
//    its operand; out-of-range chunks get an offset past the operand's end,
//    which the buffer range check turns into zeros.
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
// strides multiples of 8, 16-byte aligned bases), both operands span fewer
// than 2^31 bytes and the filter has at most 31 rows and 31 columns.
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
// copy in flight.  Completion is ordered explicitly with wait_barrier<N>().  The s_nop is the
// wait state that an LDS DMA needs after a scalar write of M0.
__device__ __forceinline__ void dma16(const void *src, unsigned char *lds_base) {
    const uint32_t lds_addr = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char *)lds_base);
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(lds_addr)
                 : "memory");
}

typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes): no stride, no swizzle, dword data format.
// Loads through it at byte offsets >= bytes return zeros (checked per dword).
__device__ __forceinline__ i32x4_t buffer_rsrc(const void *base, uint32_t bytes) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    i32x4_t r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)b);
    r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(b >> 32) & 0xffffu));
    r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
    r[3] = 0x00020000;
    return r;
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_u32(const unsigned char *p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const unsigned char *)p;
}

// One 16-byte buffer-to-LDS copy per lane: lane l's chunk, at byte offset voff of the
// buffer, lands at LDS address lds_addr + 16 l.  Ordered like dma16().
__device__ __forceinline__ void bdma16(const i32x4_t rs, uint32_t voff, uint32_t lds_addr) {
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(voff), "s"(rs), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// Bits lo .. hi-1 set (none when lo >= hi); hi <= 31.
__device__ __forceinline__ uint32_t range_mask(int lo, int hi) {
    return lo < hi ? ((1u << hi) - 1u) & ~((1u << lo) - 1u) : 0u;
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
// group to the free chunk pairs instead).  192-row k-rows are 384 bytes, so consecutive
// k-rows start alternately at bank 0 and bank 32: bit 1 of k moves k-rows 2 and 3 of a
// group by one chunk pair and bit 3 of k the second group by two, which keeps every chunk
// inside its aligned group of eight.  32-row k-rows are 64 bytes: the 4 k-rows of a group already
// cover every bank once, and bit 3 of k moves the second group to the other chunk pair.
template <int R>
__device__ __forceinline__ int kmajor_swz(int k) {
    static_assert(R == 32 || R == 64 || R == 128 || R == 192 || R == 256, "k-major tile rows");
    if constexpr (R == 32) return ((k >> 3) & 1) << 1;
    else if constexpr (R == 64) return ((k & 3) ^ ((k >> 3) & 1)) << 1;
    else if constexpr (R != 192) return ((k & 3) << 1) ^ (((k >> 3) & 1) << 3);
    else return (((k >> 1) & 1) << 1) | (((k >> 3) & 1) << 2);
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
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // (the launcher may keep the hardware order)
    const int lin_hw = (int)(blockIdx.x + gridDim.x * blockIdx.z);
    const int lin = a.xcd_order ? xcd_order(lin_hw, (int)(gridDim.x * gridDim.z)) : lin_hw;
    const int bx = lin % (int)gridDim.x;
    const int bz = lin / (int)gridDim.x;
    const int ti = bx % a.tiles_i;
    const int tj = bx / a.tiles_i;
    const int i0 = ti * BI;
    // forward row bands: the J tile is rows band_r0 .. of image band_n, indexed locally from 0
    const bool banded = DIR == DIR_FWD && a.band_rows > 0;
    int band_n = 0, band_r0 = 0;
    if (banded) {
        band_n = tj / a.bands_per_img;
        band_r0 = (tj - band_n * a.bands_per_img) * a.band_step;
    }
    const int j0 = banded ? 0 : tj * BJ;

    // ------------------------------------------------------------ direction set-up
    int MJ_ext, k_beg = 0, k_end;
    int rh = 0, rw = 0, h0 = 0, w0 = 0, Hp = 1, Wp = 1, offh = 0, offw = 0, KHp = 1, KWp = 1;
    if constexpr (DIR == DIR_FWD) {
        MJ_ext = banded ? min(a.band_rows, a.OH - band_r0) * a.OW : a.N * a.OH * a.OW;
        k_end = a.KH * a.KW * a.C;
        KHp = a.KH;
        KWp = a.KW;
        if (a.k_split > 0) {                       // split-K: blockIdx.z picks a reduction range
            k_beg = bz * a.k_split;
            k_end = min(k_end, k_beg + a.k_split);
        }
    } else if constexpr (DIR == DIR_BWD_DATA) {
        const int z = a.k_split > 0 ? 0 : bz;      // (split-K runs with one stride phase)
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
        if (a.k_split > 0) {
            k_beg = bz * a.k_split;
            k_end = min(k_end, k_beg + a.k_split);
        }
    } else {
        MJ_ext = a.KH * a.KW * a.C;
        k_beg = bz * a.k_split;
        k_end = min(a.N * a.OH * a.OW, k_beg + a.k_split);
    }
    if (j0 >= MJ_ext) {
        // (a block past this stride phase's pixels still owns its rows of bias-gradient partials)
        if (DIR == DIR_BWD_DATA && a.relu_y != nullptr && (lane & 15) == 0) {
            const int row = (bz * (int)(gridDim.x / a.tiles_i) + tj) * WGJ + (wave >> 1);
            for (int x = 0; x < MI; ++x) {
                const int i = i0 + (wave & 1) * WI + x * 16 + 4 * (lane >> 4);
                if (i < a.NI)
                    for (int q = 0; q < 4; ++q) a.db_part[(int64_t)(i + q) * a.db_rows + row] = 0.f;
            }
        }
        return;
    }
    const int nk = k_end > k_beg ? (k_end - k_beg + BK - 1) / BK : 0;
    // K-tile order (see below): with 64 | channels and several taps the tiles are visited
    // channel-chunk outer, tap inner, and a split-K range [k_beg, k_end) then counts positions
    // in that order; the tile addresses come from the position, not from k_beg.
    bool perm = false;
    if constexpr (DIR == DIR_FWD) perm = a.C % BK == 0 && a.KH * a.KW > 1;
    if constexpr (DIR == DIR_BWD_DATA) perm = a.K % BK == 0 && KHp * KWp > 1;
    const int k_addr = perm ? 0 : k_beg;

    // ------------------------------------------------------------ copy plan
    // Every copy is one buffer load into LDS with a 32-bit byte offset per lane.  The buffer
    // resource of an operand spans exactly its bytes (fewer than 2^31, checked by the
    // launcher) and the hardware range check returns zeros for offsets at or past the end, so
    // padding taps, reduction entries past the end and rows past a tensor are given such an
    // offset (kBad, or a pixel offset that lies past the tensor) instead of a branch.  Along
    // the reduction axis both operands are zero past the end.  Rows past the output extent
    // (channels beyond NI, filter taps beyond KH*KW*C) are not masked: they read other
    // elements of the same operand into output rows that the epilogue drops.
    //
    // [row][k] operands: copy r of this thread covers row 8 slot + lane/8, slot = wave*NL_op + r,
    // and the logical chunk (lane & 7) ^ (lane >> 3); it lands at byte 1024 slot of the tile.
    // k-major operands with R rows: copy r fills 16-byte positions q = 64 slot + lane of the
    // tile, position q being chunk q % (R/8) of k-row q / (R/8), which holds the logical row
    // chunk (q % (R/8)) ^ kmajor_swz(k-row).  Everything that does not depend on the K tile is
    // computed here once.
    constexpr uint32_t kBad = 0x80000000u;
    const i32x4_t rsI = buffer_rsrc(a.src_i, a.bytes_i);
    const i32x4_t rsJ = buffer_rsrc(a.src_j, a.bytes_j);
    const int dchunk = (lane & 7) ^ (lane >> 3);

    // I operand: byte offset of each copy at K-tile 0 (k-major: + kt * BK * ldI2 per tile;
    // BWD_DATA filter rows ci: + the tile's tap and channel offset)
    uint32_t ivo[NLI];
    const uint32_t ldI2 = 2u * (uint32_t)((DIR == DIR_FWD) ? (int64_t)a.K : a.ys);
    if constexpr (TI) {
        constexpr int CPR = BI / 8;
#pragma unroll
        for (int r = 0; r < NLI; ++r) {
            const int pos = (wave * NLI + r) * 64 + lane;
            const int krow = pos / CPR;
            const int co = i0 + ((pos % CPR) ^ kmajor_swz<BI>(krow)) * 8;
            ivo[r] = (uint32_t)(k_addr + krow) * ldI2 + 2u * (uint32_t)co;
        }
    } else {
#pragma unroll
        for (int r = 0; r < NLI; ++r) {
            const int ci = i0 + 8 * (wave * NLI + r) + (lane >> 3);
            ivo[r] = (uint32_t)ci * 2u * (uint32_t)a.K;
        }
    }

    // J operand.  FWD / BWD_DATA ([row][k]): byte offset of the row's pixel for tap (0, 0) and
    // the complements of the masks of filter rows / columns whose tap lies inside the image
    // (bit 31 always set: it marks reduction entries past the end).  BWD_FILTER (k-major):
    // per copy, the pixel (byte offset, oh * sh, ow * sw) of its k-row, advanced by BK pixels
    // per tile, and the byte offset and (dh, dw) displacement of its chunk's filter tap.
    uint32_t jvo[NLJ], jnh[NLJ], jnw[NLJ], tvo[NLJ];
    int ohs[NLJ], ows[NLJ], fdh[NLJ], fdw[NLJ];
    const uint32_t xs2 = 2u * (uint32_t)a.xs, ys2 = 2u * (uint32_t)a.ys;
    if constexpr (!TJ) {
        const int Hlim = (DIR == DIR_FWD) ? a.H : a.OH;
        const int Wlim = (DIR == DIR_FWD) ? a.W : a.OW;
#pragma unroll
        for (int r = 0; r < NLJ; ++r) {
            const int m = j0 + 8 * (wave * NLJ + r) + (lane >> 3);
            const bool ok = m < MJ_ext;
            const int mm = ok ? m : 0;
            int y0, x0, hlo, hhi, wlo, whi;
            if constexpr (DIR == DIR_FWD) {
                uint32_t t, owu, n, ohu;
                a.dOW.divmod((uint32_t)mm, t, owu);
                if (banded) {
                    n = (uint32_t)band_n;
                    ohu = (uint32_t)band_r0 + t;
                } else {
                    a.dOH.divmod(t, n, ohu);
                }
                const int ow = (int)owu, oh = (int)ohu;
                y0 = oh * a.sh - a.pt;     // tap kh reads row y0 + kh
                x0 = ow * a.sw - a.pl;
                jvo[r] = (uint32_t)(((((int64_t)n * a.H + y0) * a.W + x0) * a.xs) * 2);
                hlo = max(0, -y0); hhi = min(KHp, Hlim - y0);
                wlo = max(0, -x0); whi = min(KWp, Wlim - x0);
            } else {
                const int tw = mm % Wp;
                const int t = mm / Wp;
                const int th = t % Hp;
                const int n = t / Hp;
                y0 = th + offh;            // tap jh reads dy row y0 - jh
                x0 = tw + offw;
                jvo[r] = (uint32_t)(((((int64_t)n * a.OH + y0) * a.OW + x0) * a.ys) * 2);
                hlo = max(0, y0 - Hlim + 1); hhi = min(KHp, y0 + 1);
                wlo = max(0, x0 - Wlim + 1); whi = min(KWp, x0 + 1);
            }
            jnh[r] = ok ? ~range_mask(hlo, hhi) : ~0u;
            jnw[r] = ~range_mask(wlo, whi);
        }
    }
    uint32_t adv_base = 0, adv_d1 = 0, adv_d2 = 0;
    int adv_w = 0, adv_h = 0, lim_w = 0, lim_h = 0;
    if constexpr (TJ) {
        constexpr int CPR = BJ / 8;
#pragma unroll
        for (int r = 0; r < NLJ; ++r) {
            const int pos = (wave * NLJ + r) * 64 + lane;
            const int krow = pos / CPR;
            const int c = (pos % CPR) ^ kmajor_swz<BJ>(krow);
            const int r0 = j0 + c * 8;
            const int rr = r0 < MJ_ext ? r0 : 0;
            uint32_t t, ci, kh, kw;
            a.dC.divmod((uint32_t)rr, t, ci);
            a.dKW.divmod(t, kh, kw);
            fdw[r] = (int)kw - a.pl;
            fdh[r] = (int)kh - a.pt;
            tvo[r] = (uint32_t)(((((int64_t)fdh[r] * a.W + fdw[r]) * a.xs) + (int64_t)ci) * 2);
            uint32_t q, ow, n, oh;
            a.dOW.divmod((uint32_t)(k_beg + krow), q, ow);
            a.dOH.divmod(q, n, oh);
            ohs[r] = (int)oh * a.sh;
            ows[r] = (int)ow * a.sw;
            jvo[r] = (uint32_t)(((((int64_t)n * a.H + ohs[r]) * a.W + ows[r]) * a.xs) * 2);
        }
        // BK pixels = dn images + ah rows + aw columns (ah < OH, aw < OW); adding them to
        // (oh, ow) wraps each coordinate at most once.
        const int pq = a.OH * a.OW;
        const int dn = BK / pq, rem = BK % pq, ah = rem / a.OW, aw = rem % a.OW;
        adv_w = aw * a.sw; lim_w = a.OW * a.sw;
        adv_h = ah * a.sh; lim_h = a.OH * a.sh;
        const int64_t hw = (int64_t)a.H * a.W;
        adv_base = (uint32_t)(((int64_t)dn * hw + (int64_t)ah * a.sh * a.W + (int64_t)aw * a.sw) * a.xs * 2);
        adv_d1 = (uint32_t)(((int64_t)a.sh * a.W - (int64_t)a.OW * a.sw) * a.xs * 2);   // column wrap
        adv_d2 = (uint32_t)((hw - (int64_t)a.OH * a.sh * a.W) * a.xs * 2);              // row wrap
    }
    // k decomposition of this lane's chunk for [row][k] operands.  FWD J: k = (kh, kw, ci)
    // over (KH, KW, C); BWD_DATA: k = (jh, jw, co) over (KHp, KWp, K).
    FastDiv dInner, dMid;
    if constexpr (DIR == DIR_FWD) { dInner = a.dC; dMid = a.dKW; }
    if constexpr (DIR == DIR_BWD_DATA) { dInner = a.dK; dMid.init((uint32_t)(KWp > 0 ? KWp : 1)); }

    // K-tile order.  With 64 | channels, every 64-wide K-tile lies inside one filter tap,
    // and the tiles are visited channel-chunk outer, tap inner: consecutive tiles then read
    // the same input rows shifted by one tap, which stay in L1/L2.  issue() is called for
    // kt = 0, 1, 2, ... in order, so the (chunk, tap) position advances by one per call; the
    // tap and channel chunk of a tile are then the same for every lane.
    int perm_CC = 0;
    if constexpr (DIR != DIR_BWD_FILTER) perm_CC = (DIR == DIR_FWD ? a.C : a.K) / BK;
    int perm_kh = 0, perm_kw = 0, perm_cc = 0;
    if (perm && k_beg > 0) {                       // split-K: start at position k_beg / BK
        const int p0 = k_beg / BK, taps = KHp * KWp;
        perm_cc = p0 / taps;
        const int r = p0 - perm_cc * taps;
        perm_kh = r / KWp;
        perm_kw = r - perm_kh * KWp;
    }

    // Issue the copies of K-tile kt into LDS stage `st`.
    auto issue = [&](int kt_seq, unsigned char *st) __attribute__((always_inline)) {
        const uint32_t stI = lds_u32(st);
        const uint32_t stJ = stI + IB;
        int kt = kt_seq;
        uint32_t kq0 = 0, kq1 = 0, kq2 = 0;
        bool kin = true;
        if constexpr (DIR != DIR_BWD_FILTER) {
            if (perm) {
                kq0 = perm_kh; kq1 = perm_kw;
                kq2 = perm_cc * BK + dchunk * 8;
                kt = (perm_kh * KWp + perm_kw) * perm_CC + perm_cc;
                if (++perm_kw == KWp) {
                    perm_kw = 0;
                    if (++perm_kh == KHp) { perm_kh = 0; ++perm_cc; }
                }
            } else {
                const int k = k_beg + kt * BK + dchunk * 8;
                kin = k < k_end;
                uint32_t t;
                dInner.divmod((uint32_t)k, t, kq2);
                dMid.divmod(t, kq0, kq1);
            }
        }
        // ---------------- I operand
        if constexpr (TI) {
            const uint32_t step = (uint32_t)(kt * BK) * ldI2;
#pragma unroll
            for (int r = 0; r < NLI; ++r) bdma16(rsI, ivo[r] + step, stI + (wave * NLI + r) * 1024);
        } else {
            // BWD_DATA filter: w[rh + sh*jh][rw + sw*jw][ci][co..]
            const uint32_t tap = (uint32_t)(rh + a.sh * (int)kq0) * (uint32_t)a.KW + (uint32_t)(rw + a.sw * (int)kq1);
            const uint32_t koff = kin ? (tap * (uint32_t)a.C * (uint32_t)a.K + kq2) * 2u : kBad;
#pragma unroll
            for (int r = 0; r < NLI; ++r) bdma16(rsI, ivo[r] + koff, stI + (wave * NLI + r) * 1024);
        }
        // ---------------- J operand
        if constexpr (TJ) {
#pragma unroll
            for (int r = 0; r < NLJ; ++r) {
                const bool ok = (unsigned)(ohs[r] + fdh[r]) < (unsigned)a.H && (unsigned)(ows[r] + fdw[r]) < (unsigned)a.W;
                bdma16(rsJ, ok ? jvo[r] + tvo[r] : kBad, stJ + (wave * NLJ + r) * 1024);
            }
#pragma unroll
            for (int r = 0; r < NLJ; ++r) {
                ows[r] += adv_w;
                const bool c1 = ows[r] >= lim_w;
                if (c1) ows[r] -= lim_w;
                ohs[r] += adv_h + (c1 ? a.sh : 0);
                const bool c2 = ohs[r] >= lim_h;
                if (c2) ohs[r] -= lim_h;
                jvo[r] += adv_base + (c1 ? adv_d1 : 0u) + (c2 ? adv_d2 : 0u);
            }
        } else {
            uint32_t koff;
            if constexpr (DIR == DIR_FWD) koff = (kq0 * (uint32_t)a.W + kq1) * xs2 + kq2 * 2u;
            else koff = kq2 * 2u - (kq0 * (uint32_t)a.OW + kq1) * ys2;
            const uint32_t khe = kin ? kq0 : 31u;
#pragma unroll
            for (int r = 0; r < NLJ; ++r) {
                const uint32_t bad = (uint32_t)(__builtin_amdgcn_sbfe((int)jnh[r], khe, 1u) |
                                                __builtin_amdgcn_sbfe((int)jnw[r], kq1, 1u));
                bdma16(rsJ, (jvo[r] + koff) | bad, stJ + (wave * NLJ + r) * 1024);
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
        if constexpr (DIR != DIR_BWD_FILTER) {
            // A CU runs two blocks of a launch side by side, and issue arbitration favours the
            // older one's waves: it finishes well ahead and leaves the other alone on the CU for
            // the launch's tail.  The two swap the higher wave priority every 1.28 us (the
            // 100 MHz clock's bit 7; the blocks of the second dispatch round, ids 256 up, take
            // the other phase), so both progress at the shared rate.  (Scheduling only.)
            const uint64_t now = __builtin_amdgcn_s_memrealtime();
            compute(stage(S_));
            if ((((uint32_t)(now >> 7) ^ (uint32_t)(lin_hw >> 8)) & 1u) != 0) __builtin_amdgcn_s_setprio(1);
            else __builtin_amdgcn_s_setprio(0);
        } else {
            compute(stage(S_));
        }
    };

    // The forward bias of this lane's channels, loaded before the main loop so that its latency
    // hides under the first copies instead of stalling the epilogue.
    float bq[MI][4];
#pragma unroll
    for (int x = 0; x < MI; ++x)
#pragma unroll
        for (int q = 0; q < 4; ++q) bq[x][q] = 0.f;
    if constexpr (DIR == DIR_FWD) {
        if (a.bias != nullptr && a.k_split == 0) {
#pragma unroll
            for (int x = 0; x < MI; ++x) {
                const int i = i0 + wi * WI + x * 16 + 4 * lg;
                if (i < a.NI)
#pragma unroll
                    for (int q = 0; q < 4; ++q) bq[x][q] = a.bias[i + q];
            }
        }
    }

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
    // (bwd-input with relu_y: the ReLU backward of the producing layer and the per-channel sums
    // of the stored dpre over this wave's rows, in y order, then over the 16 lanes of a column
    // group by a fixed xor tree)
    const bool relu = DIR == DIR_BWD_DATA && a.relu_y != nullptr;
    // forward with a fused max-pool: the band's bf16 outputs are staged in LDS (channels of the
    // first half of the tile in lds0, of the second in lds1, [row][channel]) once every wave has
    // finished reading the operand stages
    constexpr bool kPoolFits = DIR == DIR_FWD && BJ * BI <= 128 * (BI + BJ) && BI % 4 == 0;
    const bool pooled = kPoolFits && banded && a.pool_y != nullptr;
    constexpr int HC = BI / 2;                        // channels per staging half
    if (pooled) __syncthreads();
    float cs[MI][4];
#pragma unroll
    for (int x = 0; x < MI; ++x)
#pragma unroll
        for (int q = 0; q < 4; ++q) cs[x][q] = 0.f;
    // Row offsets of this lane's output rows.  (Loading an input gradient's old values and ReLU
    // outputs for all of a wave's tiles before the first store ran its kernels faster alone but
    // the two-stream step slower, about 1 %; they stay loaded tile by tile.)
    int64_t roff[MJ];
#pragma unroll
    for (int y = 0; y < MJ; ++y) {
        const int j = j0 + wj * WJ + y * 16 + ld;
        roff[y] = 0;
        if (j >= MJ_ext) continue;
        int64_t rowoff;
        if constexpr (DIR == DIR_FWD) {
            if (banded) {
                uint32_t dr, ow;
                a.dOW.divmod((uint32_t)j, dr, ow);
                rowoff = (((int64_t)band_n * a.OH + band_r0 + (int)dr) * a.OW + (int)ow) * a.ys;
            } else {
                rowoff = (int64_t)j * a.ys;
            }
        } else if constexpr (DIR == DIR_BWD_DATA) {
            const int tw = j % Wp;
            const int t = j / Wp;
            const int th = t % Hp;
            const int n = t / Hp;
            rowoff = (((int64_t)n * a.H + h0 + a.sh * th) * a.W + w0 + a.sw * tw) * a.xs;
        } else {
            rowoff = (int64_t)bz * a.split_stride + (int64_t)j * a.K;
        }
        roff[y] = rowoff;
    }
#pragma unroll
    for (int y = 0; y < MJ; ++y) {
        const int j = j0 + wj * WJ + y * 16 + ld;
        if (j >= MJ_ext) continue;
        const int64_t rowoff = roff[y];
#pragma unroll
        for (int x = 0; x < MI; ++x) {
            const int i = i0 + wi * WI + x * 16 + 4 * lg;
            if (i >= a.NI) continue;
            const f32x4_t v = acc[x][y];
            if constexpr (DIR != DIR_BWD_FILTER) {
                if (a.k_split > 0) {                   // split-K: fp32 partial [split][row][NI]
                    float *o = reinterpret_cast<float *>(a.out) + (int64_t)bz * a.split_stride + (int64_t)j * a.NI + i;
                    *reinterpret_cast<f32x4_t *>(o) = v;
                    continue;
                }
            }
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
                    if (relu) {
                        const uint2 yy = *reinterpret_cast<const uint2 *>(
                            reinterpret_cast<const bf16_t *>(a.relu_y) + rowoff + i);
                        const float yq[4] = {bf16_to_f32(yy.x & 0xffffu), bf16_to_f32(yy.x >> 16),
                                             bf16_to_f32(yy.y & 0xffffu), bf16_to_f32(yy.y >> 16)};
#pragma unroll
                        for (int q = 0; q < 4; ++q) r4[q] = yq[q] > 0.f ? r4[q] : 0.f;
                    }
                }
                if constexpr (DIR == DIR_FWD) {
                    if (a.bias != nullptr) {      // fused bias + ReLU, rounded once (i + 3 < NI)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const float v = r4[q] + bq[x][q];
                            r4[q] = v > 0.f ? v : 0.f;
                        }
                    }
                }
                uint2 pk;
                pk.x = pack_bf16x2(r4[0], r4[1]);
                pk.y = pack_bf16x2(r4[2], r4[3]);
                *reinterpret_cast<uint2 *>(o) = pk;
                if constexpr (kPoolFits) {
                    if (pooled) {
                        const int il = wi * WI + x * 16 + 4 * lg;     // channel within the tile
                        const int rl = j;                              // band row (local pixel)
                        unsigned char *stg = il < HC ? lds0 : lds1;
                        *reinterpret_cast<uint2 *>(stg + ((int64_t)rl * HC + (il % HC)) * 2) = pk;
                    }
                }
                if (relu) {
                    cs[x][0] += bf16_to_f32(pk.x & 0xffffu);
                    cs[x][1] += bf16_to_f32(pk.x >> 16);
                    cs[x][2] += bf16_to_f32(pk.y & 0xffffu);
                    cs[x][3] += bf16_to_f32(pk.y >> 16);
                }
            }
        }
    }
    if constexpr (kPoolFits) {
        if (pooled) {
            // pool rows q0 .. q0 + nq - 1 of this band; each thread takes one channel pair of the
            // tile and every G-th pool position; taps are scanned kh outer, kw inner, and a later
            // tap replaces the running maximum only when strictly greater
            __syncthreads();
            constexpr int CP = BI / 2, G = (NW * 64) / CP > 0 ? (NW * 64) / CP : 1;
            const int band = tj - band_n * a.bands_per_img;
            const int q0 = band * a.pool_rows;
            const int nq = min(a.pool_rows, a.pOH - q0);
            const int cp = tid % CP, g = tid / CP;
            const int c = 2 * cp;
            if (g < G && i0 + c < a.NI && nq > 0) {
                const unsigned char *stg = c < HC ? lds0 : lds1;
                const int cl = c % HC;
                bf16_t *py = reinterpret_cast<bf16_t *>(a.pool_y);
                for (int p = g; p < nq * a.pOW; p += G) {
                    const int qq = p / a.pOW, pw = p - qq * a.pOW;
                    const int q = q0 + qq;
                    float b0 = 0.f, b1 = 0.f;
                    int t0 = 0, t1 = 0;
                    for (int kh = 0; kh < a.pkh; ++kh) {
                        const int rl = (q * a.psh + kh - band_r0) * a.OW + pw * a.psw;
                        for (int kw = 0; kw < a.pkw; ++kw) {
                            const uint32_t v = *reinterpret_cast<const uint32_t *>(
                                stg + ((int64_t)(rl + kw) * HC + cl) * 2);
                            const float v0 = bf16_to_f32(v & 0xffffu), v1 = bf16_to_f32(v >> 16);
                            const int t = kh * a.pkw + kw;
                            if (t == 0 || v0 > b0) { b0 = v0; t0 = t; }
                            if (t == 0 || v1 > b1) { b1 = v1; t1 = t; }
                        }
                    }
                    const int64_t opix = ((int64_t)band_n * a.pOH + q) * a.pOW + pw;
                    *reinterpret_cast<uint32_t *>(py + opix * a.pool_ys + i0 + c) = pack_bf16x2(b0, b1);
                    *reinterpret_cast<uint16_t *>(a.pool_taps + opix * a.NI + i0 + c) =
                        (uint16_t)(t0 | (t1 << 8));
                }
            }
        }
    }
    if (relu) {
        const int row = (bz * (int)(gridDim.x / a.tiles_i) + tj) * WGJ + wj;
#pragma unroll
        for (int x = 0; x < MI; ++x) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float v = cs[x][q];
                v += __shfl_xor(v, 1, 16);
                v += __shfl_xor(v, 2, 16);
                v += __shfl_xor(v, 4, 16);
                v += __shfl_xor(v, 8, 16);
                cs[x][q] = v;
            }
            const int i = i0 + wi * WI + x * 16 + 4 * lg;
            if (ld == 0 && i < a.NI) {
#pragma unroll
                for (int q = 0; q < 4; ++q) a.db_part[(int64_t)(i + q) * a.db_rows + row] = cs[x][q];
            }
        }
    }
}

}  // namespace tfk
