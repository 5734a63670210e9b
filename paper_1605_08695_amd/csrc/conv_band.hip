// First-layer convolutions (at most 4 input channels, bf16) as "band" kernels
// that stage whole input rows in LDS and form the im2col operand from there.
//
// An image layer reads 4-channel pixels (RGB padded to RGBx, 8 bytes), and its
// large strided filters make the per-pixel im2col gather of the generic
// implicit GEMM a sea of 16-byte reads of overlapping windows.  Here a
// workgroup owns a band of R output rows of one image, copies the
// (R - 1) * stride + KH input rows that band reads into LDS once (zero-filled
// outside the image), and every MFMA operand is then read out of that copy:
//
//  * forward: y[p][co] = sum_m im2col(x)[p][m] * w[m][co], m = (kh, kw, c) with
//    kw padded to an even count.  Eight consecutive m are two horizontally
//    adjacent taps of one pixel row, i.e. 16 contiguous bytes of a staged row,
//    so the pixel operand is a plain 16-byte LDS read per lane.  The filter
//    (all reduction rows, 64 output channels) stays in LDS for the whole
//    persistent workgroup.
//  * bwd-filter: dW[m][co] = sum_p x(p, m) * dy[p][co] with the reduction over
//    the band's pixels.  Each lane of a transposing LDS read
//    (ds_read_b64_tr_b16) supplies its own address, so the x operand is
//    gathered straight from the staged rows: a lane fetches the 4 channels of
//    one tap at one pixel.  Each persistent workgroup sums over its bands and
//    writes one fp32 partial; the partials are summed in a fixed order.
//
// The bands of one workgroup are double-buffered: the direct-to-LDS copies of the
// next band are in flight while the current band is multiplied.
#include "igemm_launch.h"

namespace tfk {

namespace {

constexpr int kCUs = 256;                 // MI355X compute units: one persistent workgroup each
constexpr int kXBand = 45056;             // bytes of one staged input band (5632 pixels)
constexpr int kBandPix = kXBand / 8;
constexpr int kMaxKSteps = 18;            // forward: reduction rows <= 18 * 32 (an even number of steps)
constexpr int kFiltBytes = kMaxKSteps * 32 * 128;
constexpr int kDyBandPix = 256;           // bwd-filter: pixels per band (dy rows of 64 channels)
constexpr int kBwfGroups = 40;            // bwd-filter: at most 40 16-row tap groups (5 per wave)

struct BandArgs {
    const bf16_t *x;        // [N][H][W] pixels of 4 bf16, pixel stride 4 elements
    const bf16_t *w;        // forward: HWIO filter [KH][KW][C][K]
    const bf16_t *dy;       // bwd-filter: [N][OH][OW] rows of K channels, pixel stride ys
    void *out;              // forward: y (bf16, pixel stride ys); bwd-filter: fp32 partials [splits][KH][KW][C][K]
    const float *bias;      // forward: fused bias + ReLU when set
    int64_t ys;
    int N, H, W, C, OH, OW, K, KH, KW, sh, sw, pt, pl;
    int R;                  // output rows per band
    int bands_per_img, bands;
    int run;                // bands per workgroup: workgroup g takes bands g * run .. g * run + run - 1
    int rows_in;            // staged input rows per band: (R - 1) * sh + KH
    int wst;                // staged pixels per row (even)
    int kwp;                // taps per filter row in the reduction order (forward: KW rounded to 2; bwd-filter: to 4)
    int nks;                // forward: 32-wide reduction steps (even)
    FastDiv dWst, dOW, dKwp;
};

// A zero accumulator the compiler cannot merge with the other accumulators' zeros: with one
// shared zero register as the initial value of every loop-carried accumulator, the register
// allocator shuffles all of them through copies on every iteration.
__device__ __forceinline__ f32x4_t fresh_zero4() {
    float z0, z1, z2, z3;
    asm volatile("v_mov_b32 %0, 0\n\tv_mov_b32 %1, 0\n\tv_mov_b32 %2, 0\n\tv_mov_b32 %3, 0"
                 : "=v"(z0), "=v"(z1), "=v"(z2), "=v"(z3));
    return f32x4_t{z0, z1, z2, z3};
}

// One 4-byte direct-to-LDS copy per lane: lane l's word lands at lds_base + 4 l.  The s_nop is
// the wait state that an LDS DMA needs after a scalar write of M0 (as in dma16).
__device__ __forceinline__ void dma4(const void *src, unsigned char *lds_base) {
    const uint32_t lds_addr = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char *)lds_base);
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(lds_addr)
                 : "memory");
}

// Direct-to-LDS copies of input band b (rows_in x wst pixels, pixel e at byte 8 e of the buffer;
// zero outside the image).  X16: 16-byte copies of pixel pairs (the pairs never straddle the
// image edge: even left pad and width); else 4-byte copies of half pixels.  Copy i moves 64
// units; the copies of a band are spread over the 4 waves (copy i by wave i % 4).
template <bool X16>
struct BandCopier {
    const bf16_t *img;
    int ih0, npix, ncopies;

    __device__ __forceinline__ BandCopier(const BandArgs &a, int b) {
        const int n = b / a.bands_per_img;
        const int oh0 = (b - n * a.bands_per_img) * a.R;
        ih0 = oh0 * a.sh - a.pt;
        npix = a.rows_in * a.wst;
        img = a.x + (int64_t)n * a.H * a.W * 4;
        const int units = X16 ? (npix + 1) / 2 : 2 * npix;
        ncopies = (units + 63) / 64;
    }
    // copies of wave w of NW: i = w, w + NW, ...
    template <int NW = 4>
    __device__ __forceinline__ int count(int w) const { return ncopies > w ? (ncopies - w + NW - 1) / NW : 0; }
    __device__ __forceinline__ void copy(const BandArgs &a, int i, unsigned char *buf) const {
        const int lane = threadIdx.x & 63;
        const int u = 64 * i + lane;
        const int e = X16 ? 2 * u : (u >> 1);            // first pixel of the unit
        uint32_t r, c;
        a.dWst.divmod((uint32_t)e, r, c);
        const int ih = ih0 + (int)r, iw = (int)c - a.pl;
        const bool ok = e < npix && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
        const bf16_t *src = img + ((int64_t)ih * a.W + iw) * 4 + (X16 ? 0 : 2 * (u & 1));
        const void *zero = (const void *)g_zero_chunk;
        if constexpr (X16)
            dma16(ok ? (const void *)src : zero, buf + 1024 * i);
        else
            dma4(ok ? (const void *)src : zero, buf + 256 * i);
    }
};

template <bool X16, int NW = 4>
__device__ __forceinline__ void band_dma(const BandArgs &a, int b, unsigned char *buf) {
    const int wave = threadIdx.x >> 6;
    const BandCopier<X16> bc(a, b);
    for (int i = wave; i < bc.ncopies; i += NW) bc.copy(a, i, buf);
}

// ---------------------------------------------------------------------------------- forward
// Grid: (persistent workgroups, output-channel blocks of 64).  4 waves, one per SIMD; each wave
// multiplies up to 4 groups of 16 band pixels by all 64 channels per pass.  The fragments of
// reduction step kk + 1 are read from LDS while the MFMAs of step kk run, and the outputs of a
// band are stored during the next band (after its loads are issued), so neither the LDS latency
// nor the drain of the stores stalls the single wave of a SIMD.
template <bool A16, bool X16>
__global__ __launch_bounds__(256, 1) void band_fwd_kernel(const BandArgs a) {
    __shared__ __attribute__((aligned(1024))) unsigned char filt[kFiltBytes];
    __shared__ __attribute__((aligned(1024))) unsigned char xb0[kXBand];
    __shared__ __attribute__((aligned(1024))) unsigned char xb1[kXBand];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lg = lane >> 4, ld = lane & 15;
    const int co0 = blockIdx.y * 64;
    const int ntaps = a.KH * a.kwp;

    // Filter rows m = (kh * kwp + kw) * 4 + c, k-major with the transposing-read swizzle (zero for
    // padded taps, channels and rows), copied straight to LDS: copy i covers rows 8 i .. 8 i + 7.
    for (int i = wave; i < a.nks * 4; i += 4) {
        const int m = 8 * i + (lane >> 3);
        const int ch = (lane & 7) ^ kmajor_swz<64>(m);
        const int c = m & 3;
        uint32_t kh, kw;
        a.dKwp.divmod((uint32_t)(m >> 2), kh, kw);
        const int co = co0 + ch * 8;
        const bool ok = (int)kh < a.KH && (int)kw < a.KW && c < a.C && co < a.K;
        dma16(ok ? (const void *)(a.w + (((int64_t)kh * a.KW + kw) * a.C + c) * a.K + co)
                 : (const void *)g_zero_chunk,
              filt + 1024 * i);
    }

    int b = blockIdx.x * a.run;
    const int b_end = min(a.bands, b + a.run);
    if (b < b_end) band_dma<X16>(a, b, xb0);
    wait_barrier<0>();

    // bias of the lane's output channels co0 + 16 x + 4 lg + e, read once (K % 16 == 0: a channel
    // quad is either wholly inside or wholly past K)
    float bv[4][4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const int co = co0 + 16 * x + 4 * lg;
#pragma unroll
        for (int e = 0; e < 4; ++e) bv[x][e] = (a.bias != nullptr && co < a.K) ? a.bias[co + e] : 0.f;
    }
    // Outputs of the previous pass, stored while the next pass multiplies: packed bf16 of acc[x][y]
    // and the output offset (elements) of each of the lane's pixels (-1: no pixel).
    uint2 held[4][4];
    int64_t hoff[4];
#pragma unroll
    for (int y = 0; y < 4; ++y) hoff[y] = -1;
    bf16_t *const out = reinterpret_cast<bf16_t *>(a.out);
    auto store_row = [&](int x) __attribute__((always_inline)) {
        const int co = co0 + 16 * x + 4 * lg;
        if (co >= a.K) return;
#pragma unroll
        for (int y = 0; y < 4; ++y)
            if (hoff[y] >= 0) *reinterpret_cast<uint2 *>(out + hoff[y] + co) = held[x][y];
    };

    const int groups = (a.R * a.OW + 15) >> 4;
    const int passes = (groups + 15) >> 4;
    for (int it = 0; b < b_end; ++b, ++it) {
        const unsigned char *cur = (it & 1) ? xb1 : xb0;
        unsigned char *nxt = (it & 1) ? xb0 : xb1;
        const int bn = b + 1;
        const BandCopier<X16> bc(a, bn < b_end ? bn : b);
        const int ncw = bn < b_end ? bc.count(wave) : 0;     // this wave's copies of the next band

        const int n = b / a.bands_per_img;
        const int oh0 = (b - n * a.bands_per_img) * a.R;
        const int pb = min(a.R, a.OH - oh0) * a.OW;         // valid pixels of this band
        for (int pass = 0; pass < passes; ++pass) {
            const int nc = pass == 0 ? ncw : 0;
            int boff[4];
            int64_t coff[4];
#pragma unroll
            for (int y = 0; y < 4; ++y) {
                const int q = (pass * 16 + wave + 4 * y) * 16 + ld;
                uint32_t r, ow;
                a.dOW.divmod((uint32_t)(q < pb ? q : 0), r, ow);
                boff[y] = ((int)r * a.sh * a.wst + (int)ow * a.sw) * 8;
                coff[y] = q < pb ? (((int64_t)n * a.OH + oh0 + (int)r) * a.OW + (int)ow) * a.ys : -1;
            }
            f32x4_t acc[4][4];
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) acc[x][y] = fresh_zero4();

            // tap pair (kh, kw) = (t / kwp, t % kwp) of t = 8 kk + 2 lg, advanced by 8 taps per step
            int tkh = (2 * lg) / a.kwp, tkw = (2 * lg) % a.kwp;
            auto load = [&](int kk, U4 (&fi)[4], U4 (&fj)[4]) __attribute__((always_inline)) {
                const int to = 8 * kk + 2 * lg < ntaps ? (tkh * a.wst + tkw) * 8 : 0;
                tkw += 8;
#pragma unroll
                for (int r = 0; r < 4; ++r) {           // kwp >= 2: at most 4 wraps per step
                    if (tkw >= a.kwp) {
                        tkw -= a.kwp;
                        ++tkh;
                    }
                }
#pragma unroll
                for (int y = 0; y < 4; ++y) {
                    const unsigned char *p = cur + boff[y] + to;
                    if constexpr (A16) {
                        fj[y] = *reinterpret_cast<const U4 *>(p);
                    } else {
                        const uint2 lo = *reinterpret_cast<const uint2 *>(p);
                        const uint2 hi = *reinterpret_cast<const uint2 *>(p + 8);
                        fj[y].x = lo.x; fj[y].y = lo.y; fj[y].z = hi.x; fj[y].w = hi.y;
                    }
                }
                const int k = 32 * kk + 8 * lg + (ld >> 2);
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    const int row = 16 * x + 4 * (ld & 3);
                    fi[x] = lds_tr_pair(filt + kmajor_off<64>(k, row), filt + kmajor_off<64>(k + 4, row));
                }
            };
            auto mma = [&](const U4 (&fi)[4], const U4 (&fj)[4]) __attribute__((always_inline)) {
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int y = 0; y < 4; ++y) Mfma<bf16_t>::run(acc[x][y], fi[x], fj[y]);
            };
            // Two fragment sets: the reads of step kk + 1 are issued before the MFMAs of step kk.
            // Each double step also issues two of this wave's copies of the next band and one
            // channel row of the previous pass's outputs, so that the memory instructions are
            // spread under the MFMAs instead of stalling the wave before or after them.
            U4 fiA[4], fjA[4], fiB[4], fjB[4];
            load(0, fiA, fjA);
            int j = 0;
            for (int kk = 0; kk < a.nks; kk += 2, ++j) {     // nks is even
                load(kk + 1, fiB, fjB);
                if (2 * j < nc) bc.copy(a, wave + 8 * j, nxt);
                if (2 * j + 1 < nc) bc.copy(a, wave + 8 * j + 4, nxt);
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    if (x == j) store_row(x);
                mma(fiA, fjA);
                if (kk + 2 < a.nks) load(kk + 2, fiA, fjA);
                mma(fiB, fjB);
            }
            for (int c = 2 * j; c < nc; ++c) bc.copy(a, wave + 4 * c, nxt);
#pragma unroll
            for (int x = 0; x < 4; ++x)
                if (x >= j) store_row(x);

            // lane holds channels co0 + 16 x + 4 lg .. + 3 of pixel 16 g + ld
#pragma unroll
            for (int x = 0; x < 4; ++x) {
#pragma unroll
                for (int y = 0; y < 4; ++y) {
                    float v4[4] = {acc[x][y][0], acc[x][y][1], acc[x][y][2], acc[x][y][3]};
                    if (a.bias != nullptr) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float v = v4[e] + bv[x][e];
                            v4[e] = v > 0.f ? v : 0.f;
                        }
                    }
                    held[x][y].x = pack_bf16x2(v4[0], v4[1]);
                    held[x][y].y = pack_bf16x2(v4[2], v4[3]);
                }
            }
#pragma unroll
            for (int y = 0; y < 4; ++y) hoff[y] = coff[y];
        }

        wait_barrier<0>();
    }
#pragma unroll
    for (int x = 0; x < 4; ++x) store_row(x);
}

// ---------------------------------------------------------------------------------- forward, filter in registers
// For filters of exactly KS reduction steps and bands of at most 16 UPW pixels (UPW pixel groups
// of 16), 16-byte pixel pairs and staged rows of at most 256 pixels.  Each of the 4 waves holds
// the block's whole 64-channel filter slice in registers (staged once through LDS), so one pixel
// fragment read from LDS feeds up to four MFMAs (one per 16-channel group).  The band's units
// (pixel group g, channel group x), numbered 4 g + x, are dealt to the waves in equal contiguous
// runs of UPW: the run of wave w starts S0 = UPW w mod 4 channel groups into its first pixel
// group, so every wave issues UPW MFMAs per step and reads at most four fragments.  Staged rows
// have a fixed pitch of 256 pixels (2 KiB), so a band copy is one half of one row and its address
// is one scalar row offset away from a per-lane base.  Copies of the next band and the stores of
// the previous band are issued one per step under the MFMAs (the stores a band later, so the
// barrier that ends a band does not wait for them to drain).
constexpr int kRegRowBytes = 2048;                 // staged row pitch: 256 pixels of 8 bytes
constexpr int kRegMaxRows = 23;                    // staged rows per band
constexpr int kRegBand = kRegMaxRows * kRegRowBytes;

template <int KS, int UPW, int S0>
__device__ __forceinline__ void band_fwd_reg_body(const BandArgs &a, unsigned char *xb0, unsigned char *xb1,
                                                  const float *sbias, int wave) {
    constexpr int NF = (S0 + UPW + 3) / 4;          // pixel fragments per step
    constexpr int LAST = S0 + UPW - 4 * (NF - 1);    // channel groups of the last fragment
    static_assert(NF <= 4 && LAST >= 1, "units per wave");
    const int lane = threadIdx.x & 63, lg = lane >> 4, ld = lane & 15;
    const int co0 = blockIdx.y * 64;
    const int ntaps = a.KH * a.kwp;
    const int g0 = (UPW * wave) >> 2;               // first pixel group of this wave

    // filter fragments of every step and channel group (the filter is staged over xb0/xb1)
    U4 fw[KS][4];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
        const int k = 32 * kk + 8 * lg + (ld >> 2);
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const int row = 16 * x + 4 * (ld & 3);
            fw[kk][x] = lds_tr_pair(xb0 + kmajor_off<64>(k, row), xb0 + kmajor_off<64>(k + 4, row));
        }
    }
    wait_barrier<0>();                              // every wave holds its filter: the staging area is free

    // Band copies: wave w copies half (w & 1) of staged rows (w >> 1) + 2 c, c = 0, 1, ...  Its lane
    // holds pixel pair 64 (w & 1) + lane of a row: image column iw = 2 pc - pl (pairs never
    // straddle the image edge), zero outside the image.
    const int pc = 64 * (wave & 1) + lane;
    const int iw = 2 * pc - a.pl;
    const bool lane_ok = 2 * pc < a.wst && (unsigned)iw < (unsigned)a.W;
    const int wrow = wave >> 1;
    const int64_t row_elems = (int64_t)a.W * 4;
    const bf16_t *const lane_src = a.x + (int64_t)iw * 4;
    // first image row of this wave's copies of band bb (ih0) and that row's element offset (base)
    auto band_rows0 = [&](int bb, int &ih0, int64_t &base) __attribute__((always_inline)) {
        const int n = bb / a.bands_per_img;
        ih0 = (bb - n * a.bands_per_img) * a.R * a.sh - a.pt + wrow;
        base = ((int64_t)n * a.H + ih0) * row_elems;
    };
    auto band_copy = [&](int ih0, int64_t base, int c, unsigned char *buf) __attribute__((always_inline)) {
        const bool ok = lane_ok && (unsigned)(ih0 + 2 * c) < (unsigned)a.H;
        const bf16_t *src = lane_src + base + 2 * c * row_elems;
        dma16(ok ? (const void *)src : (const void *)g_zero_chunk,
              buf + (wrow + 2 * c) * kRegRowBytes + 1024 * (wave & 1));
    };
    const int ncw = (a.rows_in - wrow + 1) >> 1;    // this wave's copies of a band

    int b = blockIdx.x * a.run;
    const int b_end = min(a.bands, b + a.run);
    if (b < b_end) {
        int ih0;
        int64_t base;
        band_rows0(b, ih0, base);
        for (int c = 0; c < ncw; ++c) band_copy(ih0, base, c, xb0);
    }
    wait_barrier<0>();

    // biases of the lane's channels co0 + 16 x + 4 lg .. + 3 (zero without a bias); with a bias the
    // outputs are bias + ReLU, rounded once
    f32x4_t bvec[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const float4 bq = *reinterpret_cast<const float4 *>(sbias + 16 * x + 4 * lg);
        bvec[x] = f32x4_t{bq.x, bq.y, bq.z, bq.w};
    }
    const bool relu = a.bias != nullptr;
    // unit u of this wave (u < UPW): fragment slot (S0 + u) / 4, channel group (S0 + u) % 4
    uint2 held[NF][4];
    int hoff[NF];
#pragma unroll
    for (int j = 0; j < NF; ++j) hoff[j] = -1;
    bf16_t *const out = reinterpret_cast<bf16_t *>(a.out);
    auto store_one = [&](int u) __attribute__((always_inline)) {
        const int j = (S0 + u) >> 2, x = (S0 + u) & 3;
        const int co = co0 + 16 * x + 4 * lg;
        if (hoff[j] >= 0 && co < a.K) *reinterpret_cast<uint2 *>(out + hoff[j] + co) = held[j][x];
    };

    for (int it = 0; b < b_end; ++b, ++it) {
        const unsigned char *cur = (it & 1) ? xb1 : xb0;
        unsigned char *nxt = (it & 1) ? xb0 : xb1;
        const int bn = b + 1;
        const int nc = bn < b_end ? ncw : 0;        // this wave's copies of the next band
        int nih0 = 0;
        int64_t nbase = 0;
        if (bn < b_end) band_rows0(bn, nih0, nbase);

        const int n = b / a.bands_per_img;
        const int oh0 = (b - n * a.bands_per_img) * a.R;
        const int pb = min(a.R, a.OH - oh0) * a.OW;             // valid pixels of this band
        int boff[NF];                                           // pixel-pair index of the window origin
        int coff[NF];                                           // output offset (elements; fits int32)
#pragma unroll
        for (int j = 0; j < NF; ++j) {
            const int q = (g0 + j) * 16 + ld;
            uint32_t r, ow;
            a.dOW.divmod((uint32_t)(q < pb ? q : 0), r, ow);
            boff[j] = (int)r * a.sh * (kRegRowBytes / 16) + (((int)ow * a.sw) >> 1);
            coff[j] = q < pb ? ((n * a.OH + oh0 + (int)r) * a.OW + (int)ow) * (int)a.ys : -1;
        }
        // Each accumulator starts at its channels' biases (zero without a bias): the first step's
        // MFMAs take them as the C operand, so no zeroing and no bias add is needed per band.
        f32x4_t acc[NF][4];

        // Tap pair (kh, kw) = (t / kwp, t % kwp) of t = 8 kk + 2 lg, advanced by 8 taps per step
        // (kw even: a pair starts at an even pixel).
        int tkh = (2 * lg) / a.kwp, tkw = (2 * lg) % a.kwp;
        auto next_tap = [&](int kk) __attribute__((always_inline)) -> int {
            const int to = 8 * kk + 2 * lg < ntaps ? tkh * (kRegRowBytes / 16) + (tkw >> 1) : 0;   // pairs
            tkw += 8;
            if (tkw >= a.kwp) {                     // kwp >= 8: at most one wrap per step
                tkw -= a.kwp;
                ++tkh;
            }
            return to;
        };
        // One fragment per slot: slot j's fragment of step kk + 1 is read right after its MFMAs of
        // step kk, so it has the other slots' MFMAs to arrive.
        U4 fj[NF];
        {
            const int to = next_tap(0);
#pragma unroll
            for (int j = 0; j < NF; ++j) fj[j] = *reinterpret_cast<const U4 *>(cur + ((boff[j] + to) << 4));
        }
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            const int to = kk + 1 < KS ? next_tap(kk + 1) : 0;
            if (kk < nc) band_copy(nih0, nbase, kk, nxt);
            if (kk < UPW) store_one(kk);
#pragma unroll
            for (int j = 0; j < NF; ++j) {
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    if ((j > 0 || x >= S0) && (j < NF - 1 || x < LAST)) {
                        if (kk == 0) acc[j][x] = bvec[x];
                        Mfma<bf16_t>::run(acc[j][x], fw[kk][x], fj[j]);
                    }
                if (kk + 1 < KS) fj[j] = *reinterpret_cast<const U4 *>(cur + ((boff[j] + to) << 4));
            }
        }
        for (int c = KS; c < nc; ++c) band_copy(nih0, nbase, c, nxt);
#pragma unroll
        for (int u = KS; u < UPW; ++u) store_one(u);

        // bias + ReLU, rounded once (lane: channels co .. co + 3 of pixel 16 g + ld)
#pragma unroll
        for (int j = 0; j < NF; ++j) {
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                if (!((j > 0 || x >= S0) && (j < NF - 1 || x < LAST))) continue;
                float v4[4] = {acc[j][x][0], acc[j][x][1], acc[j][x][2], acc[j][x][3]};
                if (relu) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) v4[e] = v4[e] > 0.f ? v4[e] : 0.f;
                }
                held[j][x].x = pack_bf16x2(v4[0], v4[1]);
                held[j][x].y = pack_bf16x2(v4[2], v4[3]);
            }
        }
#pragma unroll
        for (int j = 0; j < NF; ++j) hoff[j] = coff[j];
        wait_barrier<0>();
    }
#pragma unroll
    for (int u = 0; u < UPW; ++u) store_one(u);
}

template <int KS, int UPW>
__global__ __launch_bounds__(256, 1) void band_fwd_reg_kernel(const BandArgs a) {
    static_assert(KS * 32 * 128 <= 2 * kRegBand, "filter staging");
    __shared__ __attribute__((aligned(1024))) unsigned char xb[2 * kRegBand];
    __shared__ __attribute__((aligned(16))) float sbias[64];    // the block's biases (0 past K)
    unsigned char *const xb0 = xb, *const xb1 = xb + kRegBand;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int co0 = blockIdx.y * 64;
    if (tid < 64) sbias[tid] = (a.bias != nullptr && co0 + tid < a.K) ? a.bias[co0 + tid] : 0.f;
    // Filter rows m = (kh * kwp + kw) * 4 + c (zero past the filter), k-major with the
    // transposing-read swizzle, staged over both band buffers: copy i covers rows 8 i .. 8 i + 7.
    for (int i = wave; i < KS * 4; i += 4) {
        const int m = 8 * i + (lane >> 3);
        const int ch = (lane & 7) ^ kmajor_swz<64>(m);
        const int c = m & 3;
        uint32_t kh, kw;
        a.dKwp.divmod((uint32_t)(m >> 2), kh, kw);
        const int co = co0 + ch * 8;
        const bool ok = (int)kh < a.KH && (int)kw < a.KW && c < a.C && co < a.K;
        dma16(ok ? (const void *)(a.w + (((int64_t)kh * a.KW + kw) * a.C + c) * a.K + co)
                 : (const void *)g_zero_chunk,
              xb0 + 1024 * i);
    }
    wait_barrier<0>();
    // wave-uniform choice of the run's offset into its first pixel group (UPW even: 0 or 2)
    static_assert(UPW % 2 == 0, "runs start at channel group 0 or 2");
    if (((UPW * wave) & 3) == 0)
        band_fwd_reg_body<KS, UPW, 0>(a, xb0, xb1, sbias, wave);
    else
        band_fwd_reg_body<KS, UPW, 2>(a, xb0, xb1, sbias, wave);
}

// ---------------------------------------------------------------------------------- bwd-filter
// Grid: (persistent workgroups = splits, output-channel blocks of 64).  The reduction rows are
// 16-row groups of 4 taps x 4 channels (taps t = kh * kwp + kw, kwp = KW rounded up to 4);
// wave w of NW owns groups w, w + NW, ..., w + NW (NG - 1) (groups past the filter are computed
// on valid addresses and dropped).  Eight waves (two per SIMD) keep twice the transposing LDS reads
// in flight of four, which the LDS needs to approach its bandwidth.  As in the forward kernel, the fragments of step kk + 1 are
// read while the MFMAs of step kk run.
template <int NG, bool X16, int NW>
__global__ __launch_bounds__(NW * 64, 1) void band_bwf_kernel(const BandArgs a) {
    __shared__ __attribute__((aligned(1024))) unsigned char xb0[kXBand];
    __shared__ __attribute__((aligned(1024))) unsigned char xb1[kXBand];
    __shared__ __attribute__((aligned(1024))) unsigned char db0[kDyBandPix * 128];
    __shared__ __attribute__((aligned(1024))) unsigned char db1[kDyBandPix * 128];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lg = lane >> 4, ld = lane & 15;
    const int co0 = blockIdx.y * 64;
    const int ngroups = a.KH * (a.kwp >> 2);

    // Byte offset of this lane's tap (group g = wave + NW y, tap 4 g + (ld & 3)) inside a staged band.
    int tapb[NG];
#pragma unroll
    for (int y = 0; y < NG; ++y) {
        const int g = wave + NW * y;
        const int t = 4 * (g < ngroups ? g : 0) + (ld & 3);
        uint32_t kh, kw;
        a.dKwp.divmod((uint32_t)t, kh, kw);
        tapb[y] = ((int)kh * a.wst + (int)kw) * 8;
    }

    // dy of band b: pixel p of the band at k-row p of a k-major [256][64] tile (zero past the
    // band), 32 direct-to-LDS copies spread over the waves: copy i covers k-rows 8 i .. 8 i + 7.
    constexpr int kDyCopies = kDyBandPix / (8 * NW);             // per wave
    auto dy_copy = [&](int b, unsigned char *buf, int j) __attribute__((always_inline)) {
        const int n = b / a.bands_per_img;
        const int oh0 = (b - n * a.bands_per_img) * a.R;
        const int pb = min(a.R, a.OH - oh0) * a.OW;
        const bf16_t *base = a.dy + ((int64_t)n * a.OH + oh0) * a.OW * a.ys + co0;
        const int i = wave + NW * j;
        const int k = 8 * i + (lane >> 3);
        const int ch = (lane & 7) ^ kmajor_swz<64>(k);
        const bool ok = k < pb && co0 + ch * 8 < a.K;
        dma16(ok ? (const void *)(base + (int64_t)k * a.ys + ch * 8) : (const void *)g_zero_chunk,
              buf + 1024 * i);
    };
    auto dy_dma = [&](int b, unsigned char *buf) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < kDyCopies; ++j) dy_copy(b, buf, j);
    };

    f32x4_t acc[4][NG];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < NG; ++y) acc[x][y] = fresh_zero4();

    int b = blockIdx.x * a.run;
    const int b_end = min(a.bands, b + a.run);
    if (b < b_end) {
        band_dma<X16, NW>(a, b, xb0);
        dy_dma(b, db0);
    }
    wait_barrier<0>();

    for (int it = 0; b < b_end; ++b, ++it) {
        const unsigned char *xc = (it & 1) ? xb1 : xb0;
        const unsigned char *dc = (it & 1) ? db1 : db0;
        const int bn = b + 1;
        if (bn < b_end) {
            band_dma<X16, NW>(a, bn, (it & 1) ? xb0 : xb1);
            dy_dma(bn, (it & 1) ? db0 : db1);
        }
        const int n = b / a.bands_per_img;
        const int oh0 = (b - n * a.bands_per_img) * a.R;
        const int pb = min(a.R, a.OH - oh0) * a.OW;
        const int nk = (pb + 31) >> 5;

        // Pixel bases of the lane's two k-rows of step kk inside the band (clamped: their dy rows
        // are zero), the dy fragments of a step, and the x fragment of one tap group.
        auto pix = [&](int kk, int (&pbase)[2]) __attribute__((always_inline)) {
            const int k0 = 32 * kk + 8 * lg + (ld >> 2);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int p = k0 + 4 * h;
                uint32_t r, ow;
                a.dOW.divmod((uint32_t)(p < pb ? p : 0), r, ow);
                pbase[h] = ((int)r * a.sh * a.wst + (int)ow * a.sw) * 8;
            }
        };
        auto load_dy = [&](int kk, U4 (&fi)[4]) __attribute__((always_inline)) {
            const int k0 = 32 * kk + 8 * lg + (ld >> 2);
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                const int row = 16 * x + 4 * (ld & 3);
                fi[x] = lds_tr_pair(dc + kmajor_off<64>(k0, row), dc + kmajor_off<64>(k0 + 4, row));
            }
        };
        auto load_x = [&](const int (&pbase)[2], int y) __attribute__((always_inline)) -> U4 {
            return lds_tr_pair(xc + pbase[0] + tapb[y], xc + pbase[1] + tapb[y]);
        };
        // One reduction step: the x fragment of group y is read L groups ahead (into slot y % (L + 1));
        // the dy fragments and the first L x fragments of step kk + 1 are read during step kk.
        constexpr int L = NG >= 2 ? 2 : 1;
        U4 fj[L + 1];
        auto step = [&](int kk, const U4 (&fic)[4], U4 (&fin)[4], const int (&pbc)[2], int (&pbn)[2])
                        __attribute__((always_inline)) {
            const bool more = kk + 1 < nk;
            if (more) {
                pix(kk + 1, pbn);
                load_dy(kk + 1, fin);
            }
            U4 nx[L];
#pragma unroll
            for (int y = 0; y < NG; ++y) {
                const int ya = y + L;
                if (ya < NG) fj[ya % (L + 1)] = load_x(pbc, ya);
                else if (more) nx[ya - NG] = load_x(pbn, ya - NG);
#pragma unroll
                for (int x = 0; x < 4; ++x) Mfma<bf16_t>::run(acc[x][y], fic[x], fj[y % (L + 1)]);
            }
            if (more) {
#pragma unroll
                for (int j = 0; j < L; ++j) fj[j] = nx[j];
            }
        };
        U4 fiA[4], fiB[4];
        int pbA[2], pbB[2];
        if (nk > 0) {
            pix(0, pbA);
            load_dy(0, fiA);
#pragma unroll
            for (int j = 0; j < L; ++j) fj[j] = load_x(pbA, j);
        }
        int kk = 0;
        for (; kk + 2 <= nk; kk += 2) {
            step(kk, fiA, fiB, pbA, pbB);
            step(kk + 1, fiB, fiA, pbB, pbA);
        }
        if (kk < nk) step(kk, fiA, fiB, pbA, pbB);

        wait_barrier<0>();
    }

    // Partial of this workgroup: lane holds channels co0 + 16 x + 4 lg .. + 3 of reduction row
    // 16 g + ld = (tap 4 g + ld / 4, channel ld % 4).
    float *part = reinterpret_cast<float *>(a.out) + (int64_t)blockIdx.x * a.KH * a.KW * a.C * a.K;
#pragma unroll
    for (int y = 0; y < NG; ++y) {
        const int g = wave + NW * y;
        if (g >= ngroups) continue;
        const int t = 4 * g + (ld >> 2), c = ld & 3;
        uint32_t kh, kw;
        a.dKwp.divmod((uint32_t)t, kh, kw);
        if ((int)kw >= a.KW || c >= a.C) continue;
        float *o = part + (((int64_t)kh * a.KW + (int)kw) * a.C + c) * a.K;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const int co = co0 + 16 * x + 4 * lg;
            if (co < a.K) *reinterpret_cast<f32x4_t *>(o + co) = acc[x][y];
        }
    }
}

void fill_band_args(BandArgs &a, const ConvShape &s) {
    a.N = s.N; a.H = s.H; a.W = s.W; a.C = s.C;
    a.OH = s.OH; a.OW = s.OW; a.K = s.K;
    a.KH = s.KH; a.KW = s.KW; a.sh = s.sh; a.sw = s.sw; a.pt = s.pt; a.pl = s.pl;
}

// Band height: the most output rows whose input rows fit one staged band (and, for bwd-filter,
// whose pixels fit the dy tile).
int band_rows(const ConvShape &s, int wst, int max_pix) {
    int R = 0;
    for (int r = 1; r <= s.OH; ++r) {
        const int rows_in = (r - 1) * s.sh + s.KH;
        if ((int64_t)rows_in * wst > kBandPix || (max_pix > 0 && r * s.OW > max_pix)) break;
        R = r;
    }
    return R;
}

// Consecutive bands of an image share KH - sh input rows; a workgroup takes a run of consecutive
// bands, so those rows are read again from its L2 instead of from memory.  Runs are as long as
// one band per CU at most would need: ceil(bands / CUs).
void set_runs(BandArgs &a) { a.run = (a.bands + kCUs - 1) / kCUs; }
int band_grid(const BandArgs &a) { return (a.bands + a.run - 1) / a.run; }

bool plan(const ConvShape &s, bool bwf, BandArgs &a) {
    if (s.C > 4 || s.K % 16 != 0) return false;
    const int kwp = bwf ? (s.KW + 3) / 4 * 4 : (s.KW + 1) / 2 * 2;
    int wst = (s.OW - 1) * s.sw + kwp;
    wst += wst & 1;
    if (bwf) {
        if (s.KH * (kwp / 4) > kBwfGroups || s.KH * (kwp / 4) < 4) return false;
    } else {
        const int nks = ((s.KH * kwp * 4 + 63) / 64) * 2;     // even: the loop runs two steps at a time
        if (nks > kMaxKSteps) return false;
        a.nks = nks;
    }
    const int R = band_rows(s, wst, bwf ? kDyBandPix : 0);
    if (R < 1) return false;
    fill_band_args(a, s);
    a.kwp = kwp;
    a.wst = wst;
    a.R = R;
    a.rows_in = (R - 1) * s.sh + s.KH;
    a.bands_per_img = (s.OH + R - 1) / R;
    const int64_t bands = (int64_t)s.N * a.bands_per_img;
    if (bands > (1 << 30)) return false;
    a.bands = (int)bands;
    set_runs(a);
    a.dWst.init((uint32_t)wst);
    a.dOW.init((uint32_t)s.OW);
    a.dKwp.init((uint32_t)kwp);
    return true;
}

int bwf_splits(const BandArgs &a) { return band_grid(a); }

// 16-byte band copies need pixel pairs that never straddle the image edge.
bool pairs_aligned(const ConvShape &s) { return s.pl % 2 == 0 && s.W % 2 == 0; }

constexpr int kBwfWaves = 8;

template <bool X16>
void launch_bwf(int ng, dim3 grid, const BandArgs &a, hipStream_t st) {
    constexpr int W = kBwfWaves;
    const dim3 blk(64 * W);
    switch (ng) {
    case 1: hipLaunchKernelGGL((band_bwf_kernel<1, X16, W>), grid, blk, 0, st, a); break;
    case 2: hipLaunchKernelGGL((band_bwf_kernel<2, X16, W>), grid, blk, 0, st, a); break;
    case 3: hipLaunchKernelGGL((band_bwf_kernel<3, X16, W>), grid, blk, 0, st, a); break;
    case 4: hipLaunchKernelGGL((band_bwf_kernel<4, X16, W>), grid, blk, 0, st, a); break;
    default: hipLaunchKernelGGL((band_bwf_kernel<5, X16, W>), grid, blk, 0, st, a); break;
    }
}

}  // namespace

bool conv_band_fwd_applies(const ConvShape &s) {
    BandArgs a;
    return plan(s, false, a);
}

bool conv_band_bwf_applies(const ConvShape &s) {
    BandArgs a;
    return plan(s, true, a);
}

size_t conv_band_bwf_partial_bytes(const ConvShape &s) {
    BandArgs a;
    if (!plan(s, true, a)) return 0;
    return (size_t)bwf_splits(a) * s.KH * s.KW * s.C * s.K * sizeof(float);
}

// x4: 4-element pixels (pixel stride 4), 8-byte aligned; y 8-byte aligned with ys % 4 == 0.
hipError_t launch_conv_fwd_band(const bf16_t *x4, const void *w, void *y, int64_t ys, const ConvShape &s,
                                const float *bias, hipStream_t st) {
    BandArgs a;
    if (!plan(s, false, a)) return hipErrorInvalidValue;
    a.x = x4;
    a.w = reinterpret_cast<const bf16_t *>(w);
    a.dy = nullptr;
    a.out = y;
    a.bias = bias;
    a.ys = ys;
    const dim3 grid((unsigned)band_grid(a), (unsigned)((s.K + 63) / 64));
    const bool x16 = pairs_aligned(s);
    constexpr int kRegKS = 17, kRegUPW = 14;    // AlexNet conv1: 11 x 12 taps x 4 channels, 4 rows of 55
    const int ks = (s.KH * a.kwp * 4 + 31) / 32;
    if (ks == kRegKS && s.sw % 2 == 0 && x16 && (int64_t)s.N * s.OH * s.OW * ys < (int64_t)1 << 31) {
        const int R = band_rows(s, a.wst, 16 * kRegUPW);
        if (R >= 1 && (R * s.OW + 15) / 16 == kRegUPW && (R - 1) * s.sh + s.KH <= kRegMaxRows &&
            a.wst <= kRegRowBytes / 8 && a.kwp >= 8) {
            a.R = R;
            a.rows_in = (R - 1) * s.sh + s.KH;
            a.bands_per_img = (s.OH + R - 1) / R;
            a.bands = s.N * a.bands_per_img;
            set_runs(a);
            const dim3 g2((unsigned)band_grid(a), (unsigned)((s.K + 63) / 64));
            hipLaunchKernelGGL((band_fwd_reg_kernel<kRegKS, kRegUPW>), g2, dim3(256), 0, st, a);
            return hipGetLastError();
        }
    }
    if (s.sw % 2 == 0 && x16)
        hipLaunchKernelGGL((band_fwd_kernel<true, true>), grid, dim3(256), 0, st, a);
    else if (s.sw % 2 == 0)
        hipLaunchKernelGGL((band_fwd_kernel<true, false>), grid, dim3(256), 0, st, a);
    else if (x16)
        hipLaunchKernelGGL((band_fwd_kernel<false, true>), grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL((band_fwd_kernel<false, false>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

// part: conv_band_bwf_partial_bytes(s) of workspace, 16-byte aligned; dy 16-byte aligned with dys % 8 == 0.
hipError_t launch_conv_bwd_filter_band(const bf16_t *x4, const void *dy, int64_t dys, float *dw, const ConvShape &s,
                                       float *part, hipStream_t st) {
    BandArgs a;
    if (!plan(s, true, a)) return hipErrorInvalidValue;
    a.x = x4;
    a.w = nullptr;
    a.dy = reinterpret_cast<const bf16_t *>(dy);
    a.out = part;
    a.bias = nullptr;
    a.ys = dys;
    a.nks = 0;
    const int splits = bwf_splits(a);
    const dim3 grid((unsigned)splits, (unsigned)((s.K + 63) / 64));
    const int ng = (s.KH * (a.kwp / 4) + kBwfWaves - 1) / kBwfWaves;     // 16-row tap groups per wave
    if (pairs_aligned(s))
        launch_bwf<true>(ng, grid, a, st);
    else
        launch_bwf<false>(ng, grid, a, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_sum_splits(part, splits, (int64_t)s.KH * s.KW * s.C * s.K, dw, st);
}

}  // namespace tfk
