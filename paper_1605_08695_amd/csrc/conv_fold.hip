// Convolutions whose input channel count is not a multiple of 8 (first layers
// on RGB images) in bf16, rewritten as an equivalent convolution that the
// pipelined 16-byte-chunk kernels can run.
//
// The input is copied with its channels zero-padded to Cp (4 for RGB) -- or read in
// place when its pixels are already Cp channels apart -- and F = 8 / Cp horizontally
// adjacent pixels are read as one "virtual pixel" of 8 channels (the same bytes:
// [N][H][W][Cp] is [N][H][W/F][F*Cp]).  With
// F | stride_w, F | pad_left and F | W, the column tap kw = F j + p of output
// column ow reads virtual column ow (stride_w/F) - pad_left/F + j, element p of
// the pair.  So the convolution equals one over the virtual image with
// ceil(KW/F) column taps, horizontal stride stride_w/F and left pad pad_left/F,
// whose filter holds w[kh][F j + p][c][co] at [kh][j][p Cp + c][co] (zero for
// padded channels and for taps beyond KW).  The filter gradient of the virtual
// convolution is folded back the same way.  AlexNet's conv1 (11x11/4, pad 2,
// 224 wide, 3 channels) becomes an 11x6 convolution of stride (4, 2) over
// 8-channel virtual pixels: 528 reduction elements per output instead of 363,
// against 968 for plain zero-padding to 8 channels.
#include "igemm_launch.h"

namespace tfk {

namespace {

struct Fold {
    int F, Cp;        // pixels per virtual pixel, padded channels per pixel
    ConvShape v;      // the virtual convolution
};

// Picks the widest fold that divides stride, left pad and width; F = 1 is plain padding to 8.
bool fold_plan(const ConvShape &s, Fold &f) {
    if (s.C % 8 == 0 || s.C > 8) return false;
    for (int F = 8; F >= 1; F >>= 1) {
        const int Cp = 8 / F;
        if (Cp < s.C || s.sw % F || s.pl % F || s.W % F) continue;
        ConvShape v = s;
        v.C = 8;
        v.W = s.W / F;
        v.KW = (s.KW + F - 1) / F;
        v.sw = s.sw / F;
        v.pl = s.pl / F;
        // v keeps OW: the kernels index outputs by OW and treat columns past the
        // virtual image as zeros, exactly like the original padding.
        f.F = F;
        f.Cp = Cp;
        f.v = v;
        return true;
    }
    return false;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// x [N][H][W][C] (pixel stride xs) -> xp [N][H][W][Cp], channels >= C zero.
__global__ __launch_bounds__(256) void pad_channels_kernel(const bf16_t *__restrict__ x, int64_t npix, int C,
                                                           int64_t xs, int Cp, bf16_t *__restrict__ xp) {
    const int64_t total = npix * Cp;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = t / Cp;
        const int c = (int)(t - p * Cp);
        xp[t] = c < C ? x[p * xs + c] : (bf16_t)0;
    }
}

// w [KH][KW][C][K] -> wv [KH][KWv][8][K]: wv[kh][j][p Cp + c][co] = w[kh][F j + p][c][co].
__global__ __launch_bounds__(256) void fold_filter_kernel(const bf16_t *__restrict__ w, int KH, int KW, int C,
                                                          int K, int F, int Cp, int KWv, bf16_t *__restrict__ wv) {
    const int64_t total = (int64_t)KH * KWv * 8 * K;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int co = (int)(t % K);
        const int e = (int)((t / K) % 8);
        const int j = (int)((t / (8 * K)) % KWv);
        const int kh = (int)(t / ((int64_t)8 * K * KWv));
        const int p = e / Cp, c = e % Cp;
        const int kw = F * j + p;
        wv[t] = (kw < KW && c < C) ? w[(((int64_t)kh * KW + kw) * C + c) * K + co] : (bf16_t)0;
    }
}

// dwv [KH][KWv][8][K] (fp32) -> dw [KH][KW][C][K]: dw[kh][kw][c][co] = dwv[kh][kw/F][(kw%F) Cp + c][co].
__global__ __launch_bounds__(256) void unfold_filter_grad_kernel(const float *__restrict__ dwv, int KH, int KW, int C,
                                                                 int K, int F, int Cp, int KWv, float *__restrict__ dw) {
    const int64_t total = (int64_t)KH * KW * C * K;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int co = (int)(t % K);
        const int c = (int)((t / K) % C);
        const int kw = (int)((t / ((int64_t)K * C)) % KW);
        const int kh = (int)(t / ((int64_t)K * C * KW));
        dw[t] = dwv[(((int64_t)kh * KWv + kw / F) * 8 + (kw % F) * Cp + c) * K + co];
    }
}

// Dense input, 8 pixels per thread: 8 C elements arrive as C 16-byte loads and leave
// as Cp 16-byte stores (C, Cp <= 8); the last npix % 8 pixels take the kernel above.
template <int C, int Cp>
__global__ __launch_bounds__(256) void pad_channels_vec_kernel(const bf16_t *__restrict__ x, int64_t groups,
                                                               bf16_t *__restrict__ xp) {
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < groups;
         g += (int64_t)gridDim.x * blockDim.x) {
        uint32_t in[32];
        const U4 *src = reinterpret_cast<const U4 *>(x + g * 8 * C);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (q < C) {
                const U4 v = src[q];
                in[4 * q] = v.x; in[4 * q + 1] = v.y; in[4 * q + 2] = v.z; in[4 * q + 3] = v.w;
            }
        }
        U4 *dst = reinterpret_cast<U4 *>(xp + g * 8 * Cp);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (q < Cp) {
                uint32_t o[4];
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    uint32_t word = 0;
#pragma unroll
                    for (int half = 0; half < 2; ++half) {
                        const int e = (q * 4 + h) * 2 + half;       // output element within the 8 pixels
                        const int pix = e / Cp, c = e % Cp;
                        if (c < C) {
                            const int i = pix * C + c;              // input element
                            const uint32_t bits = (in[i >> 1] >> ((i & 1) * 16)) & 0xffffu;
                            word |= bits << (half * 16);
                        }
                    }
                    o[h] = word;
                }
                U4 v;
                v.x = o[0]; v.y = o[1]; v.z = o[2]; v.w = o[3];
                dst[q] = v;
            }
        }
    }
}

int grid_of(int64_t n) { return (int)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 16384)); }

template <int C, int Cp>
bool pad_vec(const bf16_t *x, int64_t groups, bf16_t *xp, hipStream_t st) {
    hipLaunchKernelGGL((pad_channels_vec_kernel<C, Cp>), dim3(grid_of(groups)), dim3(256), 0, st, x, groups, xp);
    return true;
}

// The 16-byte path for the channel counts of image inputs.
bool pad_vec_dispatch(int C, int Cp, const bf16_t *x, int64_t groups, bf16_t *xp, hipStream_t st) {
    if (C == 3 && Cp == 4) return pad_vec<3, 4>(x, groups, xp, st);
    if (C == 3 && Cp == 8) return pad_vec<3, 8>(x, groups, xp, st);
    if (C == 1 && Cp == 8) return pad_vec<1, 8>(x, groups, xp, st);
    if (C == 1 && Cp == 1) return pad_vec<1, 1>(x, groups, xp, st);
    if (C == 4 && Cp == 8) return pad_vec<4, 8>(x, groups, xp, st);
    return false;
}

// The padded input the virtual convolution reads: x itself when its pixels are already Cp
// channels apart (a C-channel view of a Cp-channel buffer: the channels past C meet zero
// filter weights, so they only have to be finite), else a padded copy in the workspace.
const bf16_t *padded_input(const void *x, int64_t npix, int C, int64_t xs, int Cp, bf16_t *xp, hipStream_t st);

void pad_channels(const void *x, int64_t npix, int C, int64_t xs, int Cp, bf16_t *xp, hipStream_t st) {
    const bf16_t *xb = reinterpret_cast<const bf16_t *>(x);
    int64_t done = 0;
    const int64_t groups = npix / 8;
    if (xs == C && ((uintptr_t)x & 15) == 0 && groups > 0 && pad_vec_dispatch(C, Cp, xb, groups, xp, st))
        done = groups * 8;
    if (done < npix)
        hipLaunchKernelGGL(pad_channels_kernel, dim3(grid_of((npix - done) * Cp)), dim3(256), 0, st,
                           xb + done * xs, npix - done, C, xs, Cp, xp + done * Cp);
}

const bf16_t *padded_input(const void *x, int64_t npix, int C, int64_t xs, int Cp, bf16_t *xp, hipStream_t st) {
    if (xs == Cp && ((uintptr_t)x & 15) == 0) return reinterpret_cast<const bf16_t *>(x);
    pad_channels(x, npix, C, xs, Cp, xp, st);
    return xp;
}

}  // namespace

const bf16_t *rgbx_input(const void *x, int64_t npix, int C, int64_t xs, bf16_t *xp, hipStream_t st) {
    if (xs == 4 && ((uintptr_t)x & 7) == 0) return reinterpret_cast<const bf16_t *>(x);
    pad_channels(x, npix, C, xs, 4, xp, st);
    return xp;
}

bool conv_fold_applies(int dt, const ConvShape &s) {
    Fold f;
    return dt == 1 && s.K % 8 == 0 && fold_plan(s, f);
}

// Workspace layout: [padded x][folded filter or its gradient][bwd-filter partial sums].
size_t conv_fold_ws_bytes(int op, const ConvShape &s) {
    Fold f;
    if (!fold_plan(s, f)) return 0;
    const size_t xb = align256((size_t)s.N * s.H * s.W * f.Cp * 2);
    const size_t wvn = (size_t)s.KH * f.v.KW * 8 * s.K;
    if (op == 0) return xb + align256(wvn * 2);
    return xb + align256(wvn * 4) + align256(conv_bwd_filter_ws_bytes(1, f.v));
}

hipError_t launch_conv_fwd_folded(const void *x, int64_t xs, const void *w, void *y, int64_t ys, const ConvShape &s,
                                  const float *bias, void *ws, hipStream_t st) {
    Fold f;
    fold_plan(s, f);
    unsigned char *base = reinterpret_cast<unsigned char *>(ws);
    bf16_t *xp = reinterpret_cast<bf16_t *>(base);
    bf16_t *wv = reinterpret_cast<bf16_t *>(base + align256((size_t)s.N * s.H * s.W * f.Cp * 2));
    const int64_t npix = (int64_t)s.N * s.H * s.W;
    const bf16_t *xin = padded_input(x, npix, s.C, xs, f.Cp, xp, st);
    hipLaunchKernelGGL(fold_filter_kernel, dim3(grid_of((int64_t)s.KH * f.v.KW * 8 * s.K)), dim3(256), 0, st,
                       reinterpret_cast<const bf16_t *>(w), s.KH, s.KW, s.C, s.K, f.F, f.Cp, f.v.KW, wv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_conv_fwd(1, xin, 8, wv, y, ys, f.v, bias, nullptr, st);
}

hipError_t launch_conv_bwd_filter_folded(const void *x, int64_t xs, const void *dy, int64_t dys, float *dw,
                                         const ConvShape &s, void *ws, hipStream_t st) {
    Fold f;
    fold_plan(s, f);
    unsigned char *base = reinterpret_cast<unsigned char *>(ws);
    const size_t xb = align256((size_t)s.N * s.H * s.W * f.Cp * 2);
    const size_t wvn = (size_t)s.KH * f.v.KW * 8 * s.K;
    bf16_t *xp = reinterpret_cast<bf16_t *>(base);
    float *dwv = reinterpret_cast<float *>(base + xb);
    void *ws2 = base + xb + align256(wvn * 4);
    const int64_t npix = (int64_t)s.N * s.H * s.W;
    const bf16_t *xin = padded_input(x, npix, s.C, xs, f.Cp, xp, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_conv_bwd_filter(1, xin, 8, dy, dys, dwv, f.v, ws2, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(unfold_filter_grad_kernel, dim3(grid_of((int64_t)s.KH * s.KW * s.C * s.K)), dim3(256), 0, st,
                       dwv, s.KH, s.KW, s.C, s.K, f.F, f.Cp, f.v.KW, dw);
    return hipGetLastError();
}

}  // namespace tfk
