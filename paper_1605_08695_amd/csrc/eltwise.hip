// Bandwidth-bound kernels of the training step on gfx950: fused bias+ReLU
// forward/backward with the bias-gradient reduction, max-pool forward/backward
// with argmax, the in-place SGD update, and the split-K sum of bwd-filter.
//
// Every kernel moves 16-byte chunks (8 bf16 or 4 fp32 channels) when the
// channel count, pixel stride and base pointers allow it, and falls back to
// one element per thread otherwise.  Reductions are two-pass with a fixed
// order, so results do not depend on scheduling.
#include "common.h"
#include <type_traits>

#include "kernels.h"

namespace tfk {

static inline int grid_for(int64_t work, int per_block = 256, int cap = 65536) {
    int64_t g = (work + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

// ------------------------------------------------------------------ chunk helpers
template <typename T>
__device__ __forceinline__ void chunk_to_f32(const U4 &v, float *f) {
    if constexpr (sizeof(T) == 4) {
        f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
    } else {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f[2 * j] = __uint_as_float(w[j] << 16);
            f[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
        }
    }
}

// v[e] <- +0 where element e of the chunk m is not positive (the ReLU gradient mask)
template <typename T>
__device__ __forceinline__ void relu_mask(const U4 &m, float *v) {
    constexpr int EPC = Elem<T>::kPerChunk;
    float f[EPC];
    chunk_to_f32<T>(m, f);
#pragma unroll
    for (int e = 0; e < EPC; ++e) v[e] = f[e] > 0.f ? v[e] : 0.f;
}

template <typename T>
__device__ __forceinline__ U4 f32_to_chunk(const float *f) {
    U4 v;
    if constexpr (sizeof(T) == 4) {
        v.x = __float_as_uint(f[0]); v.y = __float_as_uint(f[1]);
        v.z = __float_as_uint(f[2]); v.w = __float_as_uint(f[3]);
    } else {
        v.x = pack_bf16x2(f[0], f[1]); v.y = pack_bf16x2(f[2], f[3]);
        v.z = pack_bf16x2(f[4], f[5]); v.w = pack_bf16x2(f[6], f[7]);
    }
    return v;
}

// ------------------------------------------------------------------ bias + ReLU forward
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void bias_relu_fwd_kernel(T *__restrict__ y, int64_t P, int C,
                                                            int64_t ys, const float *__restrict__ bias,
                                                            FastDiv dCV) {
    constexpr int EPC = VEC ? Elem<T>::kPerChunk : 1;
    const int CV = C / EPC;
    const int64_t total = P * CV;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int64_t p;
        int cv;
        if (total < (1ll << 31)) {
            uint32_t q, r;
            dCV.divmod((uint32_t)t, q, r);
            p = q;
            cv = (int)r;
        } else {
            p = t / CV;
            cv = (int)(t - p * CV);
        }
        T *ptr = y + p * ys + (int64_t)cv * EPC;
        if constexpr (VEC) {
            float f[EPC];
            chunk_to_f32<T>(*reinterpret_cast<const U4 *>(ptr), f);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float v = f[e] + bias[cv * EPC + e];
                f[e] = v > 0.f ? v : 0.f;
            }
            *reinterpret_cast<U4 *>(ptr) = f32_to_chunk<T>(f);
        } else {
            const float v = Elem<T>::load(ptr) + bias[cv];
            Elem<T>::store(ptr, v > 0.f ? v : 0.f);
        }
    }
}

// ------------------------------------------------------------------ ReLU backward + bias gradient
// Pass 1: block b owns pixels [b*ppb, min(P, (b+1)*ppb)).  Thread t owns channel
// chunks cv = t % CVB (+ CVB, ...) and pixel rows t / CVB (+ R, ...).  It writes
// dpre and keeps fp32 per-channel sums; the block then reduces its R row groups
// in LDS in a fixed order and writes partial[c][b].
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void relu_bwd_partial_kernel(const T *__restrict__ y, const T *dy,
                                                               T *dpre, int64_t P, int C, int64_t ys,
                                                               int64_t ppb, float *__restrict__ partial) {
    constexpr int EPC = VEC ? Elem<T>::kPerChunk : 1;
    extern __shared__ float red[];                 // [R][C]
    const int CV = C / EPC;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    const int t = threadIdx.x;
    const int lane_cv = t % CVB;
    const int row = t / CVB;
    const int64_t p0 = (int64_t)blockIdx.x * ppb;
    const int64_t p1 = min(P, p0 + ppb);
    const bool active = row < R;
    for (int cv = lane_cv; cv < CV; cv += CVB) {
        float s[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) s[e] = 0.f;
        if (active) {
            if constexpr (VEC) {
                // Four pixels per iteration, all loads issued before the first store (dpre may be
                // dy itself, so the compiler cannot move a later pixel's loads above a store); the
                // pixels are still summed in ascending order.
                constexpr int U = 4;
                for (int64_t p = p0 + row; p < p1; p += (int64_t)R * U) {
                    U4 ly[U], ld[U];
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const int64_t pp = p + (int64_t)u * R;
                        if (pp < p1) {
                            const int64_t off = pp * ys + (int64_t)cv * EPC;
                            if (y != nullptr) ly[u] = *reinterpret_cast<const U4 *>(y + off);
                            ld[u] = *reinterpret_cast<const U4 *>(dy + off);
                        }
                    }
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const int64_t pp = p + (int64_t)u * R;
                        if (pp >= p1) break;
                        const int64_t off = pp * ys + (int64_t)cv * EPC;
                        float fy[EPC], fd[EPC];
                        if (y != nullptr) {
                            chunk_to_f32<T>(ly[u], fy);
                        } else {
#pragma unroll
                            for (int e = 0; e < EPC; ++e) fy[e] = 1.f;
                        }
                        chunk_to_f32<T>(ld[u], fd);
#pragma unroll
                        for (int e = 0; e < EPC; ++e) {
                            fd[e] = fy[e] > 0.f ? fd[e] : 0.f;
                            s[e] += fd[e];
                        }
                        *reinterpret_cast<U4 *>(dpre + off) = f32_to_chunk<T>(fd);
                    }
                }
            }
            for (int64_t p = p0 + row; !VEC && p < p1; p += R) {
                const int64_t off = p * ys + (int64_t)cv * EPC;
                if constexpr (VEC) {
                } else {
                    const float fy = y != nullptr ? Elem<T>::load(y + off) : 1.f;
                    const float fd = fy > 0.f ? Elem<T>::load(dy + off) : 0.f;
                    s[0] += fd;
                    Elem<T>::store(dpre + off, fd);
                }
            }
            // The stored dpre equals the value summed here: with bf16 storage the
            // masked dy is already a bf16 value, so rounding on store is exact.
            if (R == 1) {                    // one row group: the partial directly (no LDS)
#pragma unroll
                for (int e = 0; e < EPC; ++e) partial[(int64_t)(cv * EPC + e) * gridDim.x + blockIdx.x] = s[e];
            } else {
#pragma unroll
                for (int e = 0; e < EPC; ++e) red[row * C + cv * EPC + e] = s[e];
            }
        }
    }
    if (R == 1) return;
    __syncthreads();
    for (int c = t; c < C; c += 256) {
        float acc = 0.f;
        for (int r = 0; r < R; ++r) acc += red[r * C + c];
        partial[(int64_t)c * gridDim.x + blockIdx.x] = acc;
    }
}

// Pass 2: one block per channel sums its G partials (stored channel-major, so the reads are
// contiguous): thread t takes b = t, t + 256, ... in order (the loads of 16 consecutive b of one
// thread are issued together before they are added, in the same order), then a fixed xor tree
// combines the 64 lanes of each wave and thread 0 adds the four wave sums in wave order.
// One channel's G partials, summed by a block of 256 threads in a fixed order (strided runs per
// thread, a wave shuffle tree, the four wave sums in order); the result is valid in thread 0.
__device__ __forceinline__ float sum_partial_row(const float *__restrict__ row, int G, float *wsum) {
    float acc = 0.f;
    constexpr int U = 16;
    for (int b0 = threadIdx.x; b0 < G; b0 += 256 * U) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int b = b0 + u * 256;
            v[u] = b < G ? row[b] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (b0 + u * 256 < G) acc += v[u];
    }
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) acc += __shfl_xor(acc, m, 64);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = acc;
    __syncthreads();
    return ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

__global__ __launch_bounds__(256) void sum_partials_kernel(const float *__restrict__ partial, int G, int C,
                                                           float *__restrict__ out) {
    __shared__ float wsum[4];
    const int c = blockIdx.x;
    const float t = sum_partial_row(partial + (int64_t)c * G, G, wsum);
    if (threadIdx.x == 0) out[c] = t;
}

// Several tensors' partials in one launch: block b is channel b - chan0[i] of job i
// (chan0[i] <= b < chan0[i + 1]), summed as sum_partials_kernel sums it.
__global__ __launch_bounds__(256) void sum_partials_multi_kernel(const PartialsBatch jobs) {
    __shared__ float wsum[4];
    const int b = blockIdx.x;
    int i = 0;
    while (i + 1 < jobs.count && b >= jobs.chan0[i + 1]) ++i;
    const int c = b - jobs.chan0[i];
    const float t = sum_partial_row(jobs.part[i] + (int64_t)c * jobs.rows[i], jobs.rows[i], wsum);
    if (threadIdx.x == 0) jobs.out[i][c] = t;
}

// ------------------------------------------------------------------ pixel decomposition
// t = ((n * E2 + i2) * E1 + i1) * CV + cv.  Below 2^31 work items it is three 32-bit
// multiply-high divisions; 64-bit division (a long instruction sequence) only beyond.
struct Decode {
    FastDiv dcv, d1, d2;
    int64_t cv, e1, e2;
    bool small;
};

static Decode make_decode(int64_t cv, int64_t e1, int64_t e2, int64_t total) {
    Decode d;
    d.cv = cv;
    d.e1 = e1;
    d.e2 = e2;
    d.small = total < (1ll << 31);
    d.dcv.init((uint32_t)cv);
    d.d1.init((uint32_t)e1);
    d.d2.init((uint32_t)e2);
    return d;
}

__device__ __forceinline__ void decode(const Decode &d, int64_t t, int &cv, int64_t &pix, int &i1, int &i2, int &n) {
    if (d.small) {
        uint32_t q, r, q2, r2, q3, r3;
        d.dcv.divmod((uint32_t)t, q, r);
        d.d1.divmod(q, q2, r2);
        d.d2.divmod(q2, q3, r3);
        cv = (int)r;
        pix = q;
        i1 = (int)r2;
        i2 = (int)r3;
        n = (int)q3;
    } else {
        cv = (int)(t % d.cv);
        pix = t / d.cv;
        i1 = (int)(pix % d.e1);
        const int64_t q = pix / d.e1;
        i2 = (int)(q % d.e2);
        n = (int)(q / d.e2);
    }
}

// Index arithmetic of the pool kernels: 64-bit, or (O32: pixel counts, strides and channel
// counts below 2^24 and element offsets below 2^29, checked by the host with pool_o32) 32-bit with
// full-rate 24-bit multiplies in place of quarter-rate 64-bit ones.
template <bool O32>
struct PoolIx {
    typedef typename std::conditional<O32, uint32_t, int64_t>::type I;
    static __device__ __forceinline__ I mul(I a, I b) {
        if constexpr (O32) return __umul24(a, b);
        else return a * b;
    }
};

// ------------------------------------------------------------------ argmax formats
// A max-pool records, per output element, which input element its window selected: as the
// dense NHWC index of that element (int32_t) or as the window tap kh * KW + kw (uint8_t, a
// quarter of the bytes).  arg_enc gives the stored value of tap `tap` whose element has dense
// index `dense`; arg_store / arg_load move the N values of one channel chunk.
template <typename A> __device__ __forceinline__ int32_t arg_enc(int32_t dense, int tap);
template <> __device__ __forceinline__ int32_t arg_enc<int32_t>(int32_t dense, int) { return dense; }
template <> __device__ __forceinline__ int32_t arg_enc<uint8_t>(int32_t, int tap) { return tap; }

template <typename A, int N>
__device__ __forceinline__ void arg_store(A *p, const int32_t *v) {
    if constexpr (sizeof(A) == 4 && N % 4 == 0) {
#pragma unroll
        for (int e = 0; e < N; e += 4) {
            int4 q;
            q.x = v[e]; q.y = v[e + 1]; q.z = v[e + 2]; q.w = v[e + 3];
            *reinterpret_cast<int4 *>(p + e) = q;
        }
    } else if constexpr (sizeof(A) == 1 && N == 8) {
        uint2 q;
        q.x = (uint32_t)v[0] | ((uint32_t)v[1] << 8) | ((uint32_t)v[2] << 16) | ((uint32_t)v[3] << 24);
        q.y = (uint32_t)v[4] | ((uint32_t)v[5] << 8) | ((uint32_t)v[6] << 16) | ((uint32_t)v[7] << 24);
        *reinterpret_cast<uint2 *>(p) = q;
    } else if constexpr (sizeof(A) == 1 && N == 4) {
        *reinterpret_cast<uint32_t *>(p) =
            (uint32_t)v[0] | ((uint32_t)v[1] << 8) | ((uint32_t)v[2] << 16) | ((uint32_t)v[3] << 24);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) p[e] = (A)v[e];
    }
}

template <typename A, int N>
__device__ __forceinline__ void arg_load(const A *p, int32_t *v) {
    if constexpr (sizeof(A) == 4 && N % 4 == 0) {
#pragma unroll
        for (int e = 0; e < N; e += 4) {
            const int4 q = *reinterpret_cast<const int4 *>(p + e);
            v[e] = q.x; v[e + 1] = q.y; v[e + 2] = q.z; v[e + 3] = q.w;
        }
    } else if constexpr (sizeof(A) == 1 && N == 8) {
        const uint2 q = *reinterpret_cast<const uint2 *>(p);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[e] = (int32_t)((q.x >> (8 * e)) & 0xffu);
            v[e + 4] = (int32_t)((q.y >> (8 * e)) & 0xffu);
        }
    } else if constexpr (sizeof(A) == 1 && N == 4) {
        const uint32_t q = *reinterpret_cast<const uint32_t *>(p);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (int32_t)((q >> (8 * e)) & 0xffu);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = (int32_t)p[e];
    }
}

// ------------------------------------------------------------------ max-pool forward
template <typename T, bool VEC, typename A>
__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const T *__restrict__ x, PoolGeom g,
                                                          T *__restrict__ y, A *__restrict__ argmax, Decode dec) {
    constexpr int EPC = VEC ? Elem<T>::kPerChunk : 1;
    const int CV = g.C / EPC;
    const int64_t total = (int64_t)g.N * g.OH * g.OW * CV;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int cv, ow, oh, n;
        int64_t pix;
        decode(dec, t, cv, pix, ow, oh, n);
        float best[EPC];
        int32_t bi[EPC];
        bool have = false;
        for (int kh = 0; kh < g.KH; ++kh) {
            const int ih = oh * g.sh + kh - g.pt;
            if ((unsigned)ih >= (unsigned)g.H) continue;
            for (int kw = 0; kw < g.KW; ++kw) {
                const int iw = ow * g.sw + kw - g.pl;
                if ((unsigned)iw >= (unsigned)g.W) continue;
                const int64_t pidx = ((int64_t)n * g.H + ih) * g.W + iw;
                const int32_t dense = (int32_t)(pidx * g.C + cv * EPC);
                const int tap = kh * g.KW + kw;
                float v[EPC];
                if constexpr (VEC) {
                    chunk_to_f32<T>(*reinterpret_cast<const U4 *>(x + pidx * g.xs + cv * EPC), v);
                } else {
                    v[0] = Elem<T>::load(x + pidx * g.xs + cv);
                }
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    if (!have || v[e] > best[e]) {
                        best[e] = v[e];
                        bi[e] = arg_enc<A>(dense + e, tap);
                    }
                }
                have = true;
            }
        }
        const int64_t opix = ((int64_t)n * g.OH + oh) * g.OW + ow;
        if constexpr (VEC) {
            *reinterpret_cast<U4 *>(y + opix * g.ys + cv * EPC) = f32_to_chunk<T>(best);
            arg_store<A, EPC>(argmax + opix * g.C + cv * EPC, bi);
        } else {
            Elem<T>::store(y + opix * g.ys + cv, best[0]);
            argmax[opix * g.C + cv] = (A)bi[0];
        }
    }
}

// Fixed small windows (3x3, 2x2) on the 16-byte path: the window loop is unrolled and all of a
// thread's loads are issued before the first comparison, so their latencies overlap (the
// run-time loop above waits for each tap in turn).  Same scan order and tie rule.
template <typename T, int KH, int KW, typename A, bool O32>
__global__ __launch_bounds__(256) void maxpool_fwd_win_kernel(const T *__restrict__ x, PoolGeom g,
                                                              T *__restrict__ y, A *__restrict__ argmax,
                                                              Decode dec) {
    constexpr int EPC = Elem<T>::kPerChunk;
    typedef PoolIx<O32> M;
    typedef typename M::I I;
    const int CV = g.C / EPC;
    const int64_t total = (int64_t)g.N * g.OH * g.OW * CV;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int cv, ow, oh, n;
        int64_t pix;
        decode(dec, t, cv, pix, ow, oh, n);
        U4 v[KH * KW];
        bool ok[KH * KW];
        I pidx[KH * KW];
#pragma unroll
        for (int kh = 0; kh < KH; ++kh) {
#pragma unroll
            for (int kw = 0; kw < KW; ++kw) {
                const int q = kh * KW + kw;
                const int ih = oh * g.sh + kh - g.pt, iw = ow * g.sw + kw - g.pl;
                ok[q] = (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
                pidx[q] = M::mul(M::mul((I)n, (I)g.H) + (I)(ok[q] ? ih : 0), (I)g.W) + (I)(ok[q] ? iw : 0);
                v[q] = *reinterpret_cast<const U4 *>(x + (M::mul(pidx[q], (I)g.xs) + (I)(cv * EPC)));
            }
        }
        const I opix = M::mul(M::mul((I)n, (I)g.OH) + (I)oh, (I)g.OW) + (I)ow;
        if constexpr (std::is_same<T, bf16_t>::value && std::is_same<A, uint8_t>::value) {
            // Chunks with no sign bit in any tap (a ReLU's output): there bf16 bit patterns order
            // as their values, so each element keeps the largest (bits << 8 | 255 - tap) over its
            // taps -- one byte permute and one integer max per element and tap -- and a tie goes
            // to the first tap, as the strict > of the scan below gives it.  A sign bit (a
            // negative value or -0) or a NaN maximum leaves the chunk to that scan.
            uint32_t sg = 0;
#pragma unroll
            for (int q = 0; q < KH * KW; ++q)
                if (ok[q]) sg |= v[q].x | v[q].y | v[q].z | v[q].w;
            if ((sg & 0x80008000u) == 0) {
                uint32_t kb[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) kb[e] = 0u;
#pragma unroll
                for (int q = 0; q < KH * KW; ++q) {
                    if (!ok[q]) continue;
                    const uint32_t c = 255u - (uint32_t)q;
                    const uint32_t d[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        // (bytes: the tap code, then the element's two bytes, then zero)
                        kb[2 * w] = max(kb[2 * w], __builtin_amdgcn_perm(d[w], c, 0x0C050400u));
                        kb[2 * w + 1] = max(kb[2 * w + 1], __builtin_amdgcn_perm(d[w], c, 0x0C070600u));
                    }
                }
                uint32_t top = 0;
#pragma unroll
                for (int e = 0; e < 8; ++e) top = max(top, kb[e]);
                if ((top >> 8) <= 0x7F80u) {          // no NaN (+inf is 0x7F80)
                    U4 o;
                    o.x = __builtin_amdgcn_perm(kb[1], kb[0], 0x06050201u);
                    o.y = __builtin_amdgcn_perm(kb[3], kb[2], 0x06050201u);
                    o.z = __builtin_amdgcn_perm(kb[5], kb[4], 0x06050201u);
                    o.w = __builtin_amdgcn_perm(kb[7], kb[6], 0x06050201u);
                    int32_t tq[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) tq[e] = 255 - (int32_t)(kb[e] & 0xFFu);
                    *reinterpret_cast<U4 *>(y + (M::mul(opix, (I)g.ys) + (I)(cv * EPC))) = o;
                    arg_store<A, EPC>(argmax + (M::mul(opix, (I)g.C) + (I)(cv * EPC)), tq);
                    continue;
                }
            }
        }
        float best[EPC];
        int32_t bi[EPC];
        bool have = false;
#pragma unroll
        for (int q = 0; q < KH * KW; ++q) {
            if (!ok[q]) continue;
            float f[EPC];
            chunk_to_f32<T>(v[q], f);
            const int32_t dense = (int32_t)(M::mul(pidx[q], (I)g.C) + (I)(cv * EPC));
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                if (!have || f[e] > best[e]) {
                    best[e] = f[e];
                    bi[e] = arg_enc<A>(dense + e, q);
                }
            }
            have = true;
        }
        *reinterpret_cast<U4 *>(y + (M::mul(opix, (I)g.ys) + (I)(cv * EPC))) = f32_to_chunk<T>(best);
        arg_store<A, EPC>(argmax + (M::mul(opix, (I)g.C) + (I)(cv * EPC)), bi);
    }
}

// ------------------------------------------------------------------ max-pool backward
// Gather form: each input element visits the windows that contain it in
// ascending output order and adds the gradients routed to it.
// s[e] (e < EPC) = sum of dy over the windows whose argmax is input element
// pix * C + cv * EPC + e, pixel pix = (n, h, w) of the pool input.
// (A: argmax format.  Element e of the chunk matches window (oh, ow) when the window's stored
// value is self + e (dense index) or this pixel's tap in that window (tap index).)
// py (optional, pixel stride pys): the pool's output; a window whose output element is not
// positive routes +0 instead of its dy (the ReLU mask of the element its argmax names, whose
// value the window's output is).
template <typename T, bool VEC, typename A, bool O32 = false>
__device__ __forceinline__ void pool_gather(const T *__restrict__ dy, const A *__restrict__ argmax,
                                            const PoolGeom &g, int n, int h, int w, int64_t pix, int cv,
                                            float *s, const T *__restrict__ py = nullptr, int64_t pys = 0) {
    constexpr int EPC = VEC ? Elem<T>::kPerChunk : 1;
    constexpr bool TAP = sizeof(A) == 1;
    typedef PoolIx<O32> M;
    typedef typename M::I I;
    const int32_t self = (int32_t)(M::mul((I)pix, (I)g.C) + (I)(cv * EPC));
    const I nrow = M::mul((I)n, (I)g.OH);
    auto want = [&](int oh, int ow, int e) __attribute__((always_inline)) -> int32_t {
        if constexpr (TAP) return (h + g.pt - oh * g.sh) * g.KW + (w + g.pl - ow * g.sw);
        else return self + e;
    };
    if constexpr (VEC) {
        // At most NC x NC windows contain the element (NC = 2: windows no larger than twice the
        // stride; NC = 3: three times, e.g. 3 x 3 windows at stride 1): issue every argmax and dy
        // load of all the candidates first (clamped to a valid window, masked afterwards), so the
        // gather costs one memory round trip instead of one or two per window.
        auto candidates = [&](auto NC_) __attribute__((always_inline)) {
            constexpr int NC = decltype(NC_)::value;
            const int hp = h + g.pt, wp = w + g.pl;
            const int oh_lo = hp - g.KH + 1 <= 0 ? 0 : (hp - g.KH + 1 + g.sh - 1) / g.sh;
            const int oh_hi = min(g.OH - 1, hp / g.sh);
            const int ow_lo = wp - g.KW + 1 <= 0 ? 0 : (wp - g.KW + 1 + g.sw - 1) / g.sw;
            const int ow_hi = min(g.OW - 1, wp / g.sw);
            // (an element no window reaches has oh_lo > oh_hi; its loads go to the last window)
            const int ohc = min(oh_lo, g.OH - 1), owc = min(ow_lo, g.OW - 1);
            int32_t ai[NC * NC][EPC];
            U4 dv[NC * NC], pv[NC * NC];
            bool valid[NC * NC];
#pragma unroll
            for (int q = 0; q < NC * NC; ++q) {
                const int oh = oh_lo + q / NC, ow = ow_lo + q % NC;
                valid[q] = oh <= oh_hi && ow <= ow_hi;
                const I opix = M::mul(nrow + (I)(valid[q] ? oh : ohc), (I)g.OW) + (I)(valid[q] ? ow : owc);
                arg_load<A, EPC>(argmax + (M::mul(opix, (I)g.C) + (I)(cv * EPC)), ai[q]);
                dv[q] = *reinterpret_cast<const U4 *>(dy + (M::mul(opix, (I)g.ys) + (I)(cv * EPC)));
                if (py) pv[q] = *reinterpret_cast<const U4 *>(py + (M::mul(opix, (I)pys) + (I)(cv * EPC)));
            }
#pragma unroll
            for (int e = 0; e < EPC; ++e) s[e] = 0.f;
#pragma unroll
            for (int q = 0; q < NC * NC; ++q) {       // windows in ascending output order
                float v[EPC];
                chunk_to_f32<T>(dv[q], v);
                if (py) relu_mask<T>(pv[q], v);
                const int oh = oh_lo + q / NC, ow = ow_lo + q % NC;
#pragma unroll
                for (int e = 0; e < EPC; ++e)
                    if (valid[q] && ai[q][e] == want(oh, ow, e)) s[e] += v[e];
            }
        };
        if (g.KH <= 2 * g.sh && g.KW <= 2 * g.sw) {
            candidates(std::integral_constant<int, 2>{});
            return;
        }
        if (g.KH <= 3 * g.sh && g.KW <= 3 * g.sw) {
            candidates(std::integral_constant<int, 3>{});
            return;
        }
    }
    // windows oh with oh*sh - pt <= h <= oh*sh - pt + KH - 1
    const int hp = h + g.pt, wp = w + g.pl;
    const int oh_lo = hp - g.KH + 1 <= 0 ? 0 : (hp - g.KH + 1 + g.sh - 1) / g.sh;
    const int oh_hi = min(g.OH - 1, hp / g.sh);
    const int ow_lo = wp - g.KW + 1 <= 0 ? 0 : (wp - g.KW + 1 + g.sw - 1) / g.sw;
    const int ow_hi = min(g.OW - 1, wp / g.sw);
#pragma unroll
    for (int e = 0; e < EPC; ++e) s[e] = 0.f;
    for (int oh = oh_lo; oh <= oh_hi; ++oh) {
        for (int ow = ow_lo; ow <= ow_hi; ++ow) {
            const int64_t opix = ((int64_t)n * g.OH + oh) * g.OW + ow;
            if constexpr (VEC) {
                int32_t ai[EPC];
                arg_load<A, EPC>(argmax + opix * g.C + cv * EPC, ai);
                bool any = false;
#pragma unroll
                for (int e = 0; e < EPC; ++e) any |= (ai[e] == want(oh, ow, e));
                if (any) {
                    float v[EPC];
                    chunk_to_f32<T>(*reinterpret_cast<const U4 *>(dy + opix * g.ys + cv * EPC), v);
                    if (py) relu_mask<T>(*reinterpret_cast<const U4 *>(py + opix * pys + cv * EPC), v);
#pragma unroll
                    for (int e = 0; e < EPC; ++e)
                        if (ai[e] == want(oh, ow, e)) s[e] += v[e];
                }
            } else {
                if ((int32_t)argmax[opix * g.C + cv] == want(oh, ow, 0))
                    s[0] += py && !(Elem<T>::load(py + opix * pys + cv) > 0.f) ? 0.f : Elem<T>::load(dy + opix * g.ys + cv);
            }
        }
    }
}

template <typename T, bool VEC, typename A, bool O32>
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const T *__restrict__ dy,
                                                          const A *__restrict__ argmax, PoolGeom g,
                                                          float beta, T *dx, Decode dec) {
    constexpr int EPC = VEC ? Elem<T>::kPerChunk : 1;
    typedef PoolIx<O32> M;
    typedef typename M::I I;
    const int CV = g.C / EPC;
    const int64_t total = (int64_t)g.N * g.H * g.W * CV;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int cv, w, h, n;
        int64_t pix;
        decode(dec, t, cv, pix, w, h, n);
        float s[EPC];
        pool_gather<T, VEC, A, O32>(dy, argmax, g, n, h, w, pix, cv, s);
        T *out = dx + (M::mul((I)pix, (I)g.xs) + (I)(cv * EPC));
        if constexpr (VEC) {
            if (beta != 0.f) {
                float o[EPC];
                chunk_to_f32<T>(*reinterpret_cast<const U4 *>(out), o);
#pragma unroll
                for (int e = 0; e < EPC; ++e) s[e] += beta * o[e];
            }
            *reinterpret_cast<U4 *>(out) = f32_to_chunk<T>(s);
        } else {
            if (beta != 0.f) s[0] += beta * Elem<T>::load(out);
            Elem<T>::store(out, s[0]);
        }
    }
}

// ------------------------------------------------------------------ max-pool + ReLU + bias backward
// One pass over the pool input (= the ReLU output y of the convolution before it):
//   dpre = (y > 0) ? (beta * dpre + sum of routed dy) : 0,   db[c] = sum over pixels of dpre.
// The thread layout and the fixed-order bias-gradient reduction are those of
// relu_bwd_partial_kernel: block b owns pixels [b ppb, (b+1) ppb), thread t channel chunk
// t % CVB (+ CVB ...) and pixel rows t / CVB (+ R ...); db sums the stored (rounded) dpre,
// the tensor the filter gradient is formed from.
// With py (the pool's output, pixel stride pys; beta = 0 only) the mask is taken per window
// from it instead of per element from y, which is not read: an element receives gradient only
// from windows whose argmax it is, and each such window's output is the element's value.
template <typename T, bool VEC, typename A, bool O32>
__global__ __launch_bounds__(256) void maxpool_relu_bwd_partial_kernel(const T *__restrict__ dy,
                                                                       const A *__restrict__ argmax,
                                                                       PoolGeom g, const T *__restrict__ y,
                                                                       const T *__restrict__ py, int64_t pys, T *dpre,
                                                                       float beta, int64_t ppb, FastDiv dW, FastDiv dH,
                                                                       float *__restrict__ partial) {
    constexpr int EPC = VEC ? Elem<T>::kPerChunk : 1;
    extern __shared__ float red[];                 // [R][C]
    const int C = g.C;
    const int CV = C / EPC;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    const int t = threadIdx.x;
    const int lane_cv = t % CVB;
    const int row = t / CVB;
    const int64_t P = (int64_t)g.N * g.H * g.W;
    const int64_t p0 = (int64_t)blockIdx.x * ppb;
    const int64_t p1 = min(P, p0 + ppb);
    const bool active = row < R;
    for (int cv = lane_cv; cv < CV; cv += CVB) {
        float acc[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
        if (active) {
            for (int64_t p = p0 + row; p < p1; p += R) {
                uint32_t q, w, n, h;
                dW.divmod((uint32_t)p, q, w);
                dH.divmod(q, n, h);
                float s[EPC];
                pool_gather<T, VEC, A, O32>(dy, argmax, g, (int)n, (int)h, (int)w, p, cv, s, py, pys);
                typedef PoolIx<O32> M;
                const typename M::I off = M::mul((typename M::I)p, (typename M::I)g.xs) + (typename M::I)(cv * EPC);
                if constexpr (VEC) {
                    if (beta != 0.f) {
                        float o[EPC];
                        chunk_to_f32<T>(*reinterpret_cast<const U4 *>(dpre + off), o);
#pragma unroll
                        for (int e = 0; e < EPC; ++e) s[e] += beta * o[e];
                    }
                    if (!py) relu_mask<T>(*reinterpret_cast<const U4 *>(y + off), s);
                    const U4 packed = f32_to_chunk<T>(s);
                    *reinterpret_cast<U4 *>(dpre + off) = packed;
                    float st[EPC];
                    chunk_to_f32<T>(packed, st);           // the stored values
#pragma unroll
                    for (int e = 0; e < EPC; ++e) acc[e] += st[e];
                } else {
                    if (beta != 0.f) s[0] += beta * Elem<T>::load(dpre + off);
                    const float v = py || Elem<T>::load(y + off) > 0.f ? s[0] : 0.f;
                    Elem<T>::store(dpre + off, v);
                    acc[0] += Elem<T>::load(dpre + off);
                }
            }
#pragma unroll
            for (int e = 0; e < EPC; ++e) red[row * C + cv * EPC + e] = acc[e];
        }
    }
    __syncthreads();
    for (int c = t; c < C; c += 256) {
        float a = 0.f;
        for (int r = 0; r < R; ++r) a += red[r * C + c];
        partial[(int64_t)c * gridDim.x + blockIdx.x] = a;
    }
}

// Stride-2 pools with windows of at most 4 x 4 (AlexNet 3x3/2, VGG 2x2/2): thread work item =
// one 2 x 2 "cell" of input pixels (rows 2 ch - pt + {0,1}, columns 2 cw - pl + {0,1}) and
// one channel chunk.  Only windows ch-1, ch (rows) x cw-1, cw (columns) can hold the argmax
// of a cell pixel, so their argmax and dy are loaded once for all four pixels (the gather
// form reloads them for every pixel) and each window's gradient is routed to the pixel its
// argmax names, windows in ascending order (the same sums, in the same order, as the gather).
// Bias-gradient partials as in maxpool_relu_bwd_partial_kernel, over cells instead of pixels.
// PK > 0: the windows are PK x PK (a compile-time size, so the window/pixel pairs that can never
// match are dropped: 9 of 16 remain for 3 x 3); PK = 0: the size comes from g.
// py: as in maxpool_relu_bwd_partial_kernel (the four windows' outputs replace the four pixels'
// y as the mask).
// O32: pixel indices below 2^24 and element offsets below 2^29 (checked by the host), so the index
// arithmetic runs in 32 bits with full-rate 24-bit multiplies instead of quarter-rate 64-bit ones.
template <typename T, typename A, int PK, bool O32>
__global__ __launch_bounds__(256) void maxpool_relu_bwd_cell_kernel(const T *__restrict__ dy,
                                                                    const A *__restrict__ argmax, PoolGeom g,
                                                                    const T *__restrict__ y,
                                                                    const T *__restrict__ py, int64_t pys,
                                                                    T *dpre, float beta,
                                                                    int64_t cpb, int CH, int CW, FastDiv dCW,
                                                                    FastDiv dCH, float *__restrict__ partial) {
    constexpr int EPC = Elem<T>::kPerChunk;
    extern __shared__ float red[];                 // [R][C]
    const int C = g.C;
    const int CV = C / EPC;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    const int t = threadIdx.x;
    const int lane_cv = t % CVB;
    const int row = t / CVB;
    const int64_t ncell = (int64_t)g.N * CH * CW;
    const int64_t c0 = (int64_t)blockIdx.x * cpb;
    const int64_t c1 = min(ncell, c0 + cpb);
    const bool active = row < R;
    using Ix = typename std::conditional<O32, uint32_t, int64_t>::type;
    auto mul = [](Ix a, Ix b) __attribute__((always_inline)) -> Ix {
        if constexpr (O32) return __umul24(a, b);
        else return a * b;
    };
    for (int cv = lane_cv; cv < CV; cv += CVB) {
        float acc[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
        if (active) {
            for (int64_t cell = c0 + row; cell < c1; cell += R) {
                uint32_t q, cw, n, ch;
                dCW.divmod((uint32_t)cell, q, cw);
                dCH.divmod(q, n, ch);
                // the (up to) four windows, in ascending output order
                int32_t ai[4][EPC];
                U4 dv[4], pv[4];
                bool wok[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int oh = (int)ch - 1 + (k >> 1), ow = (int)cw - 1 + (k & 1);
                    wok[k] = (unsigned)oh < (unsigned)g.OH && (unsigned)ow < (unsigned)g.OW;
                    const Ix opix = mul(mul((Ix)n, (Ix)g.OH) + (Ix)(wok[k] ? oh : 0), (Ix)g.OW) + (Ix)(wok[k] ? ow : 0);
                    arg_load<A, EPC>(argmax + (mul(opix, (Ix)g.C) + (Ix)(cv * EPC)), ai[k]);
                    dv[k] = *reinterpret_cast<const U4 *>(dy + (mul(opix, (Ix)g.ys) + (Ix)(cv * EPC)));
                    if (py) pv[k] = *reinterpret_cast<const U4 *>(py + (mul(opix, (Ix)pys) + (Ix)(cv * EPC)));
                }
                // the four pixels of the cell
                Ix pix[4], poff[4];
                bool pok[4];
                U4 yv[4], ov[4];
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const int h = 2 * (int)ch - g.pt + (m >> 1), w = 2 * (int)cw - g.pl + (m & 1);
                    pok[m] = (unsigned)h < (unsigned)g.H && (unsigned)w < (unsigned)g.W;
                    pix[m] = mul(mul((Ix)n, (Ix)g.H) + (Ix)(pok[m] ? h : 0), (Ix)g.W) + (Ix)(pok[m] ? w : 0);
                    poff[m] = mul(pix[m], (Ix)g.xs) + (Ix)(cv * EPC);
                    if (!py) yv[m] = *reinterpret_cast<const U4 *>(y + poff[m]);
                    if (beta != 0.f) ov[m] = *reinterpret_cast<const U4 *>(dpre + poff[m]);
                }
                float s[4][EPC];
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int e = 0; e < EPC; ++e) s[m][e] = 0.f;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    float v[EPC];
                    chunk_to_f32<T>(dv[k], v);
                    if (py) relu_mask<T>(pv[k], v);
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        // pixel m is tap (2 (1 - k/2) + m/2, 2 (1 - k%2) + m%2) of window k
                        const int th = 2 * (1 - (k >> 1)) + (m >> 1), tw = 2 * (1 - (k & 1)) + (m & 1);
                        const int KH = PK > 0 ? PK : g.KH, KW = PK > 0 ? PK : g.KW;
                        if (PK > 0 && sizeof(A) == 1 && (th >= KH || tw >= KW)) continue;
                        const int32_t self = sizeof(A) == 1 ? (th < KH && tw < KW ? th * KW + tw : -1)
                                                            : (int32_t)(mul(pix[m], (Ix)g.C) + (Ix)(cv * EPC));
#pragma unroll
                        for (int e = 0; e < EPC; ++e)
                            if (wok[k] && ai[k][e] == self + (sizeof(A) == 1 ? 0 : e)) s[m][e] += v[e];
                    }
                }
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    if (!pok[m]) continue;
                    if (beta != 0.f) {
                        float o[EPC];
                        chunk_to_f32<T>(ov[m], o);
#pragma unroll
                        for (int e = 0; e < EPC; ++e) s[m][e] += beta * o[e];
                    }
                    if (!py) relu_mask<T>(yv[m], s[m]);
                    const U4 packed = f32_to_chunk<T>(s[m]);
                    *reinterpret_cast<U4 *>(dpre + poff[m]) = packed;
                    float st[EPC];
                    chunk_to_f32<T>(packed, st);
#pragma unroll
                    for (int e = 0; e < EPC; ++e) acc[e] += st[e];
                }
            }
#pragma unroll
            for (int e = 0; e < EPC; ++e) red[row * C + cv * EPC + e] = acc[e];
        }
    }
    __syncthreads();
    for (int c = t; c < C; c += 256) {
        float a = 0.f;
        for (int r = 0; r < R; ++r) a += red[r * C + c];
        partial[(int64_t)c * gridDim.x + blockIdx.x] = a;
    }
}

// ------------------------------------------------------------------ SGD
// The variable updates stream each operand once: 16-byte non-temporal loads and stores (the
// streams are not re-read by the update, so they should not displace cached activations).
typedef float f4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f4v stream_load(const float *p, int64_t t) {
    return __builtin_nontemporal_load(reinterpret_cast<const f4v *>(p) + t);
}
__device__ __forceinline__ void stream_store(float *p, int64_t t, f4v v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f4v *>(p) + t);
}

__device__ __forceinline__ void sgd_one(float *var, const float *grad, uint16_t *sh, int64_t i, float lr) {
    const float v = fmaf(-lr, grad[i], var[i]);
    var[i] = v;
    if (sh) sh[i] = (uint16_t)f32_to_bf16(v);
}

__global__ __launch_bounds__(256) void sgd_kernel(float *__restrict__ var, const float *__restrict__ grad,
                                                  int64_t n, float lr, uint16_t *__restrict__ sh, bool vec) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (vec) {
        const int64_t n4 = n / 4;
        for (int64_t t = t0; t < n4; t += stride) {
            f4v v = stream_load(var, t);
            const f4v g = stream_load(grad, t);
            v.x = fmaf(-lr, g.x, v.x); v.y = fmaf(-lr, g.y, v.y);
            v.z = fmaf(-lr, g.z, v.z); v.w = fmaf(-lr, g.w, v.w);
            stream_store(var, t, v);
            if (sh) {
                uint2 b;
                b.x = pack_bf16x2(v.x, v.y);
                b.y = pack_bf16x2(v.z, v.w);
                reinterpret_cast<uint2 *>(sh)[t] = b;
            }
        }
        for (int64_t i = n4 * 4 + t0; i < n; i += stride) sgd_one(var, grad, sh, i, lr);
    } else {
        for (int64_t i = t0; i < n; i += stride) sgd_one(var, grad, sh, i, lr);
    }
}

__global__ __launch_bounds__(256) void sgd_multi_kernel(SgdBatch b, float lr) {
    int k = 0;
    while (k + 1 < b.count && (int64_t)blockIdx.x >= b.blk_start[k + 1]) ++k;
    const int64_t first = ((int64_t)blockIdx.x - b.blk_start[k]) * 256 * 4;
    float *var = b.var[k];
    const float *grad = b.grad[k];
    uint16_t *sh = b.shadow[k];
    const int64_t n = b.n[k];
    for (int r = 0; r < 4; ++r) {
        const int64_t i = first + r * 256 + threadIdx.x;
        if (i < n) sgd_one(var, grad, sh, i, lr);
    }
}

// ------------------------------------------------------------------ Momentum, Adam
// Both keep the SGD kernel's shape: one pass over the flat variable, float4 loads and stores of
// every operand when all are 16-byte aligned, the optional bf16 shadow written beside the var.
// KIND 0: Momentum (s1 = velocity), 1: Momentum look-ahead form, 2: Adam (s1 = m, s2 = v).
template <int KIND>
__device__ __forceinline__ float opt_elem(float var, float &s1, float &s2, float g, const OptParams &p) {
    if (KIND == 2) {
        const float m = fmaf(p.b1, s1, p.omb1 * g);
        const float v = fmaf(p.b2, s2, (p.omb2 * g) * g);
        s1 = m;
        s2 = v;
        const float den = sqrtf(v * p.rc2) + p.eps;
        return fmaf(-p.lr, m / den, var);
    }
    const float a = fmaf(p.mom, s1, g);
    s1 = a;
    return fmaf(-p.lr, KIND == 1 ? fmaf(p.mom, a, g) : a, var);
}

template <int KIND>
__global__ __launch_bounds__(256) void opt_kernel(float *__restrict__ var, float *__restrict__ s1,
                                                  float *__restrict__ s2, const float *__restrict__ grad,
                                                  int64_t n, OptParams p, uint16_t *__restrict__ sh, bool vec) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t tail = 0;
    if (vec) {
        const int64_t n4 = n / 4;
        tail = n4 * 4;
        for (int64_t t = t0; t < n4; t += stride) {
            f4v v = stream_load(var, t), a = stream_load(s1, t);
            f4v b = KIND == 2 ? stream_load(s2, t) : f4v{0.f, 0.f, 0.f, 0.f};
            const f4v g = stream_load(grad, t);
            float ax = a.x, ay = a.y, az = a.z, aw = a.w, bx = b.x, by = b.y, bz = b.z, bw = b.w;
            v.x = opt_elem<KIND>(v.x, ax, bx, g.x, p);
            v.y = opt_elem<KIND>(v.y, ay, by, g.y, p);
            v.z = opt_elem<KIND>(v.z, az, bz, g.z, p);
            v.w = opt_elem<KIND>(v.w, aw, bw, g.w, p);
            stream_store(var, t, v);
            stream_store(s1, t, f4v{ax, ay, az, aw});
            if (KIND == 2) stream_store(s2, t, f4v{bx, by, bz, bw});
            if (sh) {
                uint2 q;
                q.x = pack_bf16x2(v.x, v.y);
                q.y = pack_bf16x2(v.z, v.w);
                reinterpret_cast<uint2 *>(sh)[t] = q;
            }
        }
    }
    for (int64_t i = tail + t0; i < n; i += stride) {
        float a = s1[i], b = KIND == 2 ? s2[i] : 0.f;
        const float v = opt_elem<KIND>(var[i], a, b, grad[i], p);
        var[i] = v;
        s1[i] = a;
        if (KIND == 2) s2[i] = b;
        if (sh) sh[i] = (uint16_t)f32_to_bf16(v);
    }
}

// Fixed xor-tree reductions across one wave.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// ------------------------------------------------------------------ sampled softmax
// Gather of candidate rows as the columns of a d x u_pad filter: out_t[k][j] = table[idx[j]][k]
// (zero for j >= u or an index outside [0, rows)).  Thread: one (k, j); consecutive threads
// write consecutive j.
template <typename T>
__global__ __launch_bounds__(256) void gather_rows_t_kernel(const T *__restrict__ table, int64_t rows, int d,
                                                            const int32_t *__restrict__ idx, int u, int u_pad,
                                                            T *__restrict__ out_t) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (int64_t)d * u_pad) return;
    const int k = (int)(t / u_pad), j = (int)(t - (int64_t)k * u_pad);
    T v = T(0);
    if (j < u) {
        const int64_t r = idx[j];
        if (r >= 0 && r < rows) v = table[r * d + k];
    }
    out_t[t] = v;
}

hipError_t launch_gather_rows_t(int dt, const void *table, int64_t rows, int d, const int32_t *idx, int u,
                                int u_pad, void *out_t, hipStream_t st) {
    const int64_t n = (int64_t)d * u_pad;
    const dim3 g((unsigned)((n + 255) / 256));
    if (dt == 0)
        hipLaunchKernelGGL(gather_rows_t_kernel<float>, g, dim3(256), 0, st, (const float *)table, rows, d, idx, u,
                           u_pad, (float *)out_t);
    else
        hipLaunchKernelGGL(gather_rows_t_kernel<uint16_t>, g, dim3(256), 0, st, (const uint16_t *)table, rows, d,
                           idx, u, u_pad, (uint16_t *)out_t);
    return hipGetLastError();
}

// Sampled softmax cross-entropy over candidate logits z (n x u_pad; columns j < m are the shared
// sample, tp[i] the column of row i's true class): one block per row, the same fixed reduction
// tree as softmax_xent_kernel.  Column j < m equal to tp[i] is an accidental hit and is left out.
template <typename T>
__global__ __launch_bounds__(256) void sampled_xent_kernel(const T *__restrict__ z, int u_pad, int m,
                                                           const float *__restrict__ bc, const int32_t *__restrict__ tp,
                                                           const float *__restrict__ lq_true,
                                                           const float *__restrict__ lq_sampled, float scale,
                                                           float *__restrict__ loss, T *__restrict__ dz, int u) {
    __shared__ float red[2][4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const T *zr = z + row * u_pad;
    T *dr = dz + row * u_pad;
    const int t = tp[row];
    if (t < 0 || t >= u) {                        // (uniform over the block)
        for (int j = tid; j < u_pad; j += 256) Elem<T>::store(dr + j, __builtin_nanf(""));
        if (tid == 0) loss[row] = __builtin_nanf("");
        return;
    }
    const float zt = Elem<T>::load(zr + t) + (bc ? bc[t] : 0.f) - lq_true[row];
    float mx = zt;
    for (int j = tid; j < m; j += 256)
        if (j != t) mx = fmaxf(mx, Elem<T>::load(zr + j) + (bc ? bc[j] : 0.f) - lq_sampled[j]);
    mx = wave_max(mx);
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    float sum = 0.f;
    for (int j = tid; j < m; j += 256)
        if (j != t) sum += expf(Elem<T>::load(zr + j) + (bc ? bc[j] : 0.f) - lq_sampled[j] - mx);
    sum = wave_sum(sum);
    if (lane == 0) red[1][wave] = sum;
    __syncthreads();
    const float et = expf(zt - mx);
    sum = (((red[1][0] + red[1][1]) + red[1][2]) + red[1][3]) + et;
    if (tid == 0) loss[row] = mx + logf(sum) - zt;
    const float inv = 1.f / sum;
    for (int j = tid; j < u_pad; j += 256) {
        float g = 0.f;
        if (j < m && j != t) g = scale * (expf(Elem<T>::load(zr + j) + (bc ? bc[j] : 0.f) - lq_sampled[j] - mx) * inv);
        if (j == t) g = scale * (et * inv - 1.f);
        Elem<T>::store(dr + j, g);
    }
}

hipError_t launch_sampled_xent(int dt, const void *z, int64_t n, int u, int u_pad, int m, const float *bc,
                               const int32_t *tp, const float *lq_true, const float *lq_sampled, float scale,
                               float *loss, void *dz, hipStream_t st) {
    if (dt == 0)
        hipLaunchKernelGGL(sampled_xent_kernel<float>, dim3((unsigned)n), dim3(256), 0, st, (const float *)z, u_pad, m,
                           bc, tp, lq_true, lq_sampled, scale, loss, (float *)dz, u);
    else
        hipLaunchKernelGGL(sampled_xent_kernel<bf16_t>, dim3((unsigned)n), dim3(256), 0, st, (const bf16_t *)z, u_pad,
                           m, bc, tp, lq_true, lq_sampled, scale, loss, (bf16_t *)dz, u);
    return hipGetLastError();
}

// Sparse in-place SGD of candidate rows: var[idx[j]][k] -= lr * grad_t[k][j] (j < u, k < d),
// the bf16 shadow beside.  The rows idx[j] are distinct (each element has one writer);
// an index outside [0, rows) is skipped.
__global__ __launch_bounds__(256) void scatter_sgd_kernel(float *__restrict__ var, uint16_t *__restrict__ sh,
                                                          int64_t rows, int d, const int32_t *__restrict__ idx, int u,
                                                          const float *__restrict__ grad_t, int64_t ld, float lr) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (int64_t)d * u) return;
    const int j = (int)(t / d), k = (int)(t - (int64_t)j * d);
    const int64_t r = idx[j];
    if (r < 0 || r >= rows) return;
    const int64_t o = r * d + k;
    const float v = fmaf(-lr, grad_t[(int64_t)k * ld + j], var[o]);
    var[o] = v;
    if (sh) sh[o] = (uint16_t)f32_to_bf16(v);
}

hipError_t launch_scatter_sgd(float *var, uint16_t *sh, int64_t rows, int d, const int32_t *idx, int u,
                              const float *grad_t, int64_t ld, float lr, hipStream_t st) {
    const int64_t n = (int64_t)d * u;
    hipLaunchKernelGGL(scatter_sgd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, var, sh, rows, d, idx,
                       u, grad_t, ld, lr);
    return hipGetLastError();
}

// ------------------------------------------------------------------ split-K epilogue
// One thread per output row j and group of four channels i (consecutive threads: consecutive
// groups of one row); the split partials are independent 16-byte loads, added in split order.
__global__ __launch_bounds__(256) void split_epilogue_kernel(SplitEpi e) {
    const int groups = e.ni / 4;
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int j = (int)(t / groups);
    if (j >= e.rows) return;
    const int i = (int)(t - (int64_t)j * groups) * 4;
    const float *p = e.part + (int64_t)j * e.ni + i;
    float4 v = *reinterpret_cast<const float4 *>(p);
    for (int s = 1; s < e.splits; ++s) {
        const float4 w = *reinterpret_cast<const float4 *>(p + (int64_t)s * e.split_stride);
        v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    float r[4] = {v.x, v.y, v.z, v.w};
    bf16_t *o = reinterpret_cast<bf16_t *>(e.out) + (int64_t)j * e.ostride + i;
    if (e.bias != nullptr)
        for (int q = 0; q < 4; ++q) r[q] = fmaxf(r[q] + e.bias[i + q], 0.f);
    if (e.beta != 0.f) {
        const uint2 old = *reinterpret_cast<const uint2 *>(o);
        r[0] += e.beta * bf16_to_f32(old.x & 0xffffu);
        r[1] += e.beta * bf16_to_f32(old.x >> 16);
        r[2] += e.beta * bf16_to_f32(old.y & 0xffffu);
        r[3] += e.beta * bf16_to_f32(old.y >> 16);
    }
    if (e.relu_y != nullptr) {
        const uint2 yv = *reinterpret_cast<const uint2 *>(reinterpret_cast<const bf16_t *>(e.relu_y) +
                                                          (int64_t)j * e.ostride + i);
        const float yq[4] = {bf16_to_f32(yv.x & 0xffffu), bf16_to_f32(yv.x >> 16), bf16_to_f32(yv.y & 0xffffu),
                             bf16_to_f32(yv.y >> 16)};
        for (int q = 0; q < 4; ++q) r[q] = yq[q] > 0.f ? r[q] : 0.f;
    }
    uint2 pk;
    pk.x = pack_bf16x2(r[0], r[1]);
    pk.y = pack_bf16x2(r[2], r[3]);
    *reinterpret_cast<uint2 *>(o) = pk;
    if (e.db_part != nullptr) {                   // this row's stored values: partial [i][j]
        e.db_part[(int64_t)(i + 0) * e.rows + j] = bf16_to_f32(pk.x & 0xffffu);
        e.db_part[(int64_t)(i + 1) * e.rows + j] = bf16_to_f32(pk.x >> 16);
        e.db_part[(int64_t)(i + 2) * e.rows + j] = bf16_to_f32(pk.y & 0xffffu);
        e.db_part[(int64_t)(i + 3) * e.rows + j] = bf16_to_f32(pk.y >> 16);
    }
}

hipError_t launch_split_epilogue(const SplitEpi &e, hipStream_t st) {
    const int64_t threads = (int64_t)(e.ni / 4) * e.rows;
    hipLaunchKernelGGL(split_epilogue_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, e);
    return hipGetLastError();
}

// ------------------------------------------------------------------ softmax cross-entropy
// One block of 256 threads per row of n x c logits (z = logits + bias): the row max, then the
// sum of exp(z - max), each reduced over the block by a fixed tree (xor shuffles inside each
// wave, then the four wave results in order), then the loss and the gradient
// scale * (softmax - onehot).  Each thread reads and writes only its own columns, so dz may be
// the logits buffer itself.
template <typename T>
__global__ __launch_bounds__(256) void softmax_xent_kernel(const T *z, const float *__restrict__ bias,
                                                           const int32_t *__restrict__ labels, int64_t n, int c,
                                                           float scale, float *__restrict__ loss, T *dz) {
    __shared__ float red[2][4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const T *zr = z + row * c;
    T *dr = dz + row * c;
    const int lab = labels[row];
    if (lab < 0 || lab >= c) {                    // (uniform over the block)
        for (int j = tid; j < c; j += 256) Elem<T>::store(dr + j, __builtin_nanf(""));
        if (tid == 0) loss[row] = __builtin_nanf("");
        return;
    }
    float m = -INFINITY;
    for (int j = tid; j < c; j += 256) m = fmaxf(m, Elem<T>::load(zr + j) + (bias ? bias[j] : 0.f));
    m = wave_max(m);
    if (lane == 0) red[0][wave] = m;
    __syncthreads();
    m = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    float sum = 0.f;
    for (int j = tid; j < c; j += 256) sum += expf(Elem<T>::load(zr + j) + (bias ? bias[j] : 0.f) - m);
    sum = wave_sum(sum);
    if (lane == 0) red[1][wave] = sum;
    __syncthreads();
    sum = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    if (tid == 0) loss[row] = m + logf(sum) - (Elem<T>::load(zr + lab) + (bias ? bias[lab] : 0.f));
    const float inv = 1.f / sum;
    for (int j = tid; j < c; j += 256) {
        const float p = expf(Elem<T>::load(zr + j) + (bias ? bias[j] : 0.f) - m) * inv;
        Elem<T>::store(dr + j, scale * (j == lab ? p - 1.f : p));
    }
}

hipError_t launch_softmax_xent(int dt, const void *z, const float *bias, const int32_t *labels, int64_t n, int c,
                               float scale, float *loss, void *dz, hipStream_t st) {
    if (dt == 0)
        hipLaunchKernelGGL(softmax_xent_kernel<float>, dim3((unsigned)n), dim3(256), 0, st, (const float *)z, bias,
                           labels, n, c, scale, loss, (float *)dz);
    else
        hipLaunchKernelGGL(softmax_xent_kernel<bf16_t>, dim3((unsigned)n), dim3(256), 0, st, (const bf16_t *)z, bias,
                           labels, n, c, scale, loss, (bf16_t *)dz);
    return hipGetLastError();
}

// ------------------------------------------------------------------ split-K sum / zero fill
// The split partials part[s][i] (s < splits, i < mn) are summed in a fixed order that depends
// only on the shape.  Large gradients: one pass, split order (sum_splits_direct_kernel).
// Small ones, in two fixed levels: groups of kSplitGroup consecutive splits are
// summed in split order (in place, into the group's first split), then the group sums are
// added in group order.  Each thread owns VEC consecutive elements of one group and issues
// all of the group's loads before adding, so a reduction over many splits of a small
// filter gradient still has enough loads in flight.
constexpr int kSplitGroup = 16;

template <int VEC>
struct FVec;
template <> struct FVec<1> { typedef float T; };
template <> struct FVec<4> { typedef f32x4_t T; };

template <int VEC>
__global__ __launch_bounds__(256) void sum_split_groups_kernel(float *__restrict__ part, int splits, int64_t mn,
                                                               int groups) {
    typedef typename FVec<VEC>::T V;
    const int64_t mv = mn / VEC;
    const int64_t total = mv * groups;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int g = (int)(t / mv);
        const int64_t i = t - (int64_t)g * mv;
        const int s0 = g * kSplitGroup;
        const int n = min(kSplitGroup, splits - s0);
        V *base = reinterpret_cast<V *>(part + (int64_t)s0 * mn) + i;
        V v[kSplitGroup];
#pragma unroll
        for (int s = 0; s < kSplitGroup; ++s)
            if (s < n) v[s] = base[(int64_t)s * mv];
        V acc = v[0];
#pragma unroll
        for (int s = 1; s < kSplitGroup; ++s)
            if (s < n) acc += v[s];
        base[0] = acc;
    }
}

template <int VEC>
__global__ __launch_bounds__(256) void sum_groups_kernel(const float *__restrict__ part, int groups, int64_t mn,
                                                         float *__restrict__ out) {
    typedef typename FVec<VEC>::T V;
    const int64_t mv = mn / VEC;
    const int64_t gstride = (int64_t)kSplitGroup * mv;      // between the first splits of two groups
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < mv; i += stride) {
        const V *src = reinterpret_cast<const V *>(part) + i;
        V acc = src[0];
        for (int g = 1; g < groups; ++g) acc += src[(int64_t)g * gstride];
        reinterpret_cast<V *>(out)[i] = acc;
    }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float *__restrict__ out, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) out[i] = 0.f;
}

// ------------------------------------------------------------------ host launchers
static bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

template <typename T>
static hipError_t bias_relu_fwd_t(void *y, int64_t P, int C, int64_t ys, const float *bias, hipStream_t st) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const bool vec = C % EPC == 0 && ys % EPC == 0 && aligned16(y);
    const int CV = vec ? C / EPC : C;
    const int g = grid_for(P * CV, 256, 8192);
    FastDiv d((uint32_t)CV);
    if (vec)
        hipLaunchKernelGGL((bias_relu_fwd_kernel<T, true>), dim3(g), dim3(256), 0, st, (T *)y, P, C, ys, bias, d);
    else
        hipLaunchKernelGGL((bias_relu_fwd_kernel<T, false>), dim3(g), dim3(256), 0, st, (T *)y, P, C, ys, bias, d);
    return hipGetLastError();
}

hipError_t launch_bias_relu_fwd(int dt, void *y, int64_t P, int C, int64_t ys, const float *bias, hipStream_t st) {
    return dt == 0 ? bias_relu_fwd_t<float>(y, P, C, ys, bias, st)
                   : bias_relu_fwd_t<bf16_t>(y, P, C, ys, bias, st);
}

// Partial-sum grid of the bias-gradient reduction (shared with the workspace query).
void relu_bwd_plan(int dt, int64_t P, int C, int64_t ys, int *G, int64_t *ppb) {
    const int EPC = dt == 0 ? 4 : 8;
    const bool vec = C % EPC == 0 && ys % EPC == 0;
    const int CV = vec ? C / EPC : C;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    // about 4 pixel rows per thread: the rows of one thread are a chain of dependent loads
    // (with the fused max-pool gather, argmax then dy), so parallelism comes from the grid
    int64_t g = (P + (int64_t)R * 4 - 1) / ((int64_t)R * 4);
    const int64_t cap = std::max<int64_t>(1, std::min<int64_t>(4096, (1 << 22) / std::max(C, 1)));
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    *G = (int)g;
    *ppb = (P + g - 1) / g;
}

// Partial-sum grid of the standalone ReLU backward (shared with its workspace query): its pixel
// loop batches the loads of four pixels, so a thread takes about 16 channel chunks, and never
// fewer than 4 pixel rows (each block scatters C channel-major partials, which for wide tensors
// cost more than a longer loop).
void relu_bwd_only_plan(int dt, int64_t P, int C, int64_t ys, int *G, int64_t *ppb) {
    const int EPC = dt == 0 ? 4 : 8;
    const bool vec = C % EPC == 0 && ys % EPC == 0;
    const int CV = vec ? C / EPC : C;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    const int64_t rows = (P + R - 1) / R;
    int64_t g = std::min((rows + 3) / 4, (P * CV + 256 * 16 - 1) / (256 * 16));
    const int64_t cap = std::max<int64_t>(1, std::min<int64_t>(4096, (1 << 22) / std::max(C, 1)));
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    *G = (int)g;
    *ppb = (P + g - 1) / g;
}

// The per-channel sum of G partial rows at ws into db, or, with defer, their place left for a
// later batched sum.
static hipError_t finish_partials(const float *ws, int G, int C, float *db, hipStream_t st, BiasPartials *defer) {
    if (defer != nullptr) {
        defer->part = ws;
        defer->rows = G;
        return hipGetLastError();
    }
    hipLaunchKernelGGL(sum_partials_kernel, dim3(C), dim3(256), 0, st, ws, G, C, db);
    return hipGetLastError();
}

template <typename T>
static hipError_t relu_bwd_t(const void *y, const void *dy, void *dpre, int64_t P, int C, int64_t ys,
                             float *db, float *ws, hipStream_t st, BiasPartials *defer) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const bool vec = C % EPC == 0 && ys % EPC == 0 && aligned16(y) && aligned16(dy) && aligned16(dpre);
    int G;
    int64_t ppb;
    relu_bwd_only_plan(sizeof(T) == 4 ? 0 : 1, P, C, ys, &G, &ppb);
    const int CV = vec ? C / EPC : C;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    const size_t smem = R == 1 ? 0 : (size_t)R * C * sizeof(float);
    if (vec)
        hipLaunchKernelGGL((relu_bwd_partial_kernel<T, true>), dim3(G), dim3(256), smem, st,
                           (const T *)y, (const T *)dy, (T *)dpre, P, C, ys, ppb, ws);
    else
        hipLaunchKernelGGL((relu_bwd_partial_kernel<T, false>), dim3(G), dim3(256), smem, st,
                           (const T *)y, (const T *)dy, (T *)dpre, P, C, ys, ppb, ws);
    return finish_partials(ws, G, C, db, st, defer);
}

hipError_t launch_bias_relu_bwd(int dt, const void *y, const void *dy, void *dpre, int64_t P, int C,
                                int64_t ys, float *db, float *ws, hipStream_t st, BiasPartials *defer) {
    return dt == 0 ? relu_bwd_t<float>(y, dy, dpre, P, C, ys, db, ws, st, defer)
                   : relu_bwd_t<bf16_t>(y, dy, dpre, P, C, ys, db, ws, st, defer);
}

// 32-bit index arithmetic for a pool: pixel counts below 2^24 (24-bit multiplies), strides and
// channel counts below 2^24, and every element offset below 2^29 (byte offsets below 2^31 for fp32).
static bool pool_o32(const PoolGeom &g, int64_t pys) {
    constexpr int64_t k24 = 1 << 24, k29 = 1ll << 29;
    const int64_t P = (int64_t)g.N * g.H * g.W, Q = (int64_t)g.N * g.OH * g.OW;
    return P < k24 && Q < k24 && g.C < k24 && g.xs < k24 && g.ys < k24 && pys < k24 && P * g.xs < k29 &&
           Q * g.ys < k29 && Q * g.C < k29 && Q * pys < k29 && P * g.C < k29;
}

template <typename T, typename A>
static hipError_t maxpool_relu_bwd_t(const void *dy, const A *am, const PoolGeom &g, const void *y,
                                     const void *py, int64_t pys, void *dpre, float beta, float *db, float *ws,
                                     hipStream_t st, BiasPartials *defer) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const bool vec = g.C % EPC == 0 && g.xs % EPC == 0 && g.ys % EPC == 0 && aligned16(dy) && aligned16(am) &&
                     (py ? pys % EPC == 0 && aligned16(py) : aligned16(y)) && aligned16(dpre);
    const int64_t P = (int64_t)g.N * g.H * g.W;
    int G;
    int64_t ppb;
    relu_bwd_plan(sizeof(T) == 4 ? 0 : 1, P, g.C, g.xs, &G, &ppb);
    const int CV = vec ? g.C / EPC : g.C;
    const int CVB = CV < 256 ? CV : 256;
    const int R = 256 / CVB;
    const size_t smem = (size_t)R * g.C * sizeof(float);
    const FastDiv dW((uint32_t)g.W), dH((uint32_t)g.H);
    if (vec && g.sh == 2 && g.sw == 2 && g.KH <= 4 && g.KW <= 4) {
        // cell form: ceil((H + pt) / 2) x ceil((W + pl) / 2) cells cover every input pixel; its
        // partial grid (fewer work items than pixels) fits the pixel-sized workspace
        // (about 2 cells per thread; never more partial blocks than the pixel plan's G above)
        const int CH = (g.H + g.pt + 1) / 2, CW = (g.W + g.pl + 1) / 2;
        const int64_t ncell = (int64_t)g.N * CH * CW;
        const int64_t gc = std::max<int64_t>(1, std::min<int64_t>(G, (ncell + 2 * R - 1) / (2 * R)));
        const int Gc = (int)gc;
        const int64_t cpb = (ncell + gc - 1) / gc;
        const FastDiv dCW((uint32_t)CW), dCH((uint32_t)CH);
        const bool o32 = pool_o32(g, py ? pys : 0);
        auto go = [&](auto PK_, auto O_) {
            constexpr int PK = decltype(PK_)::value;
            constexpr bool O = decltype(O_)::value;
            hipLaunchKernelGGL((maxpool_relu_bwd_cell_kernel<T, A, PK, O>), dim3(Gc), dim3(256), smem, st,
                               (const T *)dy, am, g, (const T *)y, (const T *)py, pys, (T *)dpre, beta, cpb, CH, CW,
                               dCW, dCH, ws);
        };
        using I3 = std::integral_constant<int, 3>;
        using I2 = std::integral_constant<int, 2>;
        using I0 = std::integral_constant<int, 0>;
        using BT = std::true_type;
        using BF = std::false_type;
        if (g.KH == 3 && g.KW == 3) o32 ? go(I3{}, BT{}) : go(I3{}, BF{});
        else if (g.KH == 2 && g.KW == 2) o32 ? go(I2{}, BT{}) : go(I2{}, BF{});
        else o32 ? go(I0{}, BT{}) : go(I0{}, BF{});
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        return finish_partials(ws, Gc, g.C, db, st, defer);
    }
    if (vec && pool_o32(g, py ? pys : 0))
        hipLaunchKernelGGL((maxpool_relu_bwd_partial_kernel<T, true, A, true>), dim3(G), dim3(256), smem, st,
                           (const T *)dy, am, g, (const T *)y, (const T *)py, pys, (T *)dpre, beta, ppb, dW, dH, ws);
    else if (vec)
        hipLaunchKernelGGL((maxpool_relu_bwd_partial_kernel<T, true, A, false>), dim3(G), dim3(256), smem, st,
                           (const T *)dy, am, g, (const T *)y, (const T *)py, pys, (T *)dpre, beta, ppb, dW, dH, ws);
    else
        hipLaunchKernelGGL((maxpool_relu_bwd_partial_kernel<T, false, A, false>), dim3(G), dim3(256), smem, st,
                           (const T *)dy, am, g, (const T *)y, (const T *)py, pys, (T *)dpre, beta, ppb, dW, dH, ws);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return finish_partials(ws, G, g.C, db, st, defer);
}

hipError_t launch_maxpool_relu_bwd(int dt, const void *dy, const void *am, bool taps, const PoolGeom &g,
                                   const void *y, const void *py, int64_t pys, void *dpre, float beta, float *db,
                                   float *ws, hipStream_t st, BiasPartials *defer) {
    if (taps)
        return dt == 0 ? maxpool_relu_bwd_t<float>(dy, (const uint8_t *)am, g, y, py, pys, dpre, beta, db, ws, st,
                                                   defer)
                       : maxpool_relu_bwd_t<bf16_t>(dy, (const uint8_t *)am, g, y, py, pys, dpre, beta, db, ws, st,
                                                    defer);
    return dt == 0 ? maxpool_relu_bwd_t<float>(dy, (const int32_t *)am, g, y, py, pys, dpre, beta, db, ws, st, defer)
                   : maxpool_relu_bwd_t<bf16_t>(dy, (const int32_t *)am, g, y, py, pys, dpre, beta, db, ws, st,
                                                defer);
}

template <typename T, typename A>
static hipError_t maxpool_fwd_t(const void *x, const PoolGeom &g, void *y, A *am, hipStream_t st) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const bool vec = g.C % EPC == 0 && g.xs % EPC == 0 && g.ys % EPC == 0 && aligned16(x) &&
                     aligned16(y) && aligned16(am);
    const int64_t cv = vec ? g.C / EPC : g.C;
    const int64_t work = (int64_t)g.N * g.OH * g.OW * cv;
    const int grid = grid_for(work, 256, 16384);
    const Decode dec = make_decode(cv, g.OW, g.OH, work);
    const bool o32 = pool_o32(g, 0);
    if (vec && g.KH == 3 && g.KW == 3 && o32)
        hipLaunchKernelGGL((maxpool_fwd_win_kernel<T, 3, 3, A, true>), dim3(grid), dim3(256), 0, st, (const T *)x, g,
                           (T *)y, am, dec);
    else if (vec && g.KH == 3 && g.KW == 3)
        hipLaunchKernelGGL((maxpool_fwd_win_kernel<T, 3, 3, A, false>), dim3(grid), dim3(256), 0, st, (const T *)x, g,
                           (T *)y, am, dec);
    else if (vec && g.KH == 2 && g.KW == 2 && o32)
        hipLaunchKernelGGL((maxpool_fwd_win_kernel<T, 2, 2, A, true>), dim3(grid), dim3(256), 0, st, (const T *)x, g,
                           (T *)y, am, dec);
    else if (vec && g.KH == 2 && g.KW == 2)
        hipLaunchKernelGGL((maxpool_fwd_win_kernel<T, 2, 2, A, false>), dim3(grid), dim3(256), 0, st, (const T *)x, g,
                           (T *)y, am, dec);
    else if (vec)
        hipLaunchKernelGGL((maxpool_fwd_kernel<T, true, A>), dim3(grid), dim3(256), 0, st, (const T *)x, g, (T *)y, am,
                           dec);
    else
        hipLaunchKernelGGL((maxpool_fwd_kernel<T, false, A>), dim3(grid), dim3(256), 0, st, (const T *)x, g, (T *)y, am,
                           dec);
    return hipGetLastError();
}

hipError_t launch_maxpool_fwd(int dt, const void *x, const PoolGeom &g, void *y, void *am, bool taps, hipStream_t st) {
    if (taps)
        return dt == 0 ? maxpool_fwd_t<float>(x, g, y, (uint8_t *)am, st)
                       : maxpool_fwd_t<bf16_t>(x, g, y, (uint8_t *)am, st);
    return dt == 0 ? maxpool_fwd_t<float>(x, g, y, (int32_t *)am, st) : maxpool_fwd_t<bf16_t>(x, g, y, (int32_t *)am, st);
}

template <typename T, typename A>
static hipError_t maxpool_bwd_t(const void *dy, const A *am, const PoolGeom &g, float beta, void *dx,
                                hipStream_t st) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const bool vec = g.C % EPC == 0 && g.xs % EPC == 0 && g.ys % EPC == 0 && aligned16(dx) &&
                     aligned16(dy) && aligned16(am);
    const int64_t cv = vec ? g.C / EPC : g.C;
    const int64_t work = (int64_t)g.N * g.H * g.W * cv;
    const int grid = grid_for(work, 256, 16384);
    const Decode dec = make_decode(cv, g.W, g.H, work);
    if (vec && pool_o32(g, 0))
        hipLaunchKernelGGL((maxpool_bwd_kernel<T, true, A, true>), dim3(grid), dim3(256), 0, st, (const T *)dy, am, g,
                           beta, (T *)dx, dec);
    else if (vec)
        hipLaunchKernelGGL((maxpool_bwd_kernel<T, true, A, false>), dim3(grid), dim3(256), 0, st, (const T *)dy, am, g,
                           beta, (T *)dx, dec);
    else
        hipLaunchKernelGGL((maxpool_bwd_kernel<T, false, A, false>), dim3(grid), dim3(256), 0, st, (const T *)dy, am, g,
                           beta, (T *)dx, dec);
    return hipGetLastError();
}

hipError_t launch_maxpool_bwd(int dt, const void *dy, const void *am, bool taps, const PoolGeom &g, float beta,
                              void *dx, hipStream_t st) {
    if (taps)
        return dt == 0 ? maxpool_bwd_t<float>(dy, (const uint8_t *)am, g, beta, dx, st)
                       : maxpool_bwd_t<bf16_t>(dy, (const uint8_t *)am, g, beta, dx, st);
    return dt == 0 ? maxpool_bwd_t<float>(dy, (const int32_t *)am, g, beta, dx, st)
                   : maxpool_bwd_t<bf16_t>(dy, (const int32_t *)am, g, beta, dx, st);
}

hipError_t launch_sgd(float *var, const float *grad, int64_t n, float lr, uint16_t *sh, hipStream_t st) {
    const bool vec = aligned16(var) && aligned16(grad) && (sh == nullptr || ((uintptr_t)sh & 7) == 0);
    const int grid = grid_for(vec ? (n + 3) / 4 : n, 256, 1 << 20);
    hipLaunchKernelGGL(sgd_kernel, dim3(grid), dim3(256), 0, st, var, grad, n, lr, sh, vec);
    return hipGetLastError();
}

hipError_t launch_opt(int kind, float *var, float *s1, float *s2, const float *grad, int64_t n, const OptParams &p,
                      uint16_t *sh, hipStream_t st) {
    const bool vec = aligned16(var) && aligned16(s1) && (kind != 2 || aligned16(s2)) && aligned16(grad) &&
                     (sh == nullptr || ((uintptr_t)sh & 7) == 0);
    const int grid = grid_for(vec ? (n + 3) / 4 : n, 256, 1 << 20);
    switch (kind) {
        case 0: hipLaunchKernelGGL(opt_kernel<0>, dim3(grid), dim3(256), 0, st, var, s1, s2, grad, n, p, sh, vec); break;
        case 1: hipLaunchKernelGGL(opt_kernel<1>, dim3(grid), dim3(256), 0, st, var, s1, s2, grad, n, p, sh, vec); break;
        case 2: hipLaunchKernelGGL(opt_kernel<2>, dim3(grid), dim3(256), 0, st, var, s1, s2, grad, n, p, sh, vec); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_sgd_multi(const SgdBatch &b, float lr, hipStream_t st) {
    const int64_t blocks = b.blk_start[b.count];
    if (blocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(sgd_multi_kernel, dim3((unsigned)blocks), dim3(256), 0, st, b, lr);
    return hipGetLastError();
}

// One pass when the gradient has enough elements to occupy the chip: each thread sums its VEC
// elements over all splits in split order, eight loads in flight at a time.
template <int VEC>
__global__ __launch_bounds__(256) void sum_splits_direct_kernel(const float *__restrict__ part, int splits,
                                                                int64_t mn, float *__restrict__ out) {
    typedef typename FVec<VEC>::T V;
    const int64_t mv = mn / VEC;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < mv; i += stride) {
        const V *src = reinterpret_cast<const V *>(part) + i;
        V acc = src[0];
        int s = 1;
        for (; s + 8 <= splits; s += 8) {
            V v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = src[(int64_t)(s + q) * mv];
#pragma unroll
            for (int q = 0; q < 8; ++q) acc += v[q];
        }
        for (; s < splits; ++s) acc += src[(int64_t)s * mv];
        reinterpret_cast<V *>(out)[i] = acc;
    }
}

constexpr int64_t kDirectSumMinThreads = 32768;

// The same sums with G threads per output: thread g of an output adds the splits
// [g S / G, (g + 1) S / G) in order, then the G partial sums are added in g order through
// LDS.  A block covers 256 / G consecutive outputs, so every split row is read as a
// contiguous run; G times the threads of the one-thread form keep more loads in flight.
template <int VEC, int G>
__global__ __launch_bounds__(256) void sum_splits_grouped_kernel(const float *__restrict__ part, int splits,
                                                                 int64_t mn, float *__restrict__ out) {
    typedef typename FVec<VEC>::T V;
    constexpr int COLS = 256 / G;
    __shared__ V red[G][COLS];
    const int64_t mv = mn / VEC;
    const int c = threadIdx.x % COLS, g = threadIdx.x / COLS;
    const int s0 = (int)((int64_t)g * splits / G), s1 = (int)((int64_t)(g + 1) * splits / G);
    for (int64_t base = (int64_t)blockIdx.x * COLS; base < mv; base += (int64_t)gridDim.x * COLS) {
        const int64_t i = base + c;
        V acc = V{};
        if (i < mv && s0 < s1) {
            const V *src = reinterpret_cast<const V *>(part) + i;
            acc = src[(int64_t)s0 * mv];
            int s = s0 + 1;
            for (; s + 8 <= s1; s += 8) {
                V v[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) v[q] = src[(int64_t)(s + q) * mv];
#pragma unroll
                for (int q = 0; q < 8; ++q) acc += v[q];
            }
            for (; s < s1; ++s) acc += src[(int64_t)s * mv];
        }
        red[g][c] = acc;
        __syncthreads();
        if (g == 0 && i < mv) {
            V t = red[0][c];
#pragma unroll
            for (int q = 1; q < G; ++q) t += red[q][c];
            reinterpret_cast<V *>(out)[i] = t;
        }
        __syncthreads();
    }
}

// The two fixed levels of sum_split_groups_kernel + sum_groups_kernel in one pass (the same
// sums in the same order): GP threads per output (GP a power of two >= the number of groups,
// at most 64), thread g adding group g's splits in split order, then the group sums added in
// group order through LDS.  A block covers 256 / GP consecutive outputs.
template <int VEC, int GP>
__global__ __launch_bounds__(256) void sum_split_groups_one_pass_kernel(const float *__restrict__ part, int splits,
                                                                        int64_t mn, float *__restrict__ out) {
    typedef typename FVec<VEC>::T V;
    constexpr int COLS = 256 / GP;
    __shared__ V red[GP][COLS];
    const int64_t mv = mn / VEC;
    const int groups = (splits + kSplitGroup - 1) / kSplitGroup;
    const int c = threadIdx.x % COLS, g = threadIdx.x / COLS;
    const int s0 = g * kSplitGroup, n = min(kSplitGroup, splits - s0);
    for (int64_t base = (int64_t)blockIdx.x * COLS; base < mv; base += (int64_t)gridDim.x * COLS) {
        const int64_t i = base + c;
        V acc = V{};
        if (i < mv && g < groups) {
            const V *src = reinterpret_cast<const V *>(part) + (int64_t)s0 * mv + i;
            V v[kSplitGroup];
#pragma unroll
            for (int q = 0; q < kSplitGroup; ++q)
                if (q < n) v[q] = src[(int64_t)q * mv];
            acc = v[0];
#pragma unroll
            for (int q = 1; q < kSplitGroup; ++q)
                if (q < n) acc += v[q];
        }
        red[g][c] = acc;
        __syncthreads();
        if (g == 0 && i < mv) {
            V t = red[0][c];
            for (int q = 1; q < groups; ++q) t += red[q][c];
            reinterpret_cast<V *>(out)[i] = t;
        }
        __syncthreads();
    }
}

template <int VEC>
static hipError_t sum_splits_t(float *part, int splits, int64_t mn, float *out, hipStream_t st) {
    const int groups = (splits + kSplitGroup - 1) / kSplitGroup;
    const int64_t mv = mn / VEC;
    if (mv >= kDirectSumMinThreads) {
        // about 2^18 threads in flight: 4 or 8 per output when the outputs alone give fewer
        if (splits >= 8 && mv < (1 << 17)) {
            hipLaunchKernelGGL((sum_splits_grouped_kernel<VEC, 8>), dim3(grid_for(mv, 32, 16384)), dim3(256), 0, st,
                               part, splits, mn, out);
        } else if (splits >= 4 && mv < (1 << 18)) {
            hipLaunchKernelGGL((sum_splits_grouped_kernel<VEC, 4>), dim3(grid_for(mv, 64, 16384)), dim3(256), 0, st,
                               part, splits, mn, out);
        } else {
            hipLaunchKernelGGL(sum_splits_direct_kernel<VEC>, dim3(grid_for(mv, 256, 16384)), dim3(256), 0, st, part,
                               splits, mn, out);
        }
        return hipGetLastError();
    }
    if (splits >= 64) {
        // few outputs, many splits (a first layer's per-workgroup partials): 16 threads per output
        hipLaunchKernelGGL((sum_splits_grouped_kernel<VEC, 16>), dim3(grid_for(mv, 16, 16384)), dim3(256), 0, st,
                           part, splits, mn, out);
        return hipGetLastError();
    }
    // one pass for at most 64 groups (1024 splits); the same sums in the same order as the two
    // kernels below
    if (groups <= 64) {
        int gp = 1;
        while (gp < groups) gp *= 2;
        switch (gp) {
#define TFK_ONE_PASS(G_)                                                                                          \
    case G_:                                                                                                      \
        hipLaunchKernelGGL((sum_split_groups_one_pass_kernel<VEC, G_>), dim3(grid_for(mv, 256 / G_, 16384)),      \
                           dim3(256), 0, st, (const float *)part, splits, mn, out);                               \
        return hipGetLastError();
            TFK_ONE_PASS(1) TFK_ONE_PASS(2) TFK_ONE_PASS(4) TFK_ONE_PASS(8) TFK_ONE_PASS(16) TFK_ONE_PASS(32)
            TFK_ONE_PASS(64)
#undef TFK_ONE_PASS
        default: break;
        }
    }
    hipLaunchKernelGGL(sum_split_groups_kernel<VEC>, dim3(grid_for(mv * groups, 256, 16384)), dim3(256), 0, st, part,
                       splits, mn, groups);
    hipLaunchKernelGGL(sum_groups_kernel<VEC>, dim3(grid_for(mv, 256, 16384)), dim3(256), 0, st, part, groups, mn,
                       out);
    return hipGetLastError();
}

// part is the caller's workspace and is overwritten by the first level.
hipError_t launch_sum_splits(float *part, int splits, int64_t mn, float *out, hipStream_t st) {
    if (mn % 4 == 0 && aligned16(part) && aligned16(out)) return sum_splits_t<4>(part, splits, mn, out, st);
    return sum_splits_t<1>(part, splits, mn, out, st);
}

hipError_t launch_sum_partials(const float *partial, int G, int C, float *out, hipStream_t st) {
    hipLaunchKernelGGL(sum_partials_kernel, dim3(C), dim3(256), 0, st, partial, G, C, out);
    return hipGetLastError();
}

hipError_t launch_sum_partials_multi(int count, const float *const *part, const int *rows, const int *channels,
                                     float *const *out, hipStream_t st) {
    for (int i0 = 0; i0 < count; i0 += kPartialsBatch) {
        PartialsBatch b{};
        b.count = std::min(kPartialsBatch, count - i0);
        int total = 0;
        for (int i = 0; i < b.count; ++i) {
            b.chan0[i] = total;
            b.part[i] = part[i0 + i];
            b.rows[i] = rows[i0 + i];
            b.out[i] = out[i0 + i];
            total += channels[i0 + i];
        }
        b.chan0[b.count] = total;
        if (total == 0) continue;
        hipLaunchKernelGGL(sum_partials_multi_kernel, dim3(total), dim3(256), 0, st, b);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_fill_zero(float *out, int64_t n, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const int grid = grid_for(n, 256, 8192);
    hipLaunchKernelGGL(fill_zero_kernel, dim3(grid), dim3(256), 0, st, out, n);
    return hipGetLastError();
}

}  // namespace tfk
