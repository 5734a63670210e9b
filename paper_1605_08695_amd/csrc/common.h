// Device helpers shared by the gfx950 kernels: bf16 conversion, 16-byte
// vector types and the launch-status plumbing.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"

typedef uint16_t bf16_t;   // bfloat16 bits
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

struct alignas(16) U4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16, round to nearest even; NaN stays a (quiet) NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return f32_to_bf16(lo) | (f32_to_bf16(hi) << 16);
}

// Element-type traits: storage type and conversions to/from fp32.
template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int kPerChunk = 4;             // elements per 16-byte chunk
    __device__ static float load(const float *p) { return *p; }
    __device__ static void store(float *p, float v) { *p = v; }
    __device__ static uint32_t bits(const float *p) { return __float_as_uint(*p); }
};
template <> struct Elem<bf16_t> {
    static constexpr int kPerChunk = 8;
    __device__ static float load(const bf16_t *p) { return bf16_to_f32(*p); }
    __device__ static void store(bf16_t *p, float v) { *p = (bf16_t)f32_to_bf16(v); }
    __device__ static uint32_t bits(const bf16_t *p) { return *p; }
};

// Host-side launch helpers (defined in api.cpp).
#define TFK_LAUNCH_CHECK() hipGetLastError()
