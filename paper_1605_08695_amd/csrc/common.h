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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even (NaN stays NaN): gfx950's v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two fp32 values rounded to bf16 and packed (lo in bits 0-15) by one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
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
