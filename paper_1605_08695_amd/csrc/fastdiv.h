// Division by a run-time invariant divisor with a multiply-high and a shift
// (Granlund & Montgomery, "Division by invariant integers using
// multiplication", PLDI 1994, the round-up variant).  Valid for dividends in
// [0, 2^31) and divisors in [1, 2^31).  Plain C++ so the host tests can check
// it exhaustively without a GPU.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define TFK_HD __host__ __device__ __forceinline__
#else
#define TFK_HD inline
#endif

struct FastDiv {
    uint32_t d;      // divisor
    uint32_t mul;    // magic multiplier
    uint32_t shift;  // post-shift

    TFK_HD FastDiv() : d(1), mul(1), shift(0) {}
    TFK_HD explicit FastDiv(uint32_t divisor) { init(divisor); }

    TFK_HD void init(uint32_t divisor) {
        d = divisor ? divisor : 1;
        uint32_t l = 0;
        while ((1ull << l) < d) ++l;                       // l = ceil(log2 d)
        mul = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
        shift = l;
    }

    TFK_HD uint32_t div(uint32_t n) const {
#if defined(__HIP_DEVICE_COMPILE__)
        uint32_t t = __umulhi(n, mul);
#else
        uint32_t t = (uint32_t)(((uint64_t)n * mul) >> 32);
#endif
        return (t + n) >> shift;
    }

    // q = n / d, r = n - q * d
    TFK_HD void divmod(uint32_t n, uint32_t &q, uint32_t &r) const {
        q = div(n);
        r = n - q * d;
    }
};
