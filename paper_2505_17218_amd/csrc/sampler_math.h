// Bit-reproducible float32 arithmetic of the Gumbel-max sampler and the GRPO
// advantage.  Every operation is rounded on its own (the translation units that
// include this are built with -ffp-contract=off, and divisions / square roots
// use the correctly rounded intrinsics on the device), so the GPU result depends
// only on the inputs, never on instruction scheduling.  Usable from host code
// too, which lets CPU tests check these exact functions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <math.h>

namespace dash {

__host__ __device__ inline float div_rn(float a, float b) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __fdiv_rn(a, b);
#else
    return a / b;
#endif
}

// Correctly rounded float32 square root.  On gfx950 neither sqrtf nor
// __fsqrt_rn is correctly rounded (measured: about 15% of random inputs differ
// by one ulp), so the device takes the float64 square root and rounds it to
// float32, which is correctly rounded because 53 >= 2 * 24 + 2.
__host__ __device__ inline float sqrt_rn(float a) {
#if defined(__HIP_DEVICE_COMPILE__)
    return (float)sqrt((double)a);
#else
    return sqrtf(a);
#endif
}

__host__ __device__ inline uint32_t f_bits(float f) {
    union { float f; uint32_t u; } c;
    c.f = f;
    return c.u;
}
__host__ __device__ inline float bits_f(uint32_t u) {
    union { float f; uint32_t u; } c;
    c.u = u;
    return c.f;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): per round, two 32x32->64
// products of counter words 0 and 2 with the multipliers, recombined with the
// other two words and the round key; the key advances by the Weyl increments
// before every round but the first.
struct U4 {
    uint32_t x, y, z, w;
};

__host__ __device__ inline U4 philox4x32_10(U4 c, uint32_t k0, uint32_t k1) {
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t p0 = (uint64_t)M0 * c.x;
        const uint64_t p1 = (uint64_t)M1 * c.z;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c = U4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
    }
    return c;
}

// Natural log of a positive normal float: x = 2^e m, m folded into
// [sqrt(1/2), sqrt(2)]; f = m - 1 (exact); s = f / (2 + f);
// ln m = 2 atanh(s) = s (C0 + z (C1 + z (C2 + z (C3 + z (C4 + z C5))))) with
// z = s^2 and the Taylor coefficients C_k = 2 / (2k + 1);
// ln x = e ln2_hi + (e ln2_lo + ln m), where ln2_hi keeps the top 16 bits of
// ln 2 so that e ln2_hi is exact.
__host__ __device__ inline float own_log(float x) {
    const float kC0 = (float)(2.0 / 1.0), kC1 = (float)(2.0 / 3.0), kC2 = (float)(2.0 / 5.0);
    const float kC3 = (float)(2.0 / 7.0), kC4 = (float)(2.0 / 9.0), kC5 = (float)(2.0 / 11.0);
    const float kSqrt2 = (float)1.4142135623730951;
    const uint32_t ln2_bits = f_bits((float)0.6931471805599453) & 0xFFFFFF00u;
    const float kLn2Hi = bits_f(ln2_bits);
    const float kLn2Lo = (float)(0.6931471805599453 - (double)kLn2Hi);

    const uint32_t b = f_bits(x);
    int e = (int)((b >> 23) & 0xFFu) - 127;
    float m = bits_f((b & 0x7FFFFFu) | 0x3F800000u);
    if (m > kSqrt2) {
        m = m * 0.5f;
        e += 1;
    }
    const float f = m - 1.0f;
    const float t = 2.0f + f;
    const float s = div_rn(f, t);
    const float z = s * s;
    float p = kC5;
    p = p * z;
    p = p + kC4;
    p = p * z;
    p = p + kC3;
    p = p * z;
    p = p + kC2;
    p = p * z;
    p = p + kC1;
    p = p * z;
    p = p + kC0;
    const float lm = s * p;
    const float ef = (float)e;
    float lo = ef * kLn2Lo;
    lo = lo + lm;
    const float hi = ef * kLn2Hi;
    return hi + lo;
}

// Standard Gumbel noise from 32 random bits: u = ((x >> 8) | 1) 2^-24 in (0, 1), g = -ln(-ln u).
__host__ __device__ inline float gumbel_from_bits(uint32_t x) {
    const float u = (float)((x >> 8) | 1u) * (1.0f / 16777216.0f);
    return -own_log(-own_log(u));
}

}  // namespace dash
