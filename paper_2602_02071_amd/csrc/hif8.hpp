// HiF8 codec for the HIP library: bit manipulation on the fp32 pattern,
// usable on the host and on gfx950.
//
// HiF8 (the 8-bit format the BAPS paper uses everywhere it computes in 8
// bits; Sec. 2 "Low Precision Data Formats", App. A) is a tapered float:
// 3 mantissa bits for |x| in [2^-3, 2^4), 2 bits for the exponents +-4..+-7,
// 1 bit for +-8..+-15, and powers of two only (denormals) from 2^-22 to
// 2^-16.  The largest finite value is 2^15.
//
// Rounding is to nearest with ties away from zero (or, on request, to even),
// straight from the fp32 input (one rounding).  For ties-away rounding only
// the first dropped mantissa bit matters, so the rounded value of x depends
// on nothing but the sign, the exponent and the top four mantissa bits of x:
// bits 31..19.  Ties to even also need to know whether bits 18..0 are all
// zero (only then can x sit exactly halfway).
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define HIF8_HD __host__ __device__ __forceinline__
#else
#define HIF8_HD inline
#endif

namespace hif8 {

HIF8_HD uint32_t f2u(float x) { return __builtin_bit_cast(uint32_t, x); }
HIF8_HD float u2f(uint32_t u) { return __builtin_bit_cast(float, u); }

constexpr uint32_t kMaxBits = 0x47000000u;     // 2^15, the largest finite value
constexpr uint32_t kOvfBits = 0x47200000u;     // 1.25 * 2^15, midpoint towards Inf
constexpr uint32_t kMinBits = 0x34800000u;     // 2^-22, the smallest nonzero value

// fp32 bit pattern of the HiF8 value nearest to x (ties away from zero, or
// with even to the neighbour whose significand is even: an even multiple of
// the spacing between the two neighbours, which sends a tie between the last
// value of a binade and the next power of two, and every tie among the
// powers of two below 2^-15, up, and the tie between 0 and 2^-22 down).
// saturate: finite values beyond 2^15 clamp to +-2^15 (else they round to
// +-Inf from the midpoint 1.25 * 2^15 up; at the midpoint itself, ties to
// even keep 2^15).  +-Inf stays +-Inf, NaN stays NaN, and values that round
// to zero give +0.
HIF8_HD uint32_t round_bits(uint32_t x, bool saturate, bool even = false)
{
    const uint32_t s = x & 0x80000000u;
    const uint32_t a = x & 0x7fffffffu;
    if (a >= 0x7f800000u) return x;                        // Inf, NaN
    const int e = (int)(a >> 23) - 127;
    if (e >= 15) {
        if (saturate || a < kOvfBits || (even && a == kOvfBits)) return s | kMaxBits;
        return s | 0x7f800000u;
    }
    if (e < -23) return 0u;
    if (e == -23) return (even && a == 0x34000000u) ? 0u : (s | kMinBits);   // [2^-23, 2^-22) -> 2^-22
    const int ae = e < 0 ? -e : e;
    // mantissa bits kept: 3, 2, 1, or 0 (powers of two below 2^-15)
    const int w = e < -15 ? 0 : (ae <= 3 ? 3 : (ae <= 7 ? 2 : 1));
    const uint32_t half = 1u << (22 - w);
    const uint32_t keep = ~((1u << (23 - w)) - 1u);
    // ties to even: one less than half, plus the last kept bit (w = 0: the
    // significand 2 is the even one, so a tie always goes up)
    const uint32_t odd = w == 0 ? 1u : (a >> (23 - w)) & 1u;
    const uint32_t add = even ? half - 1u + odd : half;
    return s | ((a + add) & keep);                         // a carry lands on 2^(e+1)
}

HIF8_HD float round(float x, bool saturate = true, bool even = false)
{
    return u2f(round_bits(f2u(x), saturate, even));
}

// Code of a value that is already a HiF8 value (output of round_bits).
HIF8_HD uint8_t code_of_rounded(uint32_t r)
{
    const uint32_t s = (r >> 24) & 0x80u;
    const uint32_t a = r & 0x7fffffffu;
    if (a > 0x7f800000u) return 0x80;                      // NaN
    if (a == 0x7f800000u) return (uint8_t)(s | 0x6f);      // Inf
    if (a == 0) return 0x00;
    const int e = (int)(a >> 23) - 127;
    const uint32_t m3 = (a >> 20) & 7u;
    if (e < -15) return (uint8_t)(s | (uint32_t)(e + 23)); // denormal 2^(M-23)
    const uint32_t es = e < 0 ? 1u : 0u;
    const uint32_t mag = (uint32_t)(e < 0 ? -e : e);
    uint32_t c;
    if (mag == 0) c = 0x08u | m3;                                            // dot 0001
    else if (mag == 1) c = 0x10u | (es << 3) | m3;                           // dot 001
    else if (mag <= 3) c = 0x20u | (es << 4) | ((mag & 1u) << 3) | m3;       // dot 01
    else if (mag <= 7) c = 0x40u | (es << 4) | ((mag & 3u) << 2) | (m3 >> 1);// dot 10
    else c = 0x60u | (es << 4) | ((mag & 7u) << 1) | (m3 >> 2);              // dot 11
    return (uint8_t)(s | c);
}

HIF8_HD uint8_t encode(float x, bool saturate = true, bool even = false)
{
    return code_of_rounded(round_bits(f2u(x), saturate, even));
}

// Value of a code.  0x80 is NaN, 0x6F/0xEF are +-Inf, 0x00 is zero.
HIF8_HD float decode(uint8_t code)
{
    const uint32_t s = (uint32_t)(code & 0x80u) << 24;
    const uint32_t b = code & 0x7fu;
    uint32_t es, mag, man, w;
    if (b >= 0x60u) { es = (b >> 4) & 1u; mag = 8u | ((b >> 1) & 7u); man = b & 1u; w = 1; }
    else if (b >= 0x40u) { es = (b >> 4) & 1u; mag = 4u | ((b >> 2) & 3u); man = b & 3u; w = 2; }
    else if (b >= 0x20u) { es = (b >> 4) & 1u; mag = 2u | ((b >> 3) & 1u); man = b & 7u; w = 3; }
    else if (b >= 0x10u) { es = (b >> 3) & 1u; mag = 1u; man = b & 7u; w = 3; }
    else if (b >= 0x08u) { es = 0u; mag = 0u; man = b & 7u; w = 3; }
    else {
        if (b == 0) return s ? u2f(0x7fc00000u) : 0.0f;
        return u2f(s | ((b + 127u - 23u) << 23));          // 2^(M-23)
    }
    if (es == 0 && mag == 15 && man == 1) return u2f(s | 0x7f800000u);
    const int e = es ? -(int)mag : (int)mag;
    return u2f(s | ((uint32_t)(e + 127) << 23) | (man << (23 - w)));
}

}  // namespace hif8
