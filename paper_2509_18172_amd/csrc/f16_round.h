// Exact binary64 -> binary16 rounding on the device, shared by the
// decompression, prefill and encoding kernels, and the test for when binary32
// subset sums are exact.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sbvr {

// binary64 -> binary16, round to nearest, ties to even (IEEE 754), from the
// bit fields; overflow gives infinity.  (Rounding through binary32 with the
// hardware conversions would round twice.)
__device__ __forceinline__ uint16_t f64_to_f16_rne(double x)
{
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    const uint32_t sign = (uint32_t)(u >> 48) & 0x8000u;
    const int e = (int)((u >> 52) & 0x7ff);
    if (e == 0)  // zero or a binary64 subnormal: far below binary16's range
        return (uint16_t)sign;
    const uint64_t sig = (1ull << 52) | (u & ((1ull << 52) - 1));
    int E = e - 1023;
    int shift;  // bits of sig dropped
    if (E >= -14) {
        shift = 42;  // keep 11 significant bits
    } else {
        shift = 28 - E;  // subnormal: units of 2^-24
        if (shift > 54)
            return (uint16_t)sign;  // below half the smallest subnormal
    }
    uint64_t q = sig >> shift;
    const uint64_t rem = sig & ((1ull << shift) - 1);
    const uint64_t half = 1ull << (shift - 1);
    if (rem > half || (rem == half && (q & 1)))
        ++q;
    if (E >= -14) {
        if (q == (1ull << 11)) {  // rounded up to the next binade
            q >>= 1;
            ++E;
        }
        if (E > 15)
            return (uint16_t)(sign | 0x7c00u);
        return (uint16_t)(sign | (uint32_t)(E + 15) << 10 | (uint32_t)(q & 0x3ff));
    }
    return (uint16_t)(sign | (uint32_t)q);  // q == 0x400 is the smallest normal
}

// Unbiased exponent of a binary16 bit pattern (subnormals as -14).
__device__ __forceinline__ int f16_exp(uint32_t h)
{
    const int e = (int)((h >> 10) & 0x1f);
    return e == 0 ? -14 : e - 15;
}

// True when the subset sums of these k binary16 values are exact in binary32:
// every value is a multiple of 2^(emin - 10) below 2^(emax + 1), so a sum of
// at most four needs at most emax - emin + 13 significant bits, <= 24 when the
// nonzero values' exponents span at most 11 (then one hardware rounding of
// the binary32 sum to binary16 is the correctly rounded result).
template <int K>
__device__ __forceinline__ bool f16_sums_exact_in_f32(const uint32_t *c)
{
    int emax = -30, emin = 30;
#pragma unroll
    for (int i = 0; i < K; ++i) {
        if (c[i] & 0x7fffu) {
            emax = max(emax, f16_exp(c[i]));
            emin = min(emin, f16_exp(c[i]));
        }
    }
    return emax - emin <= 11;
}

}  // namespace sbvr
