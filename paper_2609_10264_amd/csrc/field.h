// Device arithmetic in the prime field of the build, for gfx950.
//
// Two fields, one per build of the library:
//  * default:              p = 2^31 - 1 (Mersenne).  Reductions use
//                          2^31 = 1 (mod p): x = hi*2^31 + lo -> hi + lo.
//  * MVK_FIELD_BABYBEAR:   q = 15*2^27 + 1, the field of the paper's Sec. 7.1
//                          evaluation.  Reductions are Barrett's with
//                          mu = floor(2^64 / q): for x < 2^64 the quotient
//                          estimate hi64(x*mu) is floor(x/q) or one less, so
//                          x - q*hi64(x*mu) lies in [0, 2q).
// Both moduli are below 2^31, so canonical values are uint32, sums of two fit
// in 32 bits and products of two in 62 bits.  Every kernel is written against
// the functions below and kP only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mvk {

#ifdef MVK_FIELD_BABYBEAR
constexpr uint32_t kP = 2013265921u;            // 15 * 2^27 + 1
constexpr uint64_t kBarrettMu = 9162596893ull;  // floor(2^64 / kP)
#else
constexpr uint32_t kP = 2147483647u;            // 2^31 - 1
#endif

// a, b in [0, p)
__device__ __forceinline__ uint32_t fadd(uint32_t a, uint32_t b) {
    uint32_t s = a + b;  // < 2^32
    return s >= kP ? s - kP : s;
}

__device__ __forceinline__ uint32_t fsub(uint32_t a, uint32_t b) {
    return a >= b ? a - b : a + (kP - b);
}

#ifdef MVK_FIELD_BABYBEAR

// Any x < 2^64 -> [0, q).
__device__ __forceinline__ uint32_t fred64(uint64_t x) {
    const uint64_t r = x - __umul64hi(x, kBarrettMu) * (uint64_t)kP;  // [0, 2q)
    const uint32_t u = (uint32_t)r;
    return u >= kP ? u - kP : u;
}

// Partial reduction of a product of two field elements for values that are
// summed in 64 bits before a final fred64: here the full reduction (< 2^31).
__device__ __forceinline__ uint64_t ffold(uint64_t x) { return fred64(x); }

__device__ __forceinline__ uint32_t fmul(uint32_t a, uint32_t b) { return fred64((uint64_t)a * b); }

#else

// Any x < 2^64 -> [0, p).
__device__ __forceinline__ uint32_t fred64(uint64_t x) {
    uint64_t s = (x & kP) + (x >> 31);               // < 2^31 + 2^33
    uint32_t u = (uint32_t)((s & kP) + (s >> 31));   // < 2^31 + 2^3
    return u >= kP ? u - kP : u;
}

// Fold of a product of two field elements (< 2^62) to [0, 2^32): cheap partial
// reduction for values that are summed in 64 bits before a final fred64.
__device__ __forceinline__ uint64_t ffold(uint64_t x) { return (x & kP) + (x >> 31); }

// a, b in [0, p)
__device__ __forceinline__ uint32_t fmul(uint32_t a, uint32_t b) {
    uint64_t t = (uint64_t)a * b;                    // < 2^62
    uint32_t s = (uint32_t)((t & kP) + (t >> 31));   // < 2^32
    s = (s & kP) + (s >> 31);                        // <= p
    return s >= kP ? s - kP : s;
}

#endif

// Signed 64-bit value (|x| < 2^62) -> [0, p).
__device__ __forceinline__ uint32_t fred_s64(int64_t x) {
    // x + p*2^32 lies in (0, 2^64) for |x| < 2^62 (p*2^32 < 2^63) and is x mod p.
    return fred64((uint64_t)x + ((uint64_t)kP << 32));
}

// int8 weight -> field element.
__device__ __forceinline__ uint32_t femb(int8_t w) { return w < 0 ? kP + (int32_t)w : (uint32_t)w; }

// sum_d 2^(8d) S_d mod p for the four signed digit-plane sums |S_d| < 2^31 of
// the int8-limb product.
#ifdef MVK_FIELD_BABYBEAR
__device__ __forceinline__ uint32_t fdigits4(int32_t s0, int32_t s1, int32_t s2, int32_t s3) {
    // |sum| < 2^31 * (1 + 2^8 + 2^16 + 2^24) < 2^56: exact in 64 bits
    return fred_s64((int64_t)s0 + ((int64_t)s1 << 8) + ((int64_t)s2 << 16) + ((int64_t)s3 << 24));
}
#else
// In 32-bit arithmetic: S_d mod p, then multiplication by 2^(8d), which modulo
// p = 2^31 - 1 is a rotation of the 31-bit value by 8d.
__device__ __forceinline__ uint32_t frotl31(uint32_t x, int k) {
    return ((x << k) | (x >> (31 - k))) & kP;
}

__device__ __forceinline__ uint32_t fdigit_mod(int32_t v) {
    // v >= 0: v <= 2^31 - 1 = p, so v mod p is v or 0; v < 0: p + v >= 0
    const uint32_t u = v >= 0 ? (uint32_t)v : kP + (uint32_t)v;
    return u >= kP ? u - kP : u;
}

__device__ __forceinline__ uint32_t fdigits4(int32_t s0, int32_t s1, int32_t s2, int32_t s3) {
    return fadd(fadd(fdigit_mod(s0), frotl31(fdigit_mod(s1), 8)),
                fadd(frotl31(fdigit_mod(s2), 16), frotl31(fdigit_mod(s3), 24)));
}
#endif

}  // namespace mvk
