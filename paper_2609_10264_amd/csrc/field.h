// Device arithmetic in F_p, p = 2^31 - 1 (Mersenne), for gfx950.
//
// Reductions use 2^31 = 1 (mod p): x = hi*2^31 + lo  ->  x = hi + lo (mod p).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mvk {

constexpr uint32_t kP = 2147483647u;

// a, b in [0, p)
__device__ __forceinline__ uint32_t fadd(uint32_t a, uint32_t b) {
    uint32_t s = a + b;  // < 2^32
    return s >= kP ? s - kP : s;
}

__device__ __forceinline__ uint32_t fsub(uint32_t a, uint32_t b) {
    return a >= b ? a - b : a + (kP - b);
}

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

// Signed 64-bit value (|x| < 2^62) -> [0, p).
__device__ __forceinline__ uint32_t fred_s64(int64_t x) {
    // x + p*2^32 lies in (0, 2^64) for |x| < 2^62 and is x mod p.
    return fred64((uint64_t)x + ((uint64_t)kP << 32));
}

// int8 weight -> field element.
__device__ __forceinline__ uint32_t femb(int8_t w) { return w < 0 ? kP + (int32_t)w : (uint32_t)w; }

}  // namespace mvk
