// The element-wise step of the masked encode (Encrypt with a prepared mask),
// shared by its own kernel and the fused client-turn kernel; and the bounded
// flag poll its wait uses.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "field.h"

namespace mvk {

// Polls *flag (device-coherent loads, a short sleep between polls) from the
// calling thread until it holds `value`; false after `ticks` of the constant
// wall clock.
__device__ inline bool poll_flag(const uint32_t* flag, uint32_t value, uint64_t ticks) {
    const uint64_t t0 = wall_clock64();
    while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != value) {
        if (wall_clock64() - t0 > ticks) return false;
        __builtin_amdgcn_s_sleep(4);
    }
    return true;
}

// Xhat = X + Mx, element-wise over count words, PER words per thread and
// pass with the pass's loads issued first.  WAIT: the loads of X (the query,
// not covered by the flag) are issued before thread 0 of each workgroup
// polls *flag for `value`; Mx is read device-coherently after it.  The flag
// is cleared by the only workgroup, or, with several, by the last one to
// finish (counted on `counter`, which it also clears).  The caller's
// workgroup is number `bid` of the `nblocks` that share the elements.
constexpr int kAddThreads = 1024;

// Words per thread and pass of a masked encode of `count` words: the fewest
// (1, 2 or 4) that still cover the words in one pass of at most 256
// workgroups.  One word per thread spreads a stage's encode over more
// compute units, whose loads are then in flight together (measured on the
// 32-layer stack, whose encodes cover 32768 and 88064 words: 3.48 ms per
// pass against 3.53-3.62 with four words per thread); past 256 workgroups a
// second dependent pass would cost more than the wider threads.
inline int add_masks_per(size_t count) {
    const size_t one = (size_t)256 * kAddThreads;
    return count <= one ? 1 : count <= 2 * one ? 2 : 4;
}
template <bool WAIT, int PER>
__device__ __forceinline__ void add_masks_body(uint32_t bid, uint32_t nblocks, const uint32_t* X,
                                               const uint32_t* __restrict__ Mx, size_t count, uint32_t* Xhat,
                                               uint32_t* flag, uint32_t value, uint64_t ticks, uint32_t* timed_out,
                                               uint32_t* counter) {
    const size_t stride = (size_t)nblocks * kAddThreads, pass = stride * PER;
    const size_t g = (size_t)bid * kAddThreads + threadIdx.x;
    bool polled = !WAIT;
    for (size_t base = 0; base < count; base += pass) {
        uint32_t xv[PER], mv[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const size_t i = base + g + stride * u;
            xv[u] = X[i < count ? i : count - 1];
        }
        if (WAIT && !polled) {  // first pass only (uniform)
            if (threadIdx.x == 0) {
                if (!poll_flag(flag, value, ticks)) {
                    if (timed_out) atomicOr(timed_out, 1u);
                } else if (nblocks == 1) {
                    __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            __syncthreads();
            polled = true;
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const size_t i = base + g + stride * u, is = i < count ? i : count - 1;
            mv[u] = WAIT ? __hip_atomic_load(&Mx[is], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : Mx[is];
        }
        uint32_t out[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            out[u] = fadd(xv[u], mv[u]);
            // pinned in a register before the guarded store, so that the
            // compiler does not sink the loads into the branch
            asm volatile("" : "+v"(out[u]));
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const size_t i = base + g + stride * u;
            if (i < count) Xhat[i] = out[u];
        }
    }
    if constexpr (WAIT) {
        if (!polled) {  // no pass at all (count == 0): still consume the flag
            if (threadIdx.x == 0 && !poll_flag(flag, value, ticks) && timed_out) atomicOr(timed_out, 1u);
            if (threadIdx.x == 0 && nblocks == 1)
                __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (nblocks > 1 && threadIdx.x == 0 && atomicAdd(counter, 1u) == nblocks - 1) {
            atomicExch(counter, 0u);
            __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Wall-clock ticks of timeout_us on the current device.
inline hipError_t wait_ticks(uint32_t timeout_us, uint64_t* ticks) {
    int dev = 0, khz = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return e;
    if (khz <= 0) return hipErrorInvalidValue;
    *ticks = (uint64_t)timeout_us * (uint64_t)khz / 1000u;
    return hipSuccess;
}

}  // namespace mvk
