// Completion count of a launch: which workgroup finishes last?
//
// Device atomics on one address from many workgroups are serialised by the
// memory system (about 12 ns each on MI355X: one counter costs ~17 us at 1440
// workgroups), so a launch with a large grid counts in two levels: every
// workgroup on one of `slots` level-1 counters (kCountStride words apart, so
// no two share a 256-byte line), and the last workgroup of each slot on the
// top counter.  Small grids (slots == 0) count on the top counter alone.
//
// Layout in the control region: the top counter at ctrl[0], level-1 counter s
// at ctrl[kCountStride * (1 + s)].  All counters are zero before the launch
// and zero again once the last workgroup has been found.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mvk {

constexpr uint32_t kCountStride = 64;  // words between level-1 counters (256 bytes)
constexpr uint32_t kCountMaxSlots = 256;

// Level-1 counters for a grid: none up to 64 workgroups, else about
// sqrt(grid) (as many workgroups per slot as slots), between 8 and 256.
__host__ __device__ inline uint32_t count_slots(uint32_t grid) {
    if (grid <= 64) return 0;
    uint32_t s = 8;
    while (s < kCountMaxSlots && s * s < grid) ++s;
    return s;
}

// Words of the control region used by the counters (the top counter's line
// and the level-1 lines).
__host__ __device__ inline uint32_t count_words(uint32_t slots) { return kCountStride * (1 + slots); }

// Thread 0 of every workgroup calls this once, after the workgroup's memory
// operations have completed (s_waitcnt 0) and a workgroup barrier.  Returns
// true in exactly one workgroup, the last to arrive; the counters it used are
// reset before it returns.  Each decision waits for the atomic it depends on,
// so everything that completed before any workgroup's count is visible to
// device-coherent reads of the last one.
__device__ inline bool count_last(uint32_t* ctrl, uint32_t slots) {
    const uint32_t grid = gridDim.x;
    if (slots == 0) {
        if (atomicAdd(ctrl, 1u) != grid - 1) return false;
        atomicExch(ctrl, 0u);
        return true;
    }
    const uint32_t slot = blockIdx.x % slots;
    const uint32_t in_slot = (grid - slot + slots - 1) / slots;  // workgroups counting on this slot
    uint32_t* sc = ctrl + kCountStride * (1 + slot);
    if (atomicAdd(sc, 1u) != in_slot - 1) return false;
    atomicExch(sc, 0u);
    const uint32_t used = grid < slots ? grid : slots;
    if (atomicAdd(ctrl, 1u) != used - 1) return false;
    atomicExch(ctrl, 0u);
    return true;
}

}  // namespace mvk
