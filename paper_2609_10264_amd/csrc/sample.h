// Seeded sampling of the method's random draws, for the host and the device.
//
// Protocol pvMVMD draws the two RAA codes in Preprocess (App. B: uniform
// permutations pi1, pi2 and diagonals v1, v2 over F_p^*), the noise
// e_x <- E_{tx}^{Nx} in Encrypt and the challenges e <- E_{ty}^{Ny} in Verify
// (Sec. 3: E_t^N has exactly t nonzero entries; Lemma 5.1 draws the support
// uniformly and the values uniformly in F_p^*).  The paper leaves the
// generator open; the library follows this written specification, so that a
// seed reproduces every draw:
//
//   generator  SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): the state
//              advances by the golden-ratio increment 0x9E3779B97F4A7C15 and
//              each output is the state passed through the finaliser
//              z ^= z>>30; z *= 0xBF58476D1CE4E5B9; z ^= z>>27;
//              z *= 0x94D049BB133111EB; z ^= z>>31
//   streams    stream c of (seed, tag) starts from finaliser(seed ^ tag ^ finaliser(c))
//   integers   below b: outputs z >= 2^64 - (2^64 mod b) are rejected (none when
//              b divides 2^64), the value is z mod b; after 64 rejected outputs
//              the last one's z mod b is taken
//   F_p^*      the top 31 bits of an output, rejected unless in [1, p-1];
//              after 64 rejections the value 1
//   code       stream 0: pi1 then pi2 by Fisher-Yates (start from the
//              identity; for i = N-1 down to 1 swap entry i with entry
//              below(i+1)), then the N entries of v1, then those of v2
//   E_t^N      vector c uses stream c: positions below(N), a repeat is skipped,
//              until t are held (in draw order) or 2^24 positions were drawn,
//              after which the smallest free positions complete the support in
//              increasing order; then its t values in F_p^*
//
// The caps only bound every loop; with t <= N none is reached with any
// meaningful probability at the sizes the library accepts.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "field.h"

namespace mvk {
namespace draw {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr int kRejectCap = 64;
constexpr uint64_t kPositionCap = 1ull << 24;

__host__ __device__ inline uint64_t finalise(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

struct Stream {
    uint64_t state;

    __host__ __device__ static Stream open(uint64_t seed, uint64_t tag, uint64_t c) {
        return Stream{finalise(seed ^ tag ^ finalise(c))};
    }
    __host__ __device__ uint64_t next() {
        state += kGamma;
        return finalise(state);
    }
    // Uniform in [0, b), b >= 1.
    __host__ __device__ uint64_t below(uint64_t b) {
        const uint64_t cut = (0ull - b) % b;  // 2^64 mod b: outputs >= 2^64 - cut are rejected
        uint64_t z = 0;
        for (int tries = 0; tries < kRejectCap; ++tries) {
            z = next();
            if (cut == 0 || z <= ~cut) return z % b;  // ~cut = 2^64 - 1 - cut
        }
        return z % b;
    }
    // Uniform in [1, p - 1].
    __host__ __device__ uint32_t nonzero() {
        for (int tries = 0; tries < kRejectCap; ++tries) {
            const uint32_t v = (uint32_t)(next() >> 33);
            if (v != 0u && v < kP) return v;
        }
        return 1u;
    }
};

// One draw from E_t^N (t <= N) into idx[0, t), val[0, t) using stream c.
// The repeat check reads back the positions already written (t is small).
__host__ __device__ inline void sparse_vector(uint64_t seed, uint64_t tag, uint64_t c, uint32_t N, uint32_t t,
                                              uint32_t* idx, uint32_t* val) {
    Stream s = Stream::open(seed, tag, c);
    uint32_t held = 0;
    auto taken = [&](uint32_t j) {
        for (uint32_t q = 0; q < held; ++q)
            if (idx[q] == j) return true;
        return false;
    };
    for (uint64_t drawn = 0; held < t && drawn < kPositionCap; ++drawn) {
        const uint32_t j = (uint32_t)s.below(N);
        if (!taken(j)) idx[held++] = j;
    }
    for (uint32_t j = 0; held < t && j < N; ++j)
        if (!taken(j)) idx[held++] = j;
    for (uint32_t q = 0; q < t; ++q) val[q] = s.nonzero();
}

}  // namespace draw
}  // namespace mvk
