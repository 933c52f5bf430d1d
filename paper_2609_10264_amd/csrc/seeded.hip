// Seeded draws of the method's randomness (sample.h): the codes of
// Preprocess on the host, the sparse vectors of Encrypt and Verify on the
// device (so that a seeded Encrypt or Verify stays a stream-ordered call).
#include <vector>

#include "mvk_internal.h"
#include "sample.h"

namespace mvk {

namespace {

// One lane per sparse vector; the lane walks its own draws.
__global__ __launch_bounds__(64) void sample_sparse_kernel(uint64_t seed, uint64_t tag, uint32_t count, uint32_t N,
                                                           uint32_t t, uint32_t* __restrict__ idx,
                                                           uint32_t* __restrict__ val) {
    const uint32_t c = blockIdx.x * 64 + threadIdx.x;
    if (c >= count) return;
    draw::sparse_vector(seed, tag, c, N, t, idx + (size_t)c * t, val + (size_t)c * t);
}

void permutation(draw::Stream& s, uint32_t N, uint32_t* a) {
    for (uint32_t j = 0; j < N; ++j) a[j] = j;
    for (uint32_t i = N; i-- > 1;) {
        const uint32_t j = (uint32_t)s.below((uint64_t)i + 1);
        const uint32_t x = a[i];
        a[i] = a[j];
        a[j] = x;
    }
}

}  // namespace

void sample_code_host(uint32_t k, uint32_t r, uint64_t seed, uint64_t tag, uint32_t* pi1, uint32_t* pi2,
                      uint32_t* v1, uint32_t* v2) {
    const uint32_t N = k * r;
    draw::Stream s = draw::Stream::open(seed, tag, 0);
    permutation(s, N, pi1);
    permutation(s, N, pi2);
    for (uint32_t j = 0; j < N; ++j) v1[j] = s.nonzero();
    for (uint32_t j = 0; j < N; ++j) v2[j] = s.nonzero();
}

void sample_sparse_host(uint32_t count, uint32_t N, uint32_t t, uint64_t seed, uint64_t tag, uint32_t* idx,
                        uint32_t* val) {
    for (uint32_t c = 0; c < count; ++c)
        draw::sparse_vector(seed, tag, c, N, t, idx + (size_t)c * t, val + (size_t)c * t);
}

hipError_t launch_sample_sparse(uint64_t seed, uint64_t tag, uint32_t count, uint32_t N, uint32_t t, uint32_t* idx,
                                uint32_t* val, hipStream_t s) {
    if (count == 0 || t == 0) return hipSuccess;
    hipLaunchKernelGGL(sample_sparse_kernel, dim3(ceil_div(count, 64)), dim3(64), 0, s, seed, tag, count, N, t, idx,
                       val);
    return hipGetLastError();
}

}  // namespace mvk
