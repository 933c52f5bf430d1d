// Input validation (the MVK_VALIDATE mode of the C ABI): the number of words
// of a field array that are not canonical (>= p).
#include "field.h"
#include "mvk_internal.h"

namespace mvk {

namespace {

constexpr int kValThreads = 256;

__global__ __launch_bounds__(kValThreads) void count_noncanonical(const uint32_t* __restrict__ a, size_t count,
                                                                  uint32_t* __restrict__ out) {
    __shared__ uint32_t red[kValThreads / 64];
    uint32_t c = 0;
    for (size_t i = (size_t)blockIdx.x * kValThreads + threadIdx.x; i < count; i += (size_t)gridDim.x * kValThreads)
        c += a[i] >= kP ? 1u : 0u;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) c += (uint32_t)__shfl_xor((int)c, s);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
#pragma unroll
        for (int w = 0; w < kValThreads / 64; ++w) t += red[w];
        if (t) atomicAdd(out, t);
    }
}

}  // namespace

hipError_t launch_count_noncanonical(const uint32_t* a, size_t count, uint32_t* out, hipStream_t s) {
    if (count == 0) return hipSuccess;
    size_t blocks = (count + 4 * kValThreads - 1) / (4 * kValThreads);
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(count_noncanonical, dim3((uint32_t)blocks), dim3(kValThreads), 0, s, a, count, out);
    return hipGetLastError();
}

}  // namespace mvk
