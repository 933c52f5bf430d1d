// Streaming read of a device buffer: the HBM read floor that server_eval's
// W stream is compared against (same bytes, nothing computed but an XOR
// checksum).  Every thread issues all of a pass's 16-byte loads before
// combining them; the loads are non-temporal, as server_eval's W loads.  Each
// workgroup writes the XOR of everything it read to its own sink word, and
// workgroup 0 clears the words of workgroups the launch does not have.  Shape
// by size (measured on MI355X, back-to-back launches): up to 64 MiB one pass
// of 4 loads per thread over as many workgroups as that takes (16.8 MB:
// 4.6 us); above, 256 workgroups looping with 8 loads per thread (268 MB:
// 39.7 us, 6.8 TB/s; 4.9 and 42.6 us with ordinary loads).
#include "mvk_internal.h"

namespace mvk {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kReadThreads = 256;

template <int kReadPer>
__global__ __launch_bounds__(kReadThreads) void stream_read_kernel(const uint4* __restrict__ p, size_t n16,
                                                                   uint32_t* __restrict__ sink,
                                                                   uint32_t sink_words) {
    __shared__ uint32_t red[kReadThreads / 64];
    const size_t stride = (size_t)gridDim.x * kReadThreads;
    const size_t g = (size_t)blockIdx.x * kReadThreads + threadIdx.x;
    uint32_t x = 0;
    for (size_t base = 0; base < n16; base += stride * kReadPer) {
        u32x4 v[kReadPer];
#pragma unroll
        for (int u = 0; u < kReadPer; ++u) {
            const size_t i = base + g + stride * u;
            // non-temporal, as server_eval reads W
            v[u] = i < n16 ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p) + i) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kReadPer; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) x ^= (uint32_t)__shfl_xor((int)x, s);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
#pragma unroll
        for (int w = 0; w < kReadThreads / 64; ++w) t ^= red[w];
        sink[blockIdx.x] = t;
    }
    if (blockIdx.x == 0)
        for (uint32_t w = gridDim.x + threadIdx.x; w < sink_words; w += kReadThreads) sink[w] = 0u;
}

}  // namespace

hipError_t launch_stream_read(const void* data, size_t bytes, uint32_t* sink, uint32_t sink_words, hipStream_t s) {
    const size_t n16 = bytes / 16;
    const uint4* p = reinterpret_cast<const uint4*>(data);
    const size_t one_pass = (n16 + 4 * kReadThreads - 1) / (4 * kReadThreads);
    if (one_pass <= sink_words)
        hipLaunchKernelGGL(stream_read_kernel<4>, dim3((uint32_t)(one_pass ? one_pass : 1)), dim3(kReadThreads), 0, s,
                           p, n16, sink, sink_words);
    else
        hipLaunchKernelGGL(stream_read_kernel<8>, dim3(256), dim3(kReadThreads), 0, s, p, n16, sink, sink_words);
    return hipGetLastError();
}

}  // namespace mvk
