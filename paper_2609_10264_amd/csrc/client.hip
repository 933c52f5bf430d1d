// Client-side Decrypt and Verify of Protocol pvMVMD on gfx950.
//
// Decrypt:  Y_b = Yhat_b - P e_b = Yhat_b - sum_{j in supp(e_b)} e_j PT[j, :]
//           (the sparse noise selects t_x rows of PT; each row is read
//           coalesced along the output index).
// Verify:   for every repetition q with challenge e_q,
//             v_L[q][b] = (e_q^T Q) Xhat_b
//             v_R[q][b] = e_q^T (Gy^T Yhat_b) = (Gy e_q)^T Yhat_b
//           The second form of v_R is the transposition identity of App. B:
//           the syndrome r_q = Gy e_q is computed once per repetition (shared
//           by all columns) instead of one encoding Gy^T Yhat_b per column.
//           Both forms give the same field element.
//
// Dot products are accumulated in 64 bits from folded products (< 2^32 each)
// and reduced once per workgroup; per-workgroup partials (each < p) are summed
// by the finalize kernel.  All sums are exact, so results do not depend on
// the reduction order.
#include "field.h"
#include "mvk_internal.h"

namespace mvk {

namespace {

constexpr int kB = kClientBlock;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int s) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, s);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), s);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v += shfl_xor_u64(v, s);
    return v;
}

// Workgroup shape of the two gather kernels: kCols consecutive output
// columns (one per lane) x kGroups thread groups, each group taking every
// kGroups-th sparse term, so kGroups * (unrolled) row loads are in flight per
// lane.  The sparse (index, value) pairs are staged through LDS in chunks.
constexpr int kCols = kClientCols;
constexpr int kGroups = kB / kCols;
constexpr int kStage = kB;

// grid (ceil(m / kCols), B)
__global__ __launch_bounds__(kB) void decode_vr(const uint32_t* __restrict__ PT, uint32_t m, uint32_t Nx,
                                                const uint32_t* __restrict__ Yhat, uint32_t B,
                                                const uint32_t* __restrict__ ex_idx,
                                                const uint32_t* __restrict__ ex_val, uint32_t tx,
                                                const uint32_t* __restrict__ rv, uint32_t ell,
                                                uint32_t* __restrict__ Y, uint32_t* __restrict__ partR) {
    __shared__ uint32_t s_idx[kStage], s_val[kStage];
    __shared__ uint64_t part[kGroups][kCols];
    const int tid = threadIdx.x, lane = tid & 63, g = tid >> 6;
    const uint32_t b = blockIdx.y;
    const uint32_t i = blockIdx.x * kCols + lane;
    const bool act = i < m;
    const uint32_t* ei = ex_idx + (size_t)b * tx;
    const uint32_t* ev = ex_val + (size_t)b * tx;
    uint64_t acc = 0;
    for (uint32_t s0 = 0; s0 < tx; s0 += kStage) {
        const uint32_t cnt = (tx - s0) < (uint32_t)kStage ? (tx - s0) : (uint32_t)kStage;
        __syncthreads();
        if ((uint32_t)tid < cnt) {
            uint32_t j = ei[s0 + tid];
            s_idx[tid] = j < Nx ? j : Nx - 1;
            s_val[tid] = ev[s0 + tid];
        }
        __syncthreads();
#pragma unroll 8
        for (uint32_t s = g; s < cnt; s += kGroups) {
            const uint32_t p = act ? PT[(size_t)s_idx[s] * m + i] : 0u;
            acc += ffold((uint64_t)s_val[s] * p);
        }
    }
    part[g][lane] = acc;
    __syncthreads();
    if (g == 0) {
        uint64_t tot = 0;
#pragma unroll
        for (int h = 0; h < kGroups; ++h) tot += part[h][lane];
        const uint32_t yh = act ? Yhat[(size_t)b * m + i] : 0u;
        if (act) Y[(size_t)b * m + i] = fsub(yh, fred64(tot));
        const uint32_t nblk = gridDim.x;
        for (uint32_t q = 0; q < ell; ++q) {
            const uint64_t prod = act ? ffold((uint64_t)rv[(size_t)q * m + i] * yh) : 0ull;
            const uint64_t ws = wave_sum_u64(prod);
            if (lane == 0) partR[((size_t)q * B + b) * nblk + blockIdx.x] = fred64(ws);
        }
    }
}

// grid (ceil(n / kCols))
__global__ __launch_bounds__(kB) void verify_vl(const uint32_t* __restrict__ Q, uint32_t n, uint32_t Ny,
                                                const uint32_t* __restrict__ Xhat, uint32_t B,
                                                const uint32_t* __restrict__ ey_idx,
                                                const uint32_t* __restrict__ ey_val, uint32_t ty, uint32_t ell,
                                                uint32_t* __restrict__ partL) {
    __shared__ uint32_t s_idx[kStage], s_val[kStage];
    __shared__ uint64_t part[kGroups][kCols];
    __shared__ uint32_t u_s[kCols];
    const int tid = threadIdx.x, lane = tid & 63, g = tid >> 6;
    const uint32_t k = blockIdx.x * kCols + lane;
    const bool act = k < n;
    const uint32_t nblk = gridDim.x;
    for (uint32_t q = 0; q < ell; ++q) {
        const uint32_t* ei = ey_idx + (size_t)q * ty;
        const uint32_t* ev = ey_val + (size_t)q * ty;
        uint64_t acc = 0;
        for (uint32_t s0 = 0; s0 < ty; s0 += kStage) {
            const uint32_t cnt = (ty - s0) < (uint32_t)kStage ? (ty - s0) : (uint32_t)kStage;
            __syncthreads();
            if ((uint32_t)tid < cnt) {
                uint32_t j = ei[s0 + tid];
                s_idx[tid] = j < Ny ? j : Ny - 1;
                s_val[tid] = ev[s0 + tid];
            }
            __syncthreads();
#pragma unroll 8
            for (uint32_t s = g; s < cnt; s += kGroups) {
                const uint32_t qv = act ? Q[(size_t)s_idx[s] * n + k] : 0u;
                acc += ffold((uint64_t)s_val[s] * qv);
            }
        }
        part[g][lane] = acc;
        __syncthreads();
        if (g == 0) {
            uint64_t tot = 0;
#pragma unroll
            for (int h = 0; h < kGroups; ++h) tot += part[h][lane];
            u_s[lane] = fred64(tot);  // (e_q^T Q)[k]
        }
        __syncthreads();
        const uint32_t u = u_s[lane];
        for (uint32_t b = g; b < B; b += kGroups) {
            const uint32_t x = act ? Xhat[(size_t)b * n + k] : 0u;
            const uint64_t ws = wave_sum_u64(ffold((uint64_t)u * x));
            if (lane == 0) partL[((size_t)q * B + b) * nblk + blockIdx.x] = fred64(ws);
        }
    }
}

__global__ __launch_bounds__(256) void verify_finalize(const uint32_t* __restrict__ partL, uint32_t nblkL,
                                                       const uint32_t* __restrict__ partR, uint32_t nblkR,
                                                       uint32_t B, uint32_t ell, uint32_t* __restrict__ vL,
                                                       uint32_t* __restrict__ vR, uint32_t* __restrict__ accept) {
    for (uint32_t b = threadIdx.x; b < B; b += blockDim.x) {
        uint32_t ok = 1;
        for (uint32_t q = 0; q < ell; ++q) {
            uint64_t l = 0, r = 0;
            const uint32_t* pl = partL + ((size_t)q * B + b) * nblkL;
            const uint32_t* pr = partR + ((size_t)q * B + b) * nblkR;
            for (uint32_t t = 0; t < nblkL; ++t) l += pl[t];
            for (uint32_t t = 0; t < nblkR; ++t) r += pr[t];
            const uint32_t L = fred64(l), R = fred64(r);
            if (vL) vL[(size_t)q * B + b] = L;
            if (vR) vR[(size_t)q * B + b] = R;
            ok &= (L == R) ? 1u : 0u;
        }
        accept[b] = ok;
    }
}

}  // namespace

hipError_t launch_decode_vr(const uint32_t* PT, uint32_t m, uint32_t Nx, const uint32_t* Yhat, uint32_t B,
                            const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx, const uint32_t* r,
                            uint32_t ell, uint32_t* Y, uint32_t* partR, hipStream_t s) {
    hipLaunchKernelGGL(decode_vr, dim3(ceil_div(m, kCols), B), dim3(kB), 0, s, PT, m, Nx, Yhat, B, ex_idx, ex_val, tx,
                       r, ell, Y, partR);
    return hipGetLastError();
}

hipError_t launch_verify_vl(const uint32_t* Q, uint32_t n, uint32_t Ny, const uint32_t* Xhat, uint32_t B,
                            const uint32_t* ey_idx, const uint32_t* ey_val, uint32_t ty, uint32_t ell,
                            uint32_t* partL, hipStream_t s) {
    hipLaunchKernelGGL(verify_vl, dim3(ceil_div(n, kCols)), dim3(kB), 0, s, Q, n, Ny, Xhat, B, ey_idx, ey_val, ty, ell,
                       partL);
    return hipGetLastError();
}

hipError_t launch_verify_finalize(const uint32_t* partL, uint32_t nblkL, const uint32_t* partR, uint32_t nblkR,
                                  uint32_t B, uint32_t ell, uint32_t* vL, uint32_t* vR, uint32_t* accept,
                                  hipStream_t s) {
    hipLaunchKernelGGL(verify_finalize, dim3(1), dim3(256), 0, s, partL, nblkL, partR, nblkR, B, ell, vL, vR, accept);
    return hipGetLastError();
}

}  // namespace mvk
