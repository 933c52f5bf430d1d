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
// columns (one per lane) x kGroups thread groups (one wave each), each group
// taking a contiguous quarter of the sparse terms.
constexpr int kCols = kClientCols;
constexpr int kGroups = kB / kCols;

// Gathers run in batches of kBatch terms per thread group.  Each load uses an
// in-range address (clamped position, column clamped to 0 for lanes past the
// end) and is masked afterwards, so a batch is issued without branches and all
// its loads are in flight together.  The sparse (index, value) pairs are read
// with wave-uniform addresses (scalar loads).
constexpr int kBatch = 16;

// Decode role: columns [cb*kCols, cb*kCols + kCols) of response b.
__device__ __forceinline__ void decode_part(const uint32_t* __restrict__ PT, uint32_t m, uint32_t Nx,
                                            const uint32_t* __restrict__ Yhat, uint32_t B,
                                            const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val,
                                            uint32_t tx, const uint32_t* __restrict__ rv, uint32_t ell,
                                            uint32_t* __restrict__ Y, uint32_t* __restrict__ partR, uint32_t b,
                                            uint32_t cb, uint32_t nblkR, uint64_t (*part)[kCols]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int g = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform group
    const uint32_t i = cb * kCols + lane;
    const bool act = i < m;
    const uint32_t is = act ? i : 0u;
    const uint32_t* ei = ex_idx + (size_t)b * tx;
    const uint32_t* ev = ex_val + (size_t)b * tx;
    const uint32_t yraw = Yhat[(size_t)b * m + is];
    // group g takes the contiguous terms [g*chunk, min(tx, g*chunk + chunk))
    const uint32_t chunk = (tx + kGroups - 1) / kGroups;
    const uint32_t s_beg = (uint32_t)g * chunk;
    const uint32_t s_end = s_beg + chunk < tx ? s_beg + chunk : tx;
    uint64_t acc = 0;
    for (uint32_t s0 = s_beg; s0 < s_end; s0 += kBatch) {
        uint32_t pv[kBatch], ww[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const uint32_t s = s0 + (uint32_t)u;
            const bool ok = s < s_end;
            const uint32_t sl = ok ? s : s_beg;  // in-range term, value masked below
            uint32_t j = ei[sl];
            j = j < Nx ? j : Nx - 1;
            ww[u] = ok ? ev[sl] : 0u;
            pv[u] = PT[(size_t)j * m + is];
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) acc += ffold((uint64_t)ww[u] * pv[u]);
    }
    part[g][lane] = acc;
    __syncthreads();
    if (g == 0) {
        uint64_t tot = 0;
#pragma unroll
        for (int h = 0; h < kGroups; ++h) tot += part[h][lane];
        const uint32_t yh = act ? yraw : 0u;
        if (act) Y[(size_t)b * m + i] = fsub(yh, fred64(tot));
        for (uint32_t q = 0; q < ell; ++q) {
            const uint64_t prod = ffold((uint64_t)rv[(size_t)q * m + is] * yh);
            const uint64_t ws = wave_sum_u64(prod);
            if (lane == 0) partR[((size_t)q * B + b) * nblkR + cb] = fred64(ws);
        }
    }
}

// Verify role: columns [cb*kCols, cb*kCols + kCols) of u_q = e_q^T Q.
__device__ __forceinline__ void verify_part(const uint32_t* __restrict__ Q, uint32_t n, uint32_t Ny,
                                            const uint32_t* __restrict__ Xhat, uint32_t B,
                                            const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val,
                                            uint32_t ty, uint32_t ell, uint32_t* __restrict__ partL, uint32_t cb,
                                            uint32_t nblkL, uint64_t (*part)[kCols], uint32_t* u_s) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int g = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform group
    const uint32_t k = cb * kCols + lane;
    const bool act = k < n;
    const uint32_t ks = act ? k : 0u;
    const uint32_t chunk = (ty + kGroups - 1) / kGroups;
    const uint32_t s_beg = (uint32_t)g * chunk;
    const uint32_t s_end = s_beg + chunk < ty ? s_beg + chunk : ty;
    for (uint32_t q = 0; q < ell; ++q) {
        const uint32_t* ei = ey_idx + (size_t)q * ty;
        const uint32_t* ev = ey_val + (size_t)q * ty;
        uint64_t acc = 0;
        for (uint32_t s0 = s_beg; s0 < s_end; s0 += kBatch) {
            uint32_t qv[kBatch], ww[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const uint32_t s = s0 + (uint32_t)u;
                const bool ok = s < s_end;
                const uint32_t sl = ok ? s : s_beg;  // in-range term, value masked below
                uint32_t j = ei[sl];
                j = j < Ny ? j : Ny - 1;
                ww[u] = ok ? ev[sl] : 0u;
                qv[u] = Q[(size_t)j * n + ks];
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) acc += ffold((uint64_t)ww[u] * qv[u]);
        }
        part[g][lane] = acc;
        __syncthreads();
        if (g == 0) {
            uint64_t tot = 0;
#pragma unroll
            for (int h = 0; h < kGroups; ++h) tot += part[h][lane];
            u_s[lane] = act ? fred64(tot) : 0u;  // (e_q^T Q)[k]
        }
        __syncthreads();
        const uint32_t u = u_s[lane];
        for (uint32_t b = g; b < B; b += kGroups) {
            const uint32_t x = Xhat[(size_t)b * n + ks];
            const uint64_t ws = wave_sum_u64(ffold((uint64_t)u * x));
            if (lane == 0) partL[((size_t)q * B + b) * nblkL + cb] = fred64(ws);
        }
        __syncthreads();
    }
}

// One launch for Decrypt, the two inner products of Verify and the final
// comparison.  Workgroups [0, B*nblkR) take the decode role, the next nblkL
// the verify role.  Every workgroup publishes its partial sums, then counts
// itself done on `counter`; the workgroup that finishes last (it sees
// count == gridDim.x - 1) sums all partials, writes vL, vR and accept, and
// resets the counter to zero for the next launch.
__global__ __launch_bounds__(kB) void decode_verify_fused(
    const uint32_t* __restrict__ PT, const uint32_t* __restrict__ Q, uint32_t m, uint32_t n, uint32_t Nx,
    uint32_t Ny, const uint32_t* __restrict__ Xhat, const uint32_t* __restrict__ Yhat, uint32_t B,
    const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val, uint32_t tx,
    const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val, uint32_t ty, uint32_t ell,
    const uint32_t* __restrict__ rv, uint32_t* __restrict__ Y, uint32_t* partL, uint32_t* partR,
    uint32_t nblkL, uint32_t nblkR, uint32_t* counter, uint32_t* __restrict__ vL, uint32_t* __restrict__ vR,
    uint32_t* __restrict__ accept) {
    __shared__ uint64_t part[kGroups][kCols];
    __shared__ uint32_t u_s[kCols];
    __shared__ uint32_t last;
    const uint32_t bid = blockIdx.x;
    const uint32_t ndec = B * nblkR;
    if (bid < ndec)
        decode_part(PT, m, Nx, Yhat, B, ex_idx, ex_val, tx, rv, ell, Y, partR, bid / nblkR, bid % nblkR, nblkR, part);
    else
        verify_part(Q, n, Ny, Xhat, B, ey_idx, ey_val, ty, ell, partL, bid - ndec, nblkL, part, u_s);

    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();  // publish this workgroup's partials
        last = (atomicAdd(counter, 1u) == gridDim.x - 1) ? 1u : 0u;
    }
    __syncthreads();
    if (!last) return;
    __threadfence();  // see every other workgroup's partials
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (uint32_t b = wave; b < B; b += kGroups) {
        uint32_t ok = 1;
        for (uint32_t q = 0; q < ell; ++q) {
            const uint32_t* pl = partL + ((size_t)q * B + b) * nblkL;
            const uint32_t* pr = partR + ((size_t)q * B + b) * nblkR;
            uint64_t l = 0, r = 0;
            for (uint32_t t = lane; t < nblkL; t += 64) l += pl[t];
            for (uint32_t t = lane; t < nblkR; t += 64) r += pr[t];
            const uint32_t L = fred64(wave_sum_u64(l)), R = fred64(wave_sum_u64(r));
            if (lane == 0) {
                if (vL) vL[(size_t)q * B + b] = L;
                if (vR) vR[(size_t)q * B + b] = R;
            }
            ok &= (L == R) ? 1u : 0u;
        }
        if (lane == 0) accept[b] = ok;
    }
    if (threadIdx.x == 0) atomicExch(counter, 0u);
}

}  // namespace

hipError_t launch_decode_verify(const uint32_t* PT, const uint32_t* Q, uint32_t m, uint32_t n, uint32_t Nx,
                                uint32_t Ny, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx, const uint32_t* ey_idx,
                                const uint32_t* ey_val, uint32_t ty, uint32_t ell, const uint32_t* r, uint32_t* Y,
                                uint32_t* partL, uint32_t* partR, uint32_t* counter, uint32_t* vL, uint32_t* vR,
                                uint32_t* accept, hipStream_t s) {
    const uint32_t nblkL = ceil_div(n, kCols), nblkR = ceil_div(m, kCols);
    const uint32_t grid = B * nblkR + nblkL;
    hipLaunchKernelGGL(decode_verify_fused, dim3(grid), dim3(kB), 0, s, PT, Q, m, n, Nx, Ny, Xhat, Yhat, B, ex_idx,
                       ex_val, tx, ey_idx, ey_val, ty, ell, r, Y, partL, partR, nblkL, nblkR, counter, vL, vR,
                       accept);
    return hipGetLastError();
}

}  // namespace mvk
