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
// and reduced once per workgroup; the per-workgroup partials (each < p) are
// added into 64-bit accumulators with atomics and reduced by the last
// workgroup.  All sums are exact, so results do not depend on the order.
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

// Prefetch depth of the per-lane values that do not depend on the gathers:
// the r_q values of the decode role (repetitions q < kPreQ) and the query
// values of the verify role (the first kPreB columns of each wave).
constexpr int kPreQ = 4;
constexpr int kPreB = 4;
constexpr int kItems = kMaxEll;  // verify work items (repetition, chunk) per workgroup, at most

// Decode role: columns [cb*kCols, cb*kCols + kCols) of response b.
__device__ __forceinline__ void decode_part(const uint32_t* __restrict__ PT, uint32_t m, uint32_t Nx,
                                            const uint32_t* __restrict__ Yhat, uint32_t B,
                                            const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val,
                                            uint32_t tx, const uint32_t* __restrict__ rv, uint32_t ell,
                                            uint32_t* __restrict__ Y, unsigned long long* accR, uint32_t b,
                                            uint32_t cb, uint64_t (*part)[kCols]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int g = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform group
    const uint32_t i = cb * kCols + lane;
    const bool act = i < m;
    const uint32_t is = act ? i : 0u;
    const uint32_t* ei = ex_idx + (size_t)b * tx;
    const uint32_t* ev = ex_val + (size_t)b * tx;
    const uint32_t yraw = Yhat[(size_t)b * m + is];
    uint32_t rq[kPreQ];
    if (g == 0) {
#pragma unroll
        for (int q = 0; q < kPreQ; ++q) rq[q] = rv[(size_t)((uint32_t)q < ell ? q : 0) * m + is];
    }
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
        // v_R partial: sum over this block's outputs of r_q[i] * yhat[i]
        for (uint32_t q = 0; q < ell; ++q) {
            uint32_t r = 0;
#pragma unroll
            for (int u = 0; u < kPreQ; ++u)
                if ((uint32_t)u == q) r = rq[u];
            if (q >= (uint32_t)kPreQ) r = rv[(size_t)q * m + is];
            const uint64_t ws = wave_sum_u64(ffold((uint64_t)r * yh));
            if (lane == 0) atomicAdd(&accR[(size_t)q * B + b], (unsigned long long)fred64(ws));
        }
    }
}

// v_L partials of one query column: sum over this block's k of u_q[k] * x[k].
__device__ __forceinline__ void verify_column(const uint32_t (*u_s)[kCols], uint32_t ell, uint32_t B, uint32_t b,
                                              uint32_t x, unsigned long long* accL) {
    const int lane = threadIdx.x & 63;
    for (uint32_t q = 0; q < ell; ++q) {
        const uint64_t ws = wave_sum_u64(ffold((uint64_t)u_s[q][lane] * x));
        if (lane == 0) atomicAdd(&accL[(size_t)q * B + b], (unsigned long long)fred64(ws));
    }
}

// Verify role: columns [cb*kCols, cb*kCols + kCols) of u_q = e_q^T Q for every
// repetition q.  The ell*ty terms are cut into work items (repetition q, chunk
// c), C chunks per repetition so that the kGroups waves are busy, and the waves
// take the items round robin; every item is one or more batches of gathers.
__device__ __forceinline__ void verify_part(const uint32_t* __restrict__ Q, uint32_t n, uint32_t Ny,
                                            const uint32_t* __restrict__ Xhat, uint32_t B,
                                            const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val,
                                            uint32_t ty, uint32_t ell, unsigned long long* accL, uint32_t cb,
                                            uint64_t (*part)[kCols], uint32_t (*u_s)[kCols]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int g = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform group
    const uint32_t k = cb * kCols + lane;
    const bool act = k < n;
    const uint32_t ks = act ? k : 0u;
    uint32_t xp[kPreB];
#pragma unroll
    for (int u = 0; u < kPreB; ++u) {
        const uint32_t b = (uint32_t)g + kGroups * u;
        xp[u] = Xhat[(size_t)(b < B ? b : 0u) * n + ks];
    }
    const uint32_t C = ell >= (uint32_t)kGroups ? 1u : (uint32_t)kGroups / ell;
    const uint32_t chunk = (ty + C - 1) / C;
    const uint32_t items = ell * C;
    for (uint32_t w = g; w < items; w += kGroups) {
        const uint32_t q = w / C, c = w % C;
        const uint32_t* ei = ey_idx + (size_t)q * ty;
        const uint32_t* ev = ey_val + (size_t)q * ty;
        const uint32_t s_beg = c * chunk;
        const uint32_t s_end = s_beg + chunk < ty ? s_beg + chunk : ty;
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
        part[w][lane] = acc;
    }
    __syncthreads();
    for (uint32_t q = g; q < ell; q += kGroups) {
        uint64_t tot = 0;
        for (uint32_t c = 0; c < C; ++c) tot += part[q * C + c][lane];
        u_s[q][lane] = act ? fred64(tot) : 0u;  // (e_q^T Q)[k]
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kPreB; ++u) {
        const uint32_t b = (uint32_t)g + kGroups * u;
        if (b < B) verify_column(u_s, ell, B, b, xp[u], accL);
    }
    for (uint32_t b = (uint32_t)g + kGroups * kPreB; b < B; b += kGroups)
        verify_column(u_s, ell, B, b, Xhat[(size_t)b * n + ks], accL);
}

// One launch for Decrypt, the two inner products of Verify and the final
// comparison.  Workgroups [0, B*nblkR) take the decode role, the next nblkL
// the verify role.  Every workgroup adds its partial sums (each < p) into the
// 64-bit accumulators accL / accR (ell x B each; exact, so the order of the
// additions does not matter), then counts itself done on `counter`; the
// workgroup that finishes last (it sees count == gridDim.x - 1) reads and
// clears the accumulators, writes vL, vR and accept, and resets the counter,
// so every launch leaves the accumulators and the counter at zero.
__global__ __launch_bounds__(kB) void decode_verify_fused(
    const uint32_t* __restrict__ PT, const uint32_t* __restrict__ Q, uint32_t m, uint32_t n, uint32_t Nx,
    uint32_t Ny, const uint32_t* __restrict__ Xhat, const uint32_t* __restrict__ Yhat, uint32_t B,
    const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val, uint32_t tx,
    const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val, uint32_t ty, uint32_t ell,
    const uint32_t* __restrict__ rv, uint32_t* __restrict__ Y, unsigned long long* accL, unsigned long long* accR,
    uint32_t nblkR, uint32_t* counter, uint32_t* __restrict__ vL, uint32_t* __restrict__ vR,
    uint32_t* __restrict__ accept) {
    __shared__ uint64_t part[kItems][kCols];
    __shared__ uint32_t u_s[kMaxEll][kCols];
    __shared__ uint32_t last;
    const uint32_t bid = blockIdx.x;
    const uint32_t ndec = B * nblkR;
    if (bid < ndec)
        decode_part(PT, m, Nx, Yhat, B, ex_idx, ex_val, tx, rv, ell, Y, accR, bid / nblkR, bid % nblkR, part);
    else
        verify_part(Q, n, Ny, Xhat, B, ey_idx, ey_val, ty, ell, accL, bid - ndec, part, u_s);

    // Ordering without cache-wide fences: the accumulators are touched only by
    // atomics, which are performed at the device-wide coherence point.  Every
    // wave waits for its atomics to complete (vmcnt 0) before the barrier, the
    // counter increment follows the barrier, and the last workgroup reads the
    // accumulators with atomics after seeing the final count.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) last = (atomicAdd(counter, 1u) == gridDim.x - 1) ? 1u : 0u;
    __syncthreads();
    if (!last) return;
    for (uint32_t b = threadIdx.x; b < B; b += kB) {
        uint32_t ok = 1;
        for (uint32_t q = 0; q < ell; ++q) {
            const size_t o = (size_t)q * B + b;
            const uint32_t L = fred64(atomicExch(&accL[o], 0ull));
            const uint32_t R = fred64(atomicExch(&accR[o], 0ull));
            if (vL) vL[o] = L;
            if (vR) vR[o] = R;
            ok &= (L == R) ? 1u : 0u;
        }
        accept[b] = ok;
    }
    if (threadIdx.x == 0) atomicExch(counter, 0u);
}

}  // namespace

hipError_t launch_decode_verify(const uint32_t* PT, const uint32_t* Q, uint32_t m, uint32_t n, uint32_t Nx,
                                uint32_t Ny, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx, const uint32_t* ey_idx,
                                const uint32_t* ey_val, uint32_t ty, uint32_t ell, const uint32_t* r, uint32_t* Y,
                                unsigned long long* acc, uint32_t* counter, uint32_t* vL, uint32_t* vR,
                                uint32_t* accept, hipStream_t s) {
    if (ell == 0 || ell > (uint32_t)kMaxEll) return hipErrorInvalidValue;
    const uint32_t nblkL = ceil_div(n, kCols), nblkR = ceil_div(m, kCols);
    const uint32_t grid = B * nblkR + nblkL;
    hipLaunchKernelGGL(decode_verify_fused, dim3(grid), dim3(kB), 0, s, PT, Q, m, n, Nx, Ny, Xhat, Yhat, B, ex_idx,
                       ex_val, tx, ey_idx, ey_val, ty, ell, r, Y, acc, acc + (size_t)ell * B, nblkR, counter, vL, vR,
                       accept);
    return hipGetLastError();
}

}  // namespace mvk
