// Batch verification (Protocol Batch-vMVMD, Sec. 5.4) on gfx950: B claims
// M_b x_b = y_b of one shape under one primary code G, whose per-claim
// challenge projections u_b = Q_b^T e are delegated to the server and checked
// with a second code G' over F^{Bn}.
//
//   Preprocess:  QtT = [Q_1 | ... | Q_B] (N x Bn; row i = (Q_1[i,:], ..., Q_B[i,:]))
//                Qaux = QtT G'           (N x N'; row i = G'^T (row i of QtT))
//   Server:      u~(q) = Qt e(q) = sum_{j in supp(e)} e_j QtT[j, :]      (Bn)
//   Client:      original  (u_b(q))^T x_b  ==  (G e(q))^T y_b
//                secondary (e(q))^T Qaux e'(j)  ==  (G' e'(j))^T u~(q)
// The primary side uses the transposed form of App. B, as the one-claim
// Verify does: (e^T G^T) y = (G e)^T y, one syndrome per repetition.
#include "count.h"
#include "field.h"
#include "mvk_internal.h"

namespace mvk {

namespace {

constexpr int kBT = 256;     // threads per workgroup of the check kernel
constexpr int kBW = kBT / 64;

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

// Sum of one value per thread over the workgroup, added into *acc (64-bit
// atomics: exact, so the order of the additions does not matter).
__device__ __forceinline__ void block_add(uint64_t v, uint64_t* red, unsigned long long* acc) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    v = wave_sum_u64(v);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t t = 0;
#pragma unroll
        for (int w = 0; w < kBW; ++w) t += red[w];
        atomicAdd(acc, (unsigned long long)fred64(t));
    }
    __syncthreads();  // red is reused
}

struct CheckArgs {
    uint32_t m, n, B, ell, ell2, t, t2, N, N2;
    const uint32_t *X, *Y, *Ut, *R, *Rs, *Qaux;
    const uint32_t *e_idx, *e_val, *e2_idx, *e2_val;
    unsigned long long *accL, *accR, *accS, *accA;  // ell x B, ell x B, ell x ell2, ell x ell2
    uint32_t* ctrl;  // completion counters (count.h)
    uint32_t slots;
    uint32_t *vL, *vR, *sL, *sR, *accept;
    uint32_t nbL, nbR, nbS;  // 256-element blocks of n, m and Bn
};

// Workgroups [0, B*nbL): v_L terms u_b(q)[k] x_b[k]; next B*nbR: v_R terms
// R_q[i] y_b[i]; next nbS: secondary right sides r_j[c] u~(q)[c]; the last
// ell*ell2: the t x t' lookups of one secondary left side each.  Partial sums go into
// 64-bit accumulators; the workgroup that finishes last (count.h) reads and
// clears them and writes the results and the accept bits.
__global__ __launch_bounds__(kBT) void batch_check_kernel(CheckArgs a) {
    __shared__ uint64_t red[kBW];
    __shared__ uint32_t last;
    const uint32_t bid = blockIdx.x, tid = threadIdx.x;
    const uint32_t Bn = a.B * a.n;
    const uint32_t nL = a.B * a.nbL, nR = a.B * a.nbR;
    if (bid < nL) {
        const uint32_t b = bid / a.nbL, k = (bid % a.nbL) * kBT + tid;
        const bool act = k < a.n;
        const uint32_t ks = act ? k : 0u;
        const uint32_t x = act ? a.X[(size_t)b * a.n + ks] : 0u;
        for (uint32_t q = 0; q < a.ell; ++q)
            block_add(ffold((uint64_t)a.Ut[(size_t)q * Bn + (size_t)b * a.n + ks] * x), red,
                      &a.accL[(size_t)q * a.B + b]);
    } else if (bid < nL + nR) {
        const uint32_t w = bid - nL;
        const uint32_t b = w / a.nbR, i = (w % a.nbR) * kBT + tid;
        const bool act = i < a.m;
        const uint32_t is = act ? i : 0u;
        const uint32_t y = act ? a.Y[(size_t)b * a.m + is] : 0u;
        for (uint32_t q = 0; q < a.ell; ++q)
            block_add(ffold((uint64_t)a.R[(size_t)q * a.m + is] * y), red, &a.accR[(size_t)q * a.B + b]);
    } else if (bid < nL + nR + a.nbS) {
        const uint32_t c = (bid - nL - nR) * kBT + tid;
        const bool act = c < Bn;
        const uint32_t cs = act ? c : 0u;
        for (uint32_t j = 0; j < a.ell2; ++j) {
            const uint32_t rj = act ? a.Rs[(size_t)j * Bn + cs] : 0u;
            for (uint32_t q = 0; q < a.ell; ++q)
                block_add(ffold((uint64_t)rj * a.Ut[(size_t)q * Bn + cs]), red, &a.accS[(size_t)q * a.ell2 + j]);
        }
    } else {
        // one (q, j) pair per workgroup; the t x t' lookups kLook per thread
        // and pass, every load of a pass issued before the first use
        constexpr int kLook = 4;
        const uint32_t qj = bid - nL - nR - a.nbS, q = qj / a.ell2, j = qj % a.ell2;
        const uint32_t pairs = a.t * a.t2;
        uint64_t s = 0;
        for (uint32_t p0 = 0; p0 < pairs; p0 += kBT * kLook) {
            uint32_t row[kLook], col[kLook], w1[kLook], w2[kLook], ent[kLook];
#pragma unroll
            for (int u = 0; u < kLook; ++u) {
                const uint32_t p = p0 + tid + kBT * u;
                const uint32_t ps = p < pairs ? p : 0u;
                const uint32_t x = ps / a.t2, y = ps % a.t2;
                row[u] = a.e_idx[(size_t)q * a.t + x];
                col[u] = a.e2_idx[(size_t)j * a.t2 + y];
                w1[u] = a.e_val[(size_t)q * a.t + x];
                w2[u] = p < pairs ? a.e2_val[(size_t)j * a.t2 + y] : 0u;
            }
#pragma unroll
            for (int u = 0; u < kLook; ++u) {
                const uint32_t rr = row[u] < a.N ? row[u] : a.N - 1, cc = col[u] < a.N2 ? col[u] : a.N2 - 1;
                ent[u] = a.Qaux[(size_t)rr * a.N2 + cc];
            }
#pragma unroll
            for (int u = 0; u < kLook; ++u) s += ffold((uint64_t)fmul(w1[u], ent[u]) * w2[u]);
        }
        block_add(s, red, &a.accA[(size_t)q * a.ell2 + j]);
    }
    // Completion as in the decode/verify kernels: atomics complete (vmcnt 0)
    // before the barrier, the count after it, the last workgroup reads the
    // accumulators with atomics.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) last = count_last(a.ctrl, a.slots) ? 1u : 0u;
    __syncthreads();
    if (!last) return;
    // secondary checks (one bit for the batch), then the claims
    __shared__ uint32_t sec_ok;
    if (tid == 0) sec_ok = 1u;
    __syncthreads();
    for (uint32_t o = tid; o < a.ell * a.ell2; o += kBT) {
        const uint32_t L = fred64(atomicExch(&a.accA[o], 0ull));
        const uint32_t Rr = fred64(atomicExch(&a.accS[o], 0ull));
        if (a.sL) a.sL[o] = L;
        if (a.sR) a.sR[o] = Rr;
        if (L != Rr) atomicAnd(&sec_ok, 0u);
    }
    __syncthreads();
    for (uint32_t b = tid; b < a.B; b += kBT) {
        uint32_t ok = sec_ok;
        for (uint32_t q = 0; q < a.ell; ++q) {
            const size_t o = (size_t)q * a.B + b;
            const uint32_t L = fred64(atomicExch(&a.accL[o], 0ull));
            const uint32_t Rr = fred64(atomicExch(&a.accR[o], 0ull));
            if (a.vL) a.vL[o] = L;
            if (a.vR) a.vR[o] = Rr;
            ok &= (L == Rr) ? 1u : 0u;
        }
        a.accept[b] = ok;
    }
}

}  // namespace

size_t batch_ctrl_bytes(uint32_t m, uint32_t n, uint32_t B, uint32_t ell, uint32_t ell2) {
    const uint64_t grid = (uint64_t)B * (ceil_div(n, kBT) + ceil_div(m, kBT)) + ceil_div(B * n, kBT) +
                          (uint64_t)ell * ell2;
    const uint32_t slots = count_slots(grid > 0xffffffffull ? 0xffffffffu : (uint32_t)grid);
    return (size_t)count_words(slots) * 4 + ((size_t)2 * ell * B + (size_t)2 * ell * ell2) * 8;
}

hipError_t launch_batch_check(uint32_t m, uint32_t n, uint32_t B, const uint32_t* X, const uint32_t* Y,
                              const uint32_t* Ut, const uint32_t* R, const uint32_t* Rs, const uint32_t* Qaux,
                              uint32_t N, uint32_t N2, const uint32_t* e_idx, const uint32_t* e_val, uint32_t t,
                              uint32_t ell, const uint32_t* e2_idx, const uint32_t* e2_val, uint32_t t2,
                              uint32_t ell2, uint32_t* ctrl, uint32_t* vL, uint32_t* vR, uint32_t* sL, uint32_t* sR,
                              uint32_t* accept, hipStream_t s) {
    CheckArgs a;
    a.m = m, a.n = n, a.B = B, a.ell = ell, a.ell2 = ell2, a.t = t, a.t2 = t2, a.N = N, a.N2 = N2;
    a.X = X, a.Y = Y, a.Ut = Ut, a.R = R, a.Rs = Rs, a.Qaux = Qaux;
    a.e_idx = e_idx, a.e_val = e_val, a.e2_idx = e2_idx, a.e2_val = e2_val;
    a.vL = vL, a.vR = vR, a.sL = sL, a.sR = sR, a.accept = accept;
    a.nbL = ceil_div(n, kBT), a.nbR = ceil_div(m, kBT), a.nbS = ceil_div(B * n, kBT);
    const uint64_t grid = (uint64_t)B * (a.nbL + a.nbR) + a.nbS + (uint64_t)ell * ell2;
    if (grid > 0x7fffffffu) return hipErrorInvalidValue;
    a.ctrl = ctrl;
    a.slots = count_slots((uint32_t)grid);
    a.accL = reinterpret_cast<unsigned long long*>(ctrl + count_words(a.slots));
    a.accR = a.accL + (size_t)ell * B;
    a.accS = a.accR + (size_t)ell * B;
    a.accA = a.accS + (size_t)ell * ell2;
    hipLaunchKernelGGL(batch_check_kernel, dim3((uint32_t)grid), dim3(kBT), 0, s, a);
    return hipGetLastError();
}

}  // namespace mvk
