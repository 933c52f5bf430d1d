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
// Every (repetition, column) sum has nsub accumulators, 64 bits each, which
// the workgroups of a column use in turn (block index mod nsub): atomics on one
// address are serialised, so this bounds the workgroups per address.
#include <initializer_list>

#include "count.h"
#include "field.h"
#include "masks.h"
#include "mvk_internal.h"
#include "syn_block.h"

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

// Workgroup shape of the gather roles: kCols consecutive output columns (one
// per lane) x G thread groups (one wave each), each group taking a contiguous
// share of the sparse terms.  G = kB / kCols in the plain kernel, G = 8 in the
// kernel that also computes the challenge syndromes.
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

// E consecutive words at p, non-temporal (the rows these loads stream are read
// once per launch; E = 4: one 16-byte access, p 16-byte aligned).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <int E>
__device__ __forceinline__ void load_cols(const uint32_t* p, uint32_t (&v)[E]) {
    if constexpr (E == 4) {
        const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
        v[0] = t.x;
        v[1] = t.y;
        v[2] = t.z;
        v[3] = t.w;
    } else {
        v[0] = __builtin_nontemporal_load(p);
    }
}
template <int E>
__device__ __forceinline__ void store_cols(uint32_t* p, const uint32_t (&v)[E]) {
    if constexpr (E == 4)
        *reinterpret_cast<uint4*>(p) = make_uint4(v[0], v[1], v[2], v[3]);
    else
        *p = v[0];
}

// Workgroup of decode_verify_syn: 512 threads, so that one workgroup holds the
// syndrome of a block of up to 512 * 32 = 16384 positions in LDS.
constexpr int kFusedThreads = kDvSynThreads;

// decode_verify_masked runs on decode_verify_small (at most 8 workgroups) up
// to this many words of responses plus queries (B * (m + n)) and up to 4
// repetitions; above, on decode_verify_wide (up to 4 repetitions) or the
// multi-workgroup kernel above.
constexpr uint64_t kSmallDvWords = 32768;
constexpr int kFusedGroups = kFusedThreads / kCols;

// Spin limit of the wait for the challenge syndromes (s_sleep 2 per try, well
// over a second in total): a wait that does not end is reported, not hung.
constexpr uint32_t kSpinLimit = 1u << 24;

// Decode role: columns [cb*kCols*E, (cb+1)*kCols*E) of response b, E
// consecutive ones per lane, by the G*64 threads of the workgroup; the
// partial sums of the groups meet in `part` (G*E*64 values).  E = 4: m is a
// multiple of 4 and PT, Yhat, Y and rv are 16-byte aligned (16-byte loads, so
// a wave reads 1 KiB of a row of PT per term).  WAIT_R: the r_q are being written by other
// workgroups of the same launch; thread 0 waits until `rdone` reaches ell (or
// the spin limit passes, which sets *err), then, after a workgroup barrier,
// the r_q are read device-coherently.
//
// PRE: the output mask P e_b is given (My, B x m, from client_prepare) and
// replaces the gathers.
template <bool WAIT_R, int G, bool PRE = false, int E = 1>
__device__ __forceinline__ void decode_part(const uint32_t* __restrict__ PT, uint32_t m, uint32_t Nx,
                                            const uint32_t* __restrict__ Yhat, uint32_t B,
                                            const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val,
                                            uint32_t tx, const uint32_t* rv, uint32_t ell,
                                            uint32_t* __restrict__ Y, unsigned long long* accR, uint32_t nsub,
                                            uint32_t b, uint32_t cb, uint64_t* part, uint32_t* rdone,
                                            uint32_t* err, const uint32_t* __restrict__ My = nullptr) {
    static_assert(E == 1 || E == 4, "one or four columns per lane");
    const int lane = threadIdx.x & 63;
    const int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform group
    const uint32_t i0 = cb * (kCols * E) + (uint32_t)lane * E;
    const bool act = i0 < m;
    const uint32_t is = act ? i0 : 0u;
    const uint32_t* ei = ex_idx + (size_t)b * tx;
    const uint32_t* ev = ex_val + (size_t)b * tx;
    uint32_t yraw[E];
    load_cols<E>(Yhat + (size_t)b * m + is, yraw);
    uint32_t rq[kPreQ][E];
    if (!WAIT_R && g == 0) {
#pragma unroll
        for (int q = 0; q < kPreQ; ++q) load_cols<E>(rv + (size_t)((uint32_t)q < ell ? q : 0) * m + is, rq[q]);
    }
    // group g takes the contiguous terms [g*chunk, min(tx, g*chunk + chunk))
    if (PRE) tx = 0;
    const uint32_t chunk = (tx + G - 1) / G;
    const uint32_t s_beg = (uint32_t)g * chunk;
    const uint32_t s_end = s_beg + chunk < tx ? s_beg + chunk : tx;
    uint64_t acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0;
    for (uint32_t s0 = s_beg; s0 < s_end; s0 += kBatch) {
        uint32_t pv[kBatch][E], ww[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const uint32_t s = s0 + (uint32_t)u;
            const bool ok = s < s_end;
            const uint32_t sl = ok ? s : s_beg;  // in-range term, value masked below
            uint32_t j = ei[sl];
            j = j < Nx ? j : Nx - 1;
            ww[u] = ok ? ev[sl] : 0u;
            load_cols<E>(PT + (size_t)j * m + is, pv[u]);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] += ffold((uint64_t)ww[u] * pv[u][e]);
    }
    if (PRE && g == 0) {
        uint32_t mm[E];
        load_cols<E>(My + (size_t)b * m + is, mm);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = mm[e];
    }
#pragma unroll
    for (int e = 0; e < E; ++e) part[(g * E + e) * 64 + lane] = acc[e];
    __syncthreads();
    uint32_t yh[E];
#pragma unroll
    for (int e = 0; e < E; ++e) yh[e] = act ? yraw[e] : 0u;
    if (g == 0) {
        uint32_t y[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            uint64_t tot = 0;
#pragma unroll
            for (int h = 0; h < G; ++h) tot += part[(h * E + e) * 64 + lane];
            y[e] = fsub(yh[e], fred64(tot));
        }
        if (act && Y) store_cols<E>(Y + (size_t)b * m + i0, y);
    }
    if (WAIT_R) {
        if (threadIdx.x == 0) {
            uint32_t it = 0;
            while (__hip_atomic_load(rdone, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < ell) {
                if (++it > kSpinLimit) {
                    atomicOr(err, 1u);
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
        }
        __syncthreads();
        if (g == 0) {
#pragma unroll
            for (int q = 0; q < kPreQ; ++q)
#pragma unroll
                for (int e = 0; e < E; ++e)
                    rq[q][e] = __hip_atomic_load(&rv[(size_t)((uint32_t)q < ell ? q : 0) * m + is + e],
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (g == 0) {
        // v_R partial: sum over this block's outputs of r_q[i] * yhat[i]
        for (uint32_t q = 0; q < ell; ++q) {
            uint32_t r[E];
#pragma unroll
            for (int e = 0; e < E; ++e) r[e] = 0;
#pragma unroll
            for (int u = 0; u < kPreQ; ++u)
                if ((uint32_t)u == q)
#pragma unroll
                    for (int e = 0; e < E; ++e) r[e] = rq[u][e];
            if (q >= (uint32_t)kPreQ) {
#pragma unroll
                for (int e = 0; e < E; ++e)
                    r[e] = WAIT_R ? __hip_atomic_load(&rv[(size_t)q * m + is + e], __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)
                                  : rv[(size_t)q * m + is + e];
            }
            uint64_t t = 0;
#pragma unroll
            for (int e = 0; e < E; ++e) t += ffold((uint64_t)r[e] * yh[e]);
            const uint64_t ws = wave_sum_u64(t);
            if (lane == 0) atomicAdd(&accR[((size_t)q * B + b) * nsub + cb % nsub], (unsigned long long)fred64(ws));
        }
    }
}

// v_L partials of one query column: sum over this block's k of u_q[k] * x[k].
__device__ __forceinline__ void verify_column(const uint32_t (*u_s)[kCols], uint32_t ell, uint32_t B, uint32_t b,
                                              uint32_t x, unsigned long long* accL, uint32_t nsub, uint32_t sub) {
    const int lane = threadIdx.x & 63;
    for (uint32_t q = 0; q < ell; ++q) {
        const uint64_t ws = wave_sum_u64(ffold((uint64_t)u_s[q][lane] * x));
        if (lane == 0) atomicAdd(&accL[((size_t)q * B + b) * nsub + sub], (unsigned long long)fred64(ws));
    }
}

// Verify role: columns [cb*kCols, cb*kCols + kCols) of u_q = e_q^T Q for every
// repetition q.  The ell*ty terms are cut into work items (repetition q, chunk
// c), C chunks per repetition so that the kGroups waves are busy, and the waves
// take the items round robin; every item is one or more batches of gathers.
//
// PRE: u_q is given (U, ell x n, from client_prepare) and replaces the gathers.
template <int G, bool PRE = false>
__device__ __forceinline__ void verify_part(const uint32_t* __restrict__ Q, uint32_t n, uint32_t Ny,
                                            const uint32_t* __restrict__ Xhat, uint32_t B,
                                            const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val,
                                            uint32_t ty, uint32_t ell, unsigned long long* accL, uint32_t nsub,
                                            uint32_t cb, uint64_t (*part)[kCols], uint32_t (*u_s)[kCols],
                                            const uint32_t* __restrict__ U = nullptr) {
    static_assert(G <= kItems, "one work item per group at least");
    const int lane = threadIdx.x & 63;
    const int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform group
    const uint32_t k = cb * kCols + lane;
    const bool act = k < n;
    const uint32_t ks = act ? k : 0u;
    uint32_t xp[kPreB];
#pragma unroll
    for (int u = 0; u < kPreB; ++u) {
        const uint32_t b = (uint32_t)g + G * u;
        xp[u] = Xhat[(size_t)(b < B ? b : 0u) * n + ks];
    }
    const uint32_t C = ell >= (uint32_t)G ? 1u : (uint32_t)G / ell;
    const uint32_t chunk = (ty + C - 1) / C;
    const uint32_t items = PRE ? 0u : ell * C;
    for (uint32_t w = g; w < items; w += G) {
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
                qv[u] = __builtin_nontemporal_load(&Q[(size_t)j * n + ks]);  // rows read once per launch
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) acc += ffold((uint64_t)ww[u] * qv[u]);
        }
        part[w][lane] = acc;
    }
    __syncthreads();
    for (uint32_t q = g; q < ell; q += G) {
        if (PRE) {
            u_s[q][lane] = act ? U[(size_t)q * n + ks] : 0u;
        } else {
            uint64_t tot = 0;
            for (uint32_t c = 0; c < C; ++c) tot += part[q * C + c][lane];
            u_s[q][lane] = act ? fred64(tot) : 0u;  // (e_q^T Q)[k]
        }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kPreB; ++u) {
        const uint32_t b = (uint32_t)g + G * u;
        if (b < B) verify_column(u_s, ell, B, b, xp[u], accL, nsub, cb % nsub);
    }
    for (uint32_t b = (uint32_t)g + G * kPreB; b < B; b += G)
        verify_column(u_s, ell, B, b, Xhat[(size_t)b * n + ks], accL, nsub, cb % nsub);
}

// End of a decode/verify launch.  Ordering without cache-wide fences: the
// accumulators are touched only by atomics, which are performed at the
// device-wide coherence point.  Every wave waits for its atomics to complete
// (vmcnt 0) before the barrier, the completion count (count.h) follows the
// barrier, and the last workgroup reads the accumulators with atomics after
// it has been found.  It clears them, resets rdone / err (when given), and
// writes vL, vR and accept.
__device__ __forceinline__ void finish(uint32_t B, uint32_t ell, uint32_t nsub, unsigned long long* accL,
                                       unsigned long long* accR, uint32_t* ctrl, uint32_t slots, uint32_t* rdone,
                                       uint32_t* err, uint32_t* __restrict__ vL, uint32_t* __restrict__ vR,
                                       uint32_t* __restrict__ accept, uint32_t* last) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) *last = count_last(ctrl, slots) ? 1u : 0u;
    __syncthreads();
    if (!*last) return;
    const uint32_t bad = err ? __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
    for (uint32_t b = threadIdx.x; b < B; b += blockDim.x) {
        uint32_t ok = bad ? 0u : 1u;
        for (uint32_t q = 0; q < ell; ++q) {
            const size_t o = (size_t)q * B + b;
            uint64_t l = 0, r = 0;  // each accumulator < 2^61
            for (uint32_t u = 0; u < nsub; ++u) {
                l += atomicExch(&accL[o * nsub + u], 0ull);
                r += atomicExch(&accR[o * nsub + u], 0ull);
            }
            const uint32_t L = fred64(l), R = fred64(r);
            if (vL) vL[o] = L;
            if (vR) vR[o] = R;
            ok &= (L == R) ? 1u : 0u;
        }
        accept[b] = ok;
    }
    __syncthreads();  // every thread has read err
    if (threadIdx.x == 0) {
        if (rdone) atomicExch(rdone, 0u);
        if (err) atomicExch(err, 0u);
    }
}

// One launch for Decrypt, the two inner products of Verify and the final
// comparison.  Workgroups [0, B*nblkR) take the decode role, the next nblkL
// the verify role.  Every workgroup adds its partial sums (each < p) into the
// 64-bit accumulators accL / accR (ell x B x nsub each; exact, so the order of
// the additions does not matter), then counts itself done; the workgroup that
// finishes last reads and clears the accumulators and writes vL, vR and
// accept, so every launch leaves the accumulators and the counters at zero.
//
// PRE: the output masks My and the vectors u_q (U) come from client_prepare;
// the workgroups then only stream Yhat, My, r and U, Xhat.
template <bool PRE, int E>
__global__ __launch_bounds__(kB) void decode_verify_fused(
    const uint32_t* __restrict__ PT, const uint32_t* __restrict__ Q, uint32_t m, uint32_t n, uint32_t Nx,
    uint32_t Ny, const uint32_t* __restrict__ Xhat, const uint32_t* __restrict__ Yhat, uint32_t B,
    const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val, uint32_t tx,
    const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val, uint32_t ty, uint32_t ell,
    const uint32_t* __restrict__ rv, uint32_t* __restrict__ Y, unsigned long long* accL, unsigned long long* accR,
    uint32_t nsub, uint32_t nblkR, uint32_t* ctrl, uint32_t slots, uint32_t* __restrict__ vL,
    uint32_t* __restrict__ vR, uint32_t* __restrict__ accept, const uint32_t* __restrict__ My,
    const uint32_t* __restrict__ U) {
    __shared__ uint64_t part[kItems][kCols];
    __shared__ uint32_t u_s[kMaxEll][kCols];
    __shared__ uint32_t last;
    const uint32_t bid = blockIdx.x;
    const uint32_t ndec = B * nblkR;
    if (bid < ndec)
        decode_part<false, kGroups, PRE, E>(PT, m, Nx, Yhat, B, ex_idx, ex_val, tx, rv, ell, Y, accR, nsub,
                                            bid / nblkR, bid % nblkR, &part[0][0], nullptr, nullptr, My);
    else
        verify_part<kGroups, PRE>(Q, n, Ny, Xhat, B, ey_idx, ey_val, ty, ell, accL, nsub, bid - ndec, part, u_s,
                                  U);

    finish(B, ell, nsub, accL, accR, ctrl, slots, nullptr, nullptr, vL, vR, accept, &last);
}

// Syndrome role of decode_verify_syn: r_c = Gy e_c into rv (device-coherent
// stores), then rdone += 1 once every store of the workgroup has completed.
template <int U>
__device__ __forceinline__ void syn_part(uint32_t c, uint32_t k, uint32_t r, const uint32_t* __restrict__ pi1,
                                         const uint32_t* __restrict__ pi2, const uint32_t* __restrict__ v1,
                                         const uint32_t* __restrict__ v2, const uint32_t* __restrict__ ey_idx,
                                         const uint32_t* __restrict__ ey_val, uint32_t ty, uint32_t* rv,
                                         uint32_t* rdone, uint32_t* lds) {
    syn::syn_block<true, U, kFusedThreads, true>(c, k, r, pi1, pi2, v1, v2, nullptr, ey_idx, ey_val, ty, nullptr,
                                                 rv, lds);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) atomicAdd(rdone, 1u);
}

// LDS words of decode_verify_syn<U>: the syndrome work arrays, or the part and
// u_s arrays of the gather roles, whichever is larger (a workgroup has one role).
constexpr size_t kGatherWords = (sizeof(uint64_t) * kItems * kCols + sizeof(uint32_t) * kMaxEll * kCols) / 4;
constexpr size_t kDecodeWords = 2 * (size_t)kFusedGroups * 4 * kCols;  // decode role, E = 4
static_assert(kItems * kCols >= kGroups * 4 * kCols, "decode_verify_fused: part holds the decode role's sums");
template <int U>
constexpr size_t fused_lds_words() {
    constexpr size_t g = kGatherWords > kDecodeWords ? kGatherWords : kDecodeWords;
    return syn::lds_words<U, kFusedThreads>() > g ? syn::lds_words<U, kFusedThreads>() : g;
}

// decode_verify_fused with the challenge syndromes r_q = Gy e_q computed in the
// same launch (blocks of length Ny <= kFusedThreads * U).  Workgroups
// [0, ell) compute r_q (one repetition each, the whole block in LDS), the next
// nblkL take the verify role (which does not need r), the rest the decode
// role: their gathers and the Y outputs do not need r either, so only the v_R
// partials wait for the syndrome workgroups (rdone, counted up to ell).  The
// syndrome workgroups have the lowest indices and are dispatched first, so the
// waits end whatever the residency.  The last workgroup also resets rdone and
// err; if a wait ran into its spin limit, every column is rejected.
template <int U, int E>
__global__ __launch_bounds__(kFusedThreads) void decode_verify_syn(
    const uint32_t* __restrict__ PT, const uint32_t* __restrict__ Q, uint32_t m, uint32_t n, uint32_t Nx,
    uint32_t Ny, const uint32_t* __restrict__ Xhat, const uint32_t* __restrict__ Yhat, uint32_t B,
    const uint32_t* __restrict__ ex_idx, const uint32_t* __restrict__ ex_val, uint32_t tx,
    const uint32_t* __restrict__ ey_idx, const uint32_t* __restrict__ ey_val, uint32_t ty, uint32_t ell,
    uint32_t cyr, const uint32_t* __restrict__ pi1, const uint32_t* __restrict__ pi2,
    const uint32_t* __restrict__ v1, const uint32_t* __restrict__ v2, uint32_t* rv, uint32_t* __restrict__ Y,
    unsigned long long* accL, unsigned long long* accR, uint32_t nsub, uint32_t nblkR, uint32_t nblkL,
    uint32_t* ctrl, uint32_t slots, uint32_t* __restrict__ vL, uint32_t* __restrict__ vR,
    uint32_t* __restrict__ accept) {
    __shared__ __align__(16) uint32_t lds[fused_lds_words<U>()];
    __shared__ uint32_t last;
    auto part = reinterpret_cast<uint64_t (*)[kCols]>(lds);
    auto u_s = reinterpret_cast<uint32_t (*)[kCols]>(lds + 2 * kItems * kCols);
    uint32_t* rdone = &ctrl[1];
    uint32_t* err = &ctrl[2];
    const uint32_t bid = blockIdx.x;
    if (bid < ell)
        syn_part<U>(bid, m, cyr, pi1, pi2, v1, v2, ey_idx, ey_val, ty, rv, rdone, lds);
    else if (bid < ell + nblkL)
        verify_part<kFusedGroups>(Q, n, Ny, Xhat, B, ey_idx, ey_val, ty, ell, accL, nsub, bid - ell, part, u_s);
    else {
        const uint32_t d = bid - ell - nblkL;
        decode_part<true, kFusedGroups, false, E>(PT, m, Nx, Yhat, B, ex_idx, ex_val, tx, rv, ell, Y, accR, nsub,
                                                  d / nblkR, d % nblkR, reinterpret_cast<uint64_t*>(lds), rdone,
                                                  err);
    }
    finish(B, ell, nsub, accL, accR, ctrl, slots, rdone, err, vL, vR, accept, &last);
}

// decode_verify_masked for small problems, by a few workgroups (at most 8):
// thread g of the grid (g = 1024 * workgroup + thread) takes the outputs
// i = g + 1024 G u of every column (Y_b[i] = Yhat_b[i] - My_b[i] and the v_R
// terms R_q[i] Yhat_b[i]) and the inputs k = g + 1024 G u (the v_L terms
// U_q[k] Xhat_b[k]), PER of each per pass with all of a pass's loads issued
// before the first is used (addresses clamped in range, terms masked).  The
// 2 * ell partial sums of a column are reduced across the waves in LDS; with
// one workgroup the results follow directly, with several each adds its sums
// into 64-bit accumulators and the last one to finish (counter) compares.
// ell <= EL.
constexpr int kSmallThreads = 1024;
template <int EL, int PER>
__device__ __forceinline__ void dv_small_body(
    uint32_t bid, uint32_t G, uint32_t m, uint32_t n, const uint32_t* __restrict__ Xhat,
    const uint32_t* __restrict__ Yhat, uint32_t B, const uint32_t* __restrict__ My, uint32_t ell,
    const uint32_t* __restrict__ R, const uint32_t* __restrict__ U, uint32_t* __restrict__ Y,
    unsigned long long* acc, uint32_t* counter, uint32_t* __restrict__ vL, uint32_t* __restrict__ vR,
    uint32_t* __restrict__ accept) {
    constexpr int NW = kSmallThreads / 64;
    __shared__ uint64_t red[NW][2 * EL];
    __shared__ uint32_t fin[2 * EL];
    __shared__ uint32_t last;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t gt = bid * kSmallThreads + (uint32_t)tid;
    const uint32_t stride = G * kSmallThreads, pass = stride * PER;
    const uint32_t len = m > n ? m : n;
    for (uint32_t b = 0; b < B; ++b) {
        uint64_t l[EL], rr[EL];
#pragma unroll
        for (int q = 0; q < EL; ++q) l[q] = rr[q] = 0;
        for (uint32_t base = 0; base < len; base += pass) {
            uint32_t yv[PER], mv[PER], xv[PER], rv[EL][PER], uv[EL][PER];
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                const uint32_t j = base + gt + stride * u;
                const uint32_t i = j < m ? j : m - 1, k = j < n ? j : n - 1;
                yv[u] = Yhat[(size_t)b * m + i];
                mv[u] = My[(size_t)b * m + i];
                xv[u] = Xhat[(size_t)b * n + k];
#pragma unroll
                for (int q = 0; q < EL; ++q) {
                    const uint32_t qs = (uint32_t)q < ell ? (uint32_t)q : 0u;
                    rv[q][u] = R[(size_t)qs * m + i];
                    uv[q][u] = U[(size_t)qs * n + k];
                }
            }
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                const uint32_t j = base + gt + stride * u;
                // the value is pinned in a register before the guarded store, so
                // that the compiler does not sink the loads into the branch (where
                // each would wait on its own)
                uint32_t yo = fsub(yv[u], mv[u]);
                asm volatile("" : "+v"(yo));
                if (j < m) Y[(size_t)b * m + j] = yo;
                const uint32_t y = j < m ? yv[u] : 0u, x = j < n ? xv[u] : 0u;
#pragma unroll
                for (int q = 0; q < EL; ++q) {
                    rr[q] += ffold((uint64_t)rv[q][u] * y);
                    l[q] += ffold((uint64_t)uv[q][u] * x);
                }
            }
        }
#pragma unroll
        for (int q = 0; q < EL; ++q) {
            if ((uint32_t)q < ell) {
                const uint64_t sl = wave_sum_u64(l[q]), sr = wave_sum_u64(rr[q]);
                if (lane == 0) {
                    red[wave][2 * q] = sl;
                    red[wave][2 * q + 1] = sr;
                }
            }
        }
        __syncthreads();
        if ((uint32_t)tid < 2 * ell) {
            uint64_t tot = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) tot += red[w][tid];
            if (G == 1)
                fin[tid] = fred64(tot);
            else
                atomicAdd(&acc[(size_t)b * 2 * ell + tid], (unsigned long long)fred64(tot));
        }
        __syncthreads();
        if (G == 1) {
            if ((uint32_t)tid < ell) {
                if (vL) vL[(size_t)tid * B + b] = fin[2 * tid];
                if (vR) vR[(size_t)tid * B + b] = fin[2 * tid + 1];
            }
            if (tid == 0) {
                uint32_t ok = 1;
                for (uint32_t q = 0; q < ell; ++q) ok &= fin[2 * q] == fin[2 * q + 1] ? 1u : 0u;
                accept[b] = ok;
            }
            __syncthreads();  // fin is reused by the next column
        }
    }
    if (G == 1) return;
    // several workgroups: the last one to finish reads and clears the
    // accumulators (ordering as in decode_verify_fused)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) last = (atomicAdd(counter, 1u) == G - 1) ? 1u : 0u;
    __syncthreads();
    if (!last) return;
    for (uint32_t b = tid; b < B; b += kSmallThreads) {
        uint32_t ok = 1;
        for (uint32_t q = 0; q < ell; ++q) {
            const uint32_t L = fred64(atomicExch(&acc[(size_t)b * 2 * ell + 2 * q], 0ull));
            const uint32_t Rr = fred64(atomicExch(&acc[(size_t)b * 2 * ell + 2 * q + 1], 0ull));
            if (vL) vL[(size_t)q * B + b] = L;
            if (vR) vR[(size_t)q * B + b] = Rr;
            ok &= (L == Rr) ? 1u : 0u;
        }
        accept[b] = ok;
    }
    if (tid == 0) atomicExch(counter, 0u);
}

template <int EL, int PER>
__global__ __launch_bounds__(kSmallThreads) void decode_verify_small(
    uint32_t m, uint32_t n, const uint32_t* __restrict__ Xhat, const uint32_t* __restrict__ Yhat, uint32_t B,
    const uint32_t* __restrict__ My, uint32_t ell, const uint32_t* __restrict__ R, const uint32_t* __restrict__ U,
    uint32_t* __restrict__ Y, unsigned long long* acc, uint32_t* counter, uint32_t* __restrict__ vL,
    uint32_t* __restrict__ vR, uint32_t* __restrict__ accept) {
    dv_small_body<EL, PER>(blockIdx.x, gridDim.x, m, n, Xhat, Yhat, B, My, ell, R, U, Y, acc, counter, vL, vR,
                           accept);
}

// One client turn between two server calls of independent queries: the
// decode/verify of one response (dv_small_body, workgroups [0, Gd)) and the
// masked encode of the next query (add_masks_body, the other workgroups, with
// the optional wait for its preparation's flag) in one launch.  The two roles
// share no data.
template <int EL, int PER, bool WAIT, int APER>
__global__ __launch_bounds__(kSmallThreads) void client_turn(
    uint32_t Gd, uint32_t m, uint32_t n, const uint32_t* __restrict__ Xhat, const uint32_t* __restrict__ Yhat,
    uint32_t B, const uint32_t* __restrict__ My, uint32_t ell, const uint32_t* __restrict__ R,
    const uint32_t* __restrict__ U, uint32_t* __restrict__ Y, unsigned long long* acc, uint32_t* counter,
    uint32_t* __restrict__ vL, uint32_t* __restrict__ vR, uint32_t* __restrict__ accept, const uint32_t* Xn,
    const uint32_t* __restrict__ Mxn, size_t countn, uint32_t* Xhatn, uint32_t* flag, uint32_t value,
    uint64_t ticks, uint32_t* timed_out, uint32_t* add_counter) {
    static_assert(kSmallThreads == kAddThreads, "the two roles run in workgroups of one size");
    if (blockIdx.x < Gd)
        dv_small_body<EL, PER>(blockIdx.x, Gd, m, n, Xhat, Yhat, B, My, ell, R, U, Y, acc, counter, vL, vR, accept);
    else
        add_masks_body<WAIT, APER>(blockIdx.x - Gd, gridDim.x - Gd, Xn, Mxn, countn, Xhatn, flag, value, ticks,
                                timed_out, add_counter);
}

// Transpose-reduction mod p of V values per lane over the 64 lanes of a wave:
// each step sends half of the live values to the partner lane and keeps the
// other half, so V - 1 + 6 - log2 V exchanges in all.  Afterwards lane L holds
// the wave-wide sum of value index L >> (6 - log2 V).
template <int V>
__device__ __forceinline__ uint32_t wave_xreduce_mod(uint32_t (&a)[V], int lane) {
    constexpr int LOGV = (V == 64) ? 6 : (V == 32) ? 5 : (V == 16) ? 4 : (V == 8) ? 3 : -1;
    static_assert(LOGV > 0, "V must be 8, 16, 32 or 64");
#pragma unroll
    for (int step = 0; step < LOGV; ++step) {
        const int s = 32 >> step;
        const int half = V >> (step + 1);
        const bool up = (lane & s) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
            // the two values pinned in registers: otherwise the compiler turns
            // the pair of selects into a select of the array index, which it
            // then expands into compare-and-select chains over the whole array
            uint32_t lo = a[i], hi = a[i + half];
            asm volatile("" : "+v"(lo), "+v"(hi));
            const uint32_t send = up ? lo : hi;
            const uint32_t keep = up ? hi : lo;
            a[i] = fadd(keep, (uint32_t)__shfl_xor((int)send, s));
        }
    }
    uint32_t v = a[0];
#pragma unroll
    for (int s = 32 >> LOGV; s >= 1; s >>= 1) v = fadd(v, (uint32_t)__shfl_xor((int)v, s));
    return v;
}

// decode_verify_masked for larger problems (ell <= EL): workgroup (element
// block eb, column group) takes the elements j = 256 PER eb + t + 256 u
// (u < PER) of thread t, as outputs i (Y_b[i] = Yhat_b[i] - My_b[i] and the
// v_R terms R_q[i] Yhat_b[i]) and as inputs k (the v_L terms U_q[k]
// Xhat_b[k]), for C columns b; every load of the workgroup is issued before
// the first is used (addresses clamped in range, terms masked).  Per thread
// the 2 EL C sums are reduced mod p, across the wave by a transpose-reduction
// and across the waves in LDS, and added into the accumulators (sum of column
// b, repetition q: nsub of them, used by element block mod nsub); the last
// workgroup (count.h) compares.  The host picks PER and C so that the grid
// has a few hundred workgroups where the problem allows.
//
// A launch may cover G <= kMaxGroup problems that share the queries Xhat
// (several matrices applied to one input): problem g = blockIdx.y has its own
// responses, masks, challenge vectors and outputs (DvGroup) and its own
// control region, ctrl + g * ctrl_stride words.
constexpr int kWideThreads = 256;
struct DvGroup {
    const uint32_t* Yhat[kMaxGroup];
    const uint32_t* My[kMaxGroup];
    const uint32_t* R[kMaxGroup];
    const uint32_t* U[kMaxGroup];
    uint32_t* Y[kMaxGroup];
    uint32_t* vL[kMaxGroup];
    uint32_t* vR[kMaxGroup];
    uint32_t* accept[kMaxGroup];
};
template <int EL, int C, int PER>
__global__ __launch_bounds__(kWideThreads) void decode_verify_wide(
    uint32_t m, uint32_t n, const uint32_t* __restrict__ Xhat, uint32_t B, uint32_t ell, const DvGroup grp,
    size_t acc_word, uint32_t nsub, uint32_t neb, uint32_t* ctrl0, size_t ctrl_stride, uint32_t slots) {
    constexpr int NW = kWideThreads / 64, V = 2 * EL * C;
    constexpr int kWidePer = PER;
    constexpr uint32_t kWideElems = kWideThreads * PER;
    __shared__ uint32_t red[NW][V];
    __shared__ uint32_t last;
    const uint32_t g = blockIdx.y;
    const uint32_t* __restrict__ Yhat = grp.Yhat[g];
    const uint32_t* __restrict__ My = grp.My[g];
    const uint32_t* __restrict__ R = grp.R[g];
    const uint32_t* __restrict__ U = grp.U[g];
    uint32_t* __restrict__ Y = grp.Y[g];
    uint32_t* ctrl = ctrl0 + g * ctrl_stride;
    unsigned long long* accL = reinterpret_cast<unsigned long long*>(ctrl + acc_word);
    unsigned long long* accR = accL + (size_t)ell * B * nsub;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t eb = blockIdx.x % neb, b0 = (blockIdx.x / neb) * C;
    const uint32_t base = eb * kWideElems + (uint32_t)tid;
    uint32_t rv[EL][kWidePer], uv[EL][kWidePer], yv[C][kWidePer], mv[C][kWidePer], xv[C][kWidePer];
#pragma unroll
    for (int u = 0; u < kWidePer; ++u) {
        const uint32_t j = base + kWideThreads * u;
        const uint32_t i = j < m ? j : m - 1, k = j < n ? j : n - 1;
#pragma unroll
        for (int q = 0; q < EL; ++q) {
            const uint32_t qs = (uint32_t)q < ell ? (uint32_t)q : 0u;
            rv[q][u] = R[(size_t)qs * m + i];
            uv[q][u] = U[(size_t)qs * n + k];
        }
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const uint32_t b = b0 + c < B ? b0 + c : B - 1;
            yv[c][u] = Yhat[(size_t)b * m + i];
            mv[c][u] = My[(size_t)b * m + i];
            xv[c][u] = Xhat[(size_t)b * n + k];
        }
    }
    uint32_t a[V];  // index (c * EL + q) * 2 + side; side 0: v_L, 1: v_R
#pragma unroll
    for (int c = 0; c < C; ++c) {
        uint64_t l[EL], r[EL];
#pragma unroll
        for (int q = 0; q < EL; ++q) l[q] = r[q] = 0;
#pragma unroll
        for (int u = 0; u < kWidePer; ++u) {
            const uint32_t j = base + kWideThreads * u;
            // pinned before the guarded store (see decode_verify_small)
            uint32_t yo = fsub(yv[c][u], mv[c][u]);
            asm volatile("" : "+v"(yo));
            if (j < m && b0 + c < B) Y[(size_t)(b0 + c) * m + j] = yo;
            const uint32_t y = j < m ? yv[c][u] : 0u, x = j < n ? xv[c][u] : 0u;
#pragma unroll
            for (int q = 0; q < EL; ++q) {
                r[q] += ffold((uint64_t)rv[q][u] * y);
                l[q] += ffold((uint64_t)uv[q][u] * x);
            }
        }
#pragma unroll
        for (int q = 0; q < EL; ++q) {
            a[(c * EL + q) * 2] = fred64(l[q]);
            a[(c * EL + q) * 2 + 1] = fred64(r[q]);
        }
    }
    const uint32_t w = wave_xreduce_mod<V>(a, lane);
    constexpr int SH = (V == 64) ? 0 : (V == 32) ? 1 : (V == 16) ? 2 : 3;
    if ((lane & ((1 << SH) - 1)) == 0) red[wave][lane >> SH] = w;
    __syncthreads();
    if (tid < V) {
        uint32_t tot = 0;
#pragma unroll
        for (int h = 0; h < NW; ++h) tot = fadd(tot, red[h][tid]);
        const uint32_t side = (uint32_t)tid & 1u, q = ((uint32_t)tid >> 1) % EL, c = ((uint32_t)tid >> 1) / EL;
        if (q < ell && b0 + c < B) {
            unsigned long long* acc = side ? accR : accL;
            atomicAdd(&acc[((size_t)q * B + b0 + c) * nsub + eb % nsub], (unsigned long long)tot);
        }
    }
    finish(B, ell, nsub, accL, accR, ctrl, slots, nullptr, nullptr, grp.vL[g], grp.vR[g], grp.accept[g], &last);
}

// decode_verify_masked with one workgroup per query column (and problem of
// the group: grid B x G): 1024 threads take the elements j = t + 1024 u of
// their column, as outputs i (Y_b[i] = Yhat_b[i] - My_b[i] and the v_R terms
// R_q[i] Yhat_b[i]) and as inputs k (the v_L terms U_q[k] Xhat_b[k]), PER
// per pass with all of a pass's loads issued before the first is used
// (addresses clamped in range, terms masked); the 2 ell sums are reduced
// across the wave and through LDS, and the workgroup writes v_L, v_R and
// accept of its column itself: no atomics and no completion count.  ell <= EL.
template <int EL, int PER>
__global__ __launch_bounds__(kSmallThreads) void decode_verify_col(uint32_t m, uint32_t n,
                                                                   const uint32_t* __restrict__ Xhat, uint32_t B,
                                                                   uint32_t ell, const DvGroup grp) {
    constexpr int NW = kSmallThreads / 64;
    __shared__ uint64_t red[NW][2 * EL];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t b = blockIdx.x, g = blockIdx.y;
    const uint32_t* __restrict__ Yhat = grp.Yhat[g] + (size_t)b * m;
    const uint32_t* __restrict__ My = grp.My[g] + (size_t)b * m;
    const uint32_t* __restrict__ R = grp.R[g];
    const uint32_t* __restrict__ U = grp.U[g];
    const uint32_t* __restrict__ xh = Xhat + (size_t)b * n;
    uint32_t* __restrict__ Y = grp.Y[g] + (size_t)b * m;
    const uint32_t len = m > n ? m : n;
    constexpr uint32_t pass = kSmallThreads * PER;
    uint64_t l[EL], rr[EL];
#pragma unroll
    for (int q = 0; q < EL; ++q) l[q] = rr[q] = 0;
    for (uint32_t base = 0; base < len; base += pass) {
        uint32_t yv[PER], mv[PER], xv[PER], rv[EL][PER], uv[EL][PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const uint32_t j = base + (uint32_t)tid + kSmallThreads * u;
            const uint32_t i = j < m ? j : m - 1, k = j < n ? j : n - 1;
            yv[u] = Yhat[i];
            mv[u] = My[i];
            xv[u] = xh[k];
#pragma unroll
            for (int q = 0; q < EL; ++q) {
                const uint32_t qs = (uint32_t)q < ell ? (uint32_t)q : 0u;
                rv[q][u] = R[(size_t)qs * m + i];
                uv[q][u] = U[(size_t)qs * n + k];
            }
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const uint32_t j = base + (uint32_t)tid + kSmallThreads * u;
            // pinned before the guarded store (see decode_verify_small)
            uint32_t yo = fsub(yv[u], mv[u]);
            asm volatile("" : "+v"(yo));
            if (j < m) Y[j] = yo;
            const uint32_t y = j < m ? yv[u] : 0u, x = j < n ? xv[u] : 0u;
#pragma unroll
            for (int q = 0; q < EL; ++q) {
                rr[q] += ffold((uint64_t)rv[q][u] * y);
                l[q] += ffold((uint64_t)uv[q][u] * x);
            }
        }
    }
#pragma unroll
    for (int q = 0; q < EL; ++q) {
        const uint64_t sl = wave_sum_u64(fred64(l[q])), sr = wave_sum_u64(fred64(rr[q]));
        if (lane == 0) {
            red[wave][2 * q] = sl;
            red[wave][2 * q + 1] = sr;
        }
    }
    __syncthreads();
    if (tid < 64) {
        // lane 2q: v_L of repetition q, lane 2q + 1: v_R
        uint64_t tot = 0;
        if (tid < 2 * EL)
#pragma unroll
            for (int w = 0; w < NW; ++w) tot += red[w][tid];
        const uint32_t v = fred64(tot);
        const uint32_t other = (uint32_t)__shfl_xor((int)v, 1);
        const uint32_t q = (uint32_t)tid >> 1;
        const bool mine = q < ell && tid < 2 * EL;
        if (mine && (tid & 1) == 0 && grp.vL[g]) grp.vL[g][(size_t)q * B + b] = v;
        if (mine && (tid & 1) == 1 && grp.vR[g]) grp.vR[g][(size_t)q * B + b] = v;
        // accept: every repetition's v_L equals its v_R
        const bool bad = mine && (tid & 1) == 0 && v != other;
        const bool any_bad = __ballot(bad) != 0;
        if (tid == 0) grp.accept[g][b] = any_bad ? 0u : 1u;
    }
}

// decode_verify_masked for up to CB <= 8 query columns, spread over the chip
// (grid S x G, problem g = blockIdx.y): workgroup s takes the elements
// j = 256 PER s + t + 256 u (u < PER) of thread t for every column at once,
// so that the challenge vectors r_q and u_q of a segment are read once for
// all columns: as outputs i (Y_b[i] = Yhat_b[i] - My_b[i] and the v_R terms
// R_q[i] Yhat_b[i]) and as inputs k (the v_L terms U_q[k] Xhat_b[k]); every
// load of the workgroup is issued before the first is used (addresses
// clamped in range, terms masked).  The 2 EL CB sums are reduced mod p across
// the wave (transpose-reduction) and the waves (LDS) and added into the
// workgroup's own slot of the control region (no two workgroups share an
// address, so the device atomics do not queue behind each other); the last
// of the S workgroups of the problem (count.h) reads and clears every slot,
// sums them and writes v_L, v_R and accept.
constexpr uint32_t kSegMaxB = 8, kSegMaxLen = 65536, kSegMaxSlots = 64, kSegSlotWords = 64;
template <int EL, int CB, int PER>
__global__ __launch_bounds__(kWideThreads) void decode_verify_seg(uint32_t m, uint32_t n,
                                                                  const uint32_t* __restrict__ Xhat, uint32_t B,
                                                                  uint32_t ell, const DvGroup grp, size_t part_word,
                                                                  uint32_t* ctrl0, size_t ctrl_stride) {
    constexpr int NW = kWideThreads / 64, V = 2 * EL * CB, TPV = kWideThreads / V;
    static_assert(V <= 64, "one wave compares");
    __shared__ uint32_t red[NW][V];
    __shared__ uint32_t fin[TPV][V];
    __shared__ uint32_t last;
    const uint32_t g = blockIdx.y;
    const uint32_t* __restrict__ Yhat = grp.Yhat[g];
    const uint32_t* __restrict__ My = grp.My[g];
    const uint32_t* __restrict__ R = grp.R[g];
    const uint32_t* __restrict__ U = grp.U[g];
    uint32_t* __restrict__ Y = grp.Y[g];
    uint32_t* ctrl = ctrl0 + g * ctrl_stride;
    uint32_t* part = ctrl + part_word;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t base = blockIdx.x * (uint32_t)(kWideThreads * PER) + (uint32_t)tid;
    uint32_t rv[EL][PER], uv[EL][PER], yv[CB][PER], mv[CB][PER], xv[CB][PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const uint32_t j = base + kWideThreads * u;
        const uint32_t i = j < m ? j : m - 1, k = j < n ? j : n - 1;
#pragma unroll
        for (int q = 0; q < EL; ++q) {
            const uint32_t qs = (uint32_t)q < ell ? (uint32_t)q : 0u;
            rv[q][u] = R[(size_t)qs * m + i];
            uv[q][u] = U[(size_t)qs * n + k];
        }
#pragma unroll
        for (int c = 0; c < CB; ++c) {
            const uint32_t b = (uint32_t)c < B ? (uint32_t)c : B - 1;
            yv[c][u] = Yhat[(size_t)b * m + i];
            mv[c][u] = My[(size_t)b * m + i];
            xv[c][u] = Xhat[(size_t)b * n + k];
        }
    }
    uint32_t a[V];  // index (c * EL + q) * 2 + side; side 0: v_L, 1: v_R
#pragma unroll
    for (int c = 0; c < CB; ++c) {
        uint64_t l[EL], r[EL];
#pragma unroll
        for (int q = 0; q < EL; ++q) l[q] = r[q] = 0;
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const uint32_t j = base + kWideThreads * u;
            // pinned before the guarded store (see decode_verify_small)
            uint32_t yo = fsub(yv[c][u], mv[c][u]);
            asm volatile("" : "+v"(yo));
            if (j < m && (uint32_t)c < B) Y[(size_t)c * m + j] = yo;
            const uint32_t y = j < m ? yv[c][u] : 0u, x = j < n ? xv[c][u] : 0u;
#pragma unroll
            for (int q = 0; q < EL; ++q) {
                r[q] += ffold((uint64_t)rv[q][u] * y);
                l[q] += ffold((uint64_t)uv[q][u] * x);
            }
        }
#pragma unroll
        for (int q = 0; q < EL; ++q) {
            a[(c * EL + q) * 2] = fred64(l[q]);
            a[(c * EL + q) * 2 + 1] = fred64(r[q]);
        }
    }
    const uint32_t w = wave_xreduce_mod<V>(a, lane);
    constexpr int SH = (V == 64) ? 0 : (V == 32) ? 1 : (V == 16) ? 2 : 3;
    if ((lane & ((1 << SH) - 1)) == 0) red[wave][lane >> SH] = w;
    __syncthreads();
    if (tid < V) {
        uint32_t tot = 0;
#pragma unroll
        for (int h = 0; h < NW; ++h) tot = fadd(tot, red[h][tid]);
        atomicAdd(&part[(size_t)blockIdx.x * kSegSlotWords + tid], tot);  // a zero word before
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) last = count_last(ctrl, 0u) ? 1u : 0u;
    __syncthreads();
    if (!last) return;
    // the last workgroup: TPV threads per value read and clear the slots
    const uint32_t v = (uint32_t)tid % V, h = (uint32_t)tid / V;
    uint32_t sum = 0;
    for (uint32_t s2 = h; s2 < gridDim.x; s2 += TPV)
        sum = fadd(sum, atomicExch(&part[(size_t)s2 * kSegSlotWords + v], 0u));
    fin[h][v] = sum;
    __syncthreads();
    if (tid < 64) {
        uint32_t val = 0;
        if (tid < V)
#pragma unroll
            for (int h2 = 0; h2 < TPV; ++h2) val = fadd(val, fin[h2][tid]);
        const uint32_t other = (uint32_t)__shfl_xor((int)val, 1);
        const uint32_t side = (uint32_t)tid & 1u, q = ((uint32_t)tid >> 1) % EL, c = ((uint32_t)tid >> 1) / EL;
        const bool valid = tid < V && q < ell && c < B;
        if (valid && side == 0 && grp.vL[g]) grp.vL[g][(size_t)q * B + c] = val;
        if (valid && side == 1 && grp.vR[g]) grp.vR[g][(size_t)q * B + c] = val;
        // accept of column c: every repetition's v_L equals its v_R
        const uint64_t bad = __ballot(valid && side == 0 && val != other);
        if (tid < V && (uint32_t)tid % (2 * EL) == 0 && c < B)
            grp.accept[g][c] = ((bad >> tid) & ((1ull << (2 * EL)) - 1)) == 0 ? 1u : 0u;
    }
}

template <int U, int E>
int fused_blocks_per_cu() {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, decode_verify_syn<U, E>, kFusedThreads, 0) != hipSuccess)
        return 0;
    return nb;
}

}  // namespace

namespace {
// Control region of a decode/verify launch: the counters (count.h; rdone and
// err in words 1 and 2 of the top counter's line), then the accumulators,
// 2 x ell x B x nsub 64-bit words.  Sized for the largest grid of the three
// kernels, so that one layout serves every call with the same (m, n, B, ell).
struct DvLayout {
    uint32_t slots, nsub;
    size_t acc_word;  // first accumulator, in 32-bit words from ctrl
    size_t bytes;
};

DvLayout dv_layout(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) {
    const uint32_t nblkL = ceil_div(n, kCols), nblkR = ceil_div(m, kCols);
    // the largest grid: decode_verify_syn, or decode_verify_wide with one
    // element per thread and one column per workgroup
    const uint64_t g_fused = (uint64_t)B * nblkR + nblkL + ell;
    const uint64_t g_wide = (uint64_t)ceil_div(m > n ? m : n, (uint32_t)kWideThreads) * B;
    const uint64_t grid = g_fused > g_wide ? g_fused : g_wide;
    DvLayout l;
    l.slots = count_slots(grid > 0xffffffffull ? 0xffffffffu : (uint32_t)grid);
    // workgroups per accumulator address: at most ~32
    const uint32_t per = nblkR > nblkL ? nblkR : nblkL;
    l.nsub = per <= 32 ? 1u : (per >= 8 * 32 ? 8u : ceil_div(per, 32u));
    l.acc_word = count_words(l.slots);
    l.bytes = l.acc_word * 4 + (size_t)2 * ell * B * l.nsub * 8;
    // decode_verify_seg's slots in the same place
    const size_t seg = l.acc_word * 4 + (size_t)kSegMaxSlots * kSegSlotWords * 4;
    l.bytes = seg > l.bytes ? seg : l.bytes;
    return l;
}
}  // namespace

size_t dv_ctrl_bytes(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) { return dv_layout(m, n, B, ell).bytes; }

uint32_t dv_decode_cols(uint32_t m, uint32_t B, const void* PT, const void* Yhat, const void* Y, const void* r) {
    // Four columns per lane take a quarter of the workgroups: only when those
    // still fill the chip (measured: B = 1 at m = 4096 slows down from 24 to
    // 28 us with four, 16 columns at m = 11008 speed up).
    if (m % 4 != 0 || (uint64_t)B * ceil_div(m, kCols * 4) < 256) return 1u;
    for (const void* p : {PT, Yhat, Y, r})
        if ((uintptr_t)p & 15) return 1u;
    return 4u;
}

uint32_t dv_syn_u(uint32_t Ny) {
    for (uint32_t U : {8u, 16u, 24u, 32u})
        if (Ny <= (uint32_t)kFusedThreads * U) return U;
    return 0;
}

bool dv_syn_fits(uint32_t m, uint32_t n, uint32_t Ny, uint32_t B, uint32_t ell, uint32_t E) {
    const uint32_t U = dv_syn_u(Ny);
    if (U == 0 || ell == 0 || ell > (uint32_t)kMaxEll || Ny == 0 || (E != 1 && E != 4)) return false;
    // residency of one workgroup per CU at least, per device, U and E (cached)
    constexpr int kMaxDevices = 64;
    static int cache[kMaxDevices][4][2];  // blocks per CU x CUs, plus one; 0 = not yet known
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return false;
    const int ui = (int)U / 8 - 1, ei = E == 4 ? 1 : 0;
    if (cache[dev][ui][ei] == 0) {
        int ncu = 0;
        if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return false;
        int nb = 0;
        if (E == 4)
            nb = U == 8 ? fused_blocks_per_cu<8, 4>() : U == 16 ? fused_blocks_per_cu<16, 4>()
               : U == 24 ? fused_blocks_per_cu<24, 4>() : fused_blocks_per_cu<32, 4>();
        else
            nb = U == 8 ? fused_blocks_per_cu<8, 1>() : U == 16 ? fused_blocks_per_cu<16, 1>()
               : U == 24 ? fused_blocks_per_cu<24, 1>() : fused_blocks_per_cu<32, 1>();
        cache[dev][ui][ei] = nb * ncu + 1;
    }
    const uint64_t grid = (uint64_t)ell + ceil_div(n, kCols) + (uint64_t)B * ceil_div(m, kCols * E);
    return grid <= (uint64_t)(cache[dev][ui][ei] - 1);
}

hipError_t launch_decode_verify_syn(const uint32_t* PT, const uint32_t* Q, uint32_t m, uint32_t n, uint32_t Nx,
                                    uint32_t Ny, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                    const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx,
                                    const uint32_t* ey_idx, const uint32_t* ey_val, uint32_t ty, uint32_t ell,
                                    uint32_t cyr, const uint32_t* pi1, const uint32_t* pi2, const uint32_t* v1,
                                    const uint32_t* v2, uint32_t* r, uint32_t* Y, uint32_t* ctrl, uint32_t* vL,
                                    uint32_t* vR, uint32_t* accept, hipStream_t s) {
    const uint32_t U = dv_syn_u(Ny);
    if (U == 0 || ell == 0 || ell > (uint32_t)kMaxEll || (uint64_t)cyr * m != Ny) return hipErrorInvalidValue;
    const uint32_t E = dv_decode_cols(m, B, PT, Yhat, Y, r);
    const uint32_t nblkL = ceil_div(n, kCols), nblkR = ceil_div(m, kCols * E);
    const uint32_t grid = ell + nblkL + B * nblkR;
    const DvLayout l = dv_layout(m, n, B, ell);
    unsigned long long* acc = reinterpret_cast<unsigned long long*>(ctrl + l.acc_word);
    const uint32_t slots = count_slots(grid);
#define MVK_DVS(UU, EE)                                                                                           \
    hipLaunchKernelGGL((decode_verify_syn<UU, EE>), dim3(grid), dim3(kFusedThreads), 0, s, PT, Q, m, n, Nx, Ny,   \
                       Xhat, Yhat, B, ex_idx, ex_val, tx, ey_idx, ey_val, ty, ell, cyr, pi1, pi2, v1, v2, r, Y,    \
                       acc, acc + (size_t)ell * B * l.nsub, l.nsub, nblkR, nblkL, ctrl, slots, vL, vR, accept)
#define MVK_DVS_E(UU) \
    if (E == 4) MVK_DVS(UU, 4); else MVK_DVS(UU, 1)
    if (U == 8) { MVK_DVS_E(8); }
    else if (U == 16) { MVK_DVS_E(16); }
    else if (U == 24) { MVK_DVS_E(24); }
    else { MVK_DVS_E(32); }
#undef MVK_DVS_E
#undef MVK_DVS
    return hipGetLastError();
}

hipError_t launch_decode_verify(const uint32_t* PT, const uint32_t* Q, uint32_t m, uint32_t n, uint32_t Nx,
                                uint32_t Ny, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx, const uint32_t* ey_idx,
                                const uint32_t* ey_val, uint32_t ty, uint32_t ell, const uint32_t* r, uint32_t* Y,
                                uint32_t* ctrl, uint32_t* vL, uint32_t* vR, uint32_t* accept, hipStream_t s) {
    if (ell == 0 || ell > (uint32_t)kMaxEll) return hipErrorInvalidValue;
    const uint32_t E = dv_decode_cols(m, B, PT, Yhat, Y, r);
    const uint32_t nblkL = ceil_div(n, kCols), nblkR = ceil_div(m, kCols * E);
    const uint32_t grid = B * nblkR + nblkL;
    const DvLayout l = dv_layout(m, n, B, ell);
    unsigned long long* acc = reinterpret_cast<unsigned long long*>(ctrl + l.acc_word);
#define MVK_DVF(EE)                                                                                                \
    hipLaunchKernelGGL((decode_verify_fused<false, EE>), dim3(grid), dim3(kB), 0, s, PT, Q, m, n, Nx, Ny, Xhat,    \
                       Yhat, B, ex_idx, ex_val, tx, ey_idx, ey_val, ty, ell, r, Y, acc,                            \
                       acc + (size_t)ell * B * l.nsub, l.nsub, nblkR, ctrl, count_slots(grid), vL, vR, accept,     \
                       nullptr, nullptr)
    if (E == 4) MVK_DVF(4); else MVK_DVF(1);
#undef MVK_DVF
    return hipGetLastError();
}

namespace {
// The decode_verify_wide configuration for a problem (ell <= 4): element
// blocks x column groups, all loads of a workgroup in flight together: 4
// elements per thread and 16 / EL columns per workgroup, or (grids below 256
// workgroups) 1 element and 4 / EL columns.
struct WideShape {
    uint32_t el, per, cols, neb;
    uint64_t grid;
};
WideShape wide_shape(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) {
    const uint32_t len = m > n ? m : n;
    const uint32_t el = ell <= 2 ? 2u : 4u;
    const bool wide = (uint64_t)ceil_div(len, 4u * kWideThreads) * ceil_div(B, 16u / el) >= 256u;
    WideShape w;
    w.el = el;
    w.per = wide ? 4u : 1u;
    w.cols = wide ? 16u / el : 4u / el;
    w.neb = ceil_div(len, w.per * kWideThreads);
    w.grid = (uint64_t)w.neb * ceil_div(B, w.cols);
    return w;
}

bool takes_small(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) {
    return (uint64_t)B * ((uint64_t)m + n) <= kSmallDvWords && ell <= 4;
}

// One workgroup per column (decode_verify_col) from kColsMinB columns up to
// kColsMaxLen elements per column, ell <= 4: every column's sums stay in its
// workgroup.
constexpr uint32_t kColsMinB = 2, kColsMaxLen = 65536, kColsMaxB = 65535;
bool takes_cols(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) {
    const uint32_t len = m > n ? m : n;
    return ell <= 4 && B >= kColsMinB && B <= kColsMaxB && len <= kColsMaxLen && !takes_small(m, n, B, ell);
}

// decode_verify_seg above the length one workgroup per column takes in one
// pass (4096) up to kSegMaxLen elements, above the one-workgroup size: 1 to
// kSegMaxB columns with ell <= 2, 1 to 4 with ell <= 4 (64 sums per thread
// would spill).  The elements per thread (1, 2 or 4) keep a problem's
// segments at 32 or fewer where the length allows.  (Eight columns: 7.0 us
// against 7.5 for one workgroup per column at 4096 x 11008, 7.1 against 7.9
// for two problems at 11008 x 4096; at 4096 x 4096 5.8 against 5.1.)
bool takes_seg(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) {
    const uint32_t len = m > n ? m : n;
    return ell >= 1 && ell <= 4 && B >= 1 && B <= (ell <= 2 ? kSegMaxB : kSegMaxB / 2) &&
           len > 4u * kSmallThreads && len <= kSegMaxLen && !takes_small(m, n, B, ell);
}

hipError_t launch_seg(uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B, uint32_t ell, const DvGroup& grp,
                      uint32_t G, uint32_t* ctrl, size_t ctrl_stride, hipStream_t s) {
    const DvLayout l = dv_layout(m, n, B, ell);
    const uint32_t len = m > n ? m : n;
    uint32_t per = 1;
    while (per < 4 && ceil_div(len, per * (uint32_t)kWideThreads) > 32) per *= 2;
    const uint32_t S = ceil_div(len, per * (uint32_t)kWideThreads);
    if (S > kSegMaxSlots || count_words(0) > l.acc_word ||
        (size_t)S * kSegSlotWords * 4 > l.bytes - l.acc_word * 4)
        return hipErrorInvalidValue;  // the layout holds the counter and the slots
    const dim3 grid(S, G);
#define MVK_SEG(EL, CB, PER)                                                                               \
    hipLaunchKernelGGL((decode_verify_seg<EL, CB, PER>), grid, dim3(kWideThreads), 0, s, m, n, Xhat, B, ell, \
                       grp, l.acc_word, ctrl, ctrl_stride)
#define MVK_SEG_PER(EL, CB) \
    if (per == 1) MVK_SEG(EL, CB, 1); else if (per == 2) MVK_SEG(EL, CB, 2); else MVK_SEG(EL, CB, 4)
    if (ell <= 2) {
        if (B <= 2) { MVK_SEG_PER(2, 2); } else if (B <= 4) { MVK_SEG_PER(2, 4); } else { MVK_SEG_PER(2, 8); }
    } else {
        if (B <= 2) { MVK_SEG_PER(4, 2); } else { MVK_SEG_PER(4, 4); }
    }
#undef MVK_SEG_PER
#undef MVK_SEG
    return hipGetLastError();
}

hipError_t launch_cols(uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B, uint32_t ell, const DvGroup& grp,
                       uint32_t G, hipStream_t s) {
    const dim3 grid(B, G);
    if (ell <= 2)
        hipLaunchKernelGGL((decode_verify_col<2, 4>), grid, dim3(kSmallThreads), 0, s, m, n, Xhat, B, ell, grp);
    else
        hipLaunchKernelGGL((decode_verify_col<4, 4>), grid, dim3(kSmallThreads), 0, s, m, n, Xhat, B, ell, grp);
    return hipGetLastError();
}

// decode_verify_wide over G problems (grid.y = G); each control region as
// dv_layout(m, n, B, ell), ctrl_stride words apart.
hipError_t launch_wide(uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B, uint32_t ell, const DvGroup& grp,
                       uint32_t G, uint32_t* ctrl, size_t ctrl_stride, hipStream_t s) {
    const DvLayout l = dv_layout(m, n, B, ell);
    const WideShape w = wide_shape(m, n, B, ell);
    if (w.grid > 0x7fffffffu) return hipErrorInvalidValue;
    const uint32_t slots = count_slots((uint32_t)w.grid);
    if (count_words(slots) > l.acc_word) return hipErrorInvalidValue;  // the layout holds the counters
    const dim3 grid((uint32_t)w.grid, G);
#define MVK_DVW(EL, C, PER)                                                                                 \
    hipLaunchKernelGGL((decode_verify_wide<EL, C, PER>), grid, dim3(kWideThreads), 0, s, m, n, Xhat, B, ell, \
                       grp, l.acc_word, l.nsub, w.neb, ctrl, ctrl_stride, slots)
    if (w.el == 2) {
        if (w.per == 4) MVK_DVW(2, 8, 4); else MVK_DVW(2, 2, 1);
    } else {
        if (w.per == 4) MVK_DVW(4, 4, 4); else MVK_DVW(4, 1, 1);
    }
#undef MVK_DVW
    return hipGetLastError();
}
}  // namespace

hipError_t launch_decode_verify_masked(uint32_t m, uint32_t n, const uint32_t* Xhat, const uint32_t* Yhat,
                                       uint32_t B, const uint32_t* My, uint32_t ell, const uint32_t* r,
                                       const uint32_t* U, uint32_t* Y, uint32_t* ctrl, uint32_t* vL, uint32_t* vR,
                                       uint32_t* accept, hipStream_t s) {
    if (ell == 0 || ell > (uint32_t)kMaxEll) return hipErrorInvalidValue;
    const DvLayout l = dv_layout(m, n, B, ell);
    unsigned long long* acc = reinterpret_cast<unsigned long long*>(ctrl + l.acc_word);
    uint32_t* counter = ctrl;
    if (takes_seg(m, n, B, ell) || takes_cols(m, n, B, ell)) {
        DvGroup grp{};
        grp.Yhat[0] = Yhat;
        grp.My[0] = My;
        grp.R[0] = r;
        grp.U[0] = U;
        grp.Y[0] = Y;
        grp.vL[0] = vL;
        grp.vR[0] = vR;
        grp.accept[0] = accept;
        if (takes_seg(m, n, B, ell)) return launch_seg(m, n, Xhat, B, ell, grp, 1, ctrl, 0, s);
        return launch_cols(m, n, Xhat, B, ell, grp, 1, s);
    }
    if (takes_small(m, n, B, ell)) {
        // four elements per thread, one pass per column: a single workgroup up
        // to 4096 elements (no accumulators or counter), else up to 8.  (One
        // workgroup with all of a column's loads in flight beat four with one
        // element per thread: 15.2 vs 16.3 us per step at 4096 x 4096, B = 1.)
        const uint32_t len = m > n ? m : n;
        uint32_t G = ceil_div(len, 4u * kSmallThreads);
        G = G < 1u ? 1u : (G > 8u ? 8u : G);
#define MVK_DVS(EL)                                                                                          \
    hipLaunchKernelGGL((decode_verify_small<EL, 4>), dim3(G), dim3(kSmallThreads), 0, s, m, n, Xhat, Yhat, B, \
                       My, ell, r, U, Y, acc, counter, vL, vR, accept)
        if (ell <= 2) MVK_DVS(2); else MVK_DVS(4);
#undef MVK_DVS
        return hipGetLastError();
    }
    if (ell <= 4) {
        DvGroup grp{};
        grp.Yhat[0] = Yhat;
        grp.My[0] = My;
        grp.R[0] = r;
        grp.U[0] = U;
        grp.Y[0] = Y;
        grp.vL[0] = vL;
        grp.vR[0] = vR;
        grp.accept[0] = accept;
        return launch_wide(m, n, Xhat, B, ell, grp, 1, ctrl, 0, s);
    }
    const uint32_t nblkL = ceil_div(n, kCols), nblkR = ceil_div(m, kCols);
    const uint32_t grid = B * nblkR + nblkL;
    hipLaunchKernelGGL((decode_verify_fused<true, 1>), dim3(grid), dim3(kB), 0, s, nullptr, nullptr, m, n, 0u, 0u,
                       Xhat, Yhat, B, nullptr, nullptr, 0u, nullptr, nullptr, 0u, ell, r, Y, acc,
                       acc + (size_t)ell * B * l.nsub, l.nsub, nblkR, ctrl, count_slots(grid), vL, vR, accept, My, U);
    return hipGetLastError();
}

hipError_t launch_client_turn(uint32_t m, uint32_t n, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                              const uint32_t* My, uint32_t ell, const uint32_t* r, const uint32_t* U, uint32_t* Y,
                              uint32_t* ctrl, uint32_t* vL, uint32_t* vR, uint32_t* accept, const uint32_t* Xn,
                              const uint32_t* Mxn, size_t countn, uint32_t* Xhatn, uint32_t* flag, uint32_t value,
                              uint32_t timeout_us, uint32_t* timed_out, uint32_t* add_counter, hipStream_t s) {
    if (ell == 0 || ell > (uint32_t)kMaxEll) return hipErrorInvalidValue;
    if (!takes_small(m, n, B, ell) || countn == 0) {
        // larger problems: the two steps as their own launches
        hipError_t e = launch_decode_verify_masked(m, n, Xhat, Yhat, B, My, ell, r, U, Y, ctrl, vL, vR, accept, s);
        if (e == hipSuccess)
            e = launch_add_masks(Xn, Mxn, countn, Xhatn, flag, value, timeout_us, timed_out, add_counter, s);
        return e;
    }
    const DvLayout l = dv_layout(m, n, B, ell);
    unsigned long long* acc = reinterpret_cast<unsigned long long*>(ctrl + l.acc_word);
    // decode/verify workgroups as launch_decode_verify_masked's small form,
    // masked-encode workgroups as launch_add_masks'
    const uint32_t len = m > n ? m : n;
    uint32_t Gd = ceil_div(len, 4u * kSmallThreads);
    Gd = Gd < 1u ? 1u : (Gd > 8u ? 8u : Gd);
    const int aper = add_masks_per(countn);
    size_t Ga = (countn + (size_t)aper * kAddThreads - 1) / ((size_t)aper * kAddThreads);
    Ga = Ga > 256 ? 256 : (Ga == 0 ? 1 : Ga);
    uint64_t ticks = 0;
    if (flag) {
        const hipError_t e = wait_ticks(timeout_us, &ticks);
        if (e != hipSuccess) return e;
    }
    const dim3 grid(Gd + (uint32_t)Ga), block(kSmallThreads);
#define MVK_TURN_A(EL, W, A)                                                                                        \
    hipLaunchKernelGGL((client_turn<EL, 4, W, A>), grid, block, 0, s, Gd, m, n, Xhat, Yhat, B, My, ell, r, U, Y, acc, \
                       ctrl, vL, vR, accept, Xn, Mxn, countn, Xhatn, flag, value, ticks, timed_out, add_counter)
#define MVK_TURN(EL, W) \
    if (aper == 1) MVK_TURN_A(EL, W, 1); else if (aper == 2) MVK_TURN_A(EL, W, 2); else MVK_TURN_A(EL, W, 4)
    if (ell <= 2) {
        if (flag) { MVK_TURN(2, true); } else { MVK_TURN(2, false); }
    } else {
        if (flag) { MVK_TURN(4, true); } else { MVK_TURN(4, false); }
    }
#undef MVK_TURN
#undef MVK_TURN_A
    return hipGetLastError();
}

size_t dv_group_ctrl_stride(uint32_t m, uint32_t n, uint32_t B, uint32_t ell) {
    return (dv_ctrl_bytes(m, n, B, ell) + 255) / 256 * 64;  // words, whole 256-byte lines
}

hipError_t launch_decode_verify_masked_group(uint32_t G, uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B,
                                             const uint32_t* const* Yhat, const uint32_t* const* My, uint32_t ell,
                                             const uint32_t* const* R, const uint32_t* const* U, uint32_t* const* Y,
                                             uint32_t* const* vL, uint32_t* const* vR, uint32_t* const* accept,
                                             uint32_t* ctrl, hipStream_t s) {
    if (G == 0 || G > kMaxGroup || ell == 0 || ell > (uint32_t)kMaxEll) return hipErrorInvalidValue;
    const size_t stride = dv_group_ctrl_stride(m, n, B, ell);
    if (takes_seg(m, n, B, ell) || takes_cols(m, n, B, ell)) {
        DvGroup grp{};
        for (uint32_t g = 0; g < G; ++g) {
            grp.Yhat[g] = Yhat[g];
            grp.My[g] = My[g];
            grp.R[g] = R[g];
            grp.U[g] = U[g];
            grp.Y[g] = Y[g];
            grp.vL[g] = vL ? vL[g] : nullptr;
            grp.vR[g] = vR ? vR[g] : nullptr;
            grp.accept[g] = accept[g];
        }
        if (takes_seg(m, n, B, ell)) return launch_seg(m, n, Xhat, B, ell, grp, G, ctrl, stride, s);
        return launch_cols(m, n, Xhat, B, ell, grp, G, s);
    }
    if (!takes_small(m, n, B, ell) && ell <= 4) {
        DvGroup grp{};
        for (uint32_t g = 0; g < G; ++g) {
            grp.Yhat[g] = Yhat[g];
            grp.My[g] = My[g];
            grp.R[g] = R[g];
            grp.U[g] = U[g];
            grp.Y[g] = Y[g];
            grp.vL[g] = vL ? vL[g] : nullptr;
            grp.vR[g] = vR ? vR[g] : nullptr;
            grp.accept[g] = accept[g];
        }
        return launch_wide(m, n, Xhat, B, ell, grp, G, ctrl, stride, s);
    }
    for (uint32_t g = 0; g < G; ++g) {
        const hipError_t e = launch_decode_verify_masked(m, n, Xhat, Yhat[g], B, My[g], ell, R[g], U[g], Y[g],
                                                         ctrl + g * stride, vL ? vL[g] : nullptr,
                                                         vR ? vR[g] : nullptr, accept[g], s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mvk
