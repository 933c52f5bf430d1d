// Client preparation of Protocol pvMVMD on gfx950: the parts of Encrypt,
// Decrypt and Verify that depend on neither the query nor the server's
// response, so that a client can compute them ahead of time (the paper's
// boost mode) or for the next query while the server evaluates the current
// one (the pipelining of its standard mode, Sec. 7):
//   input mask   Mx_b = Gx e_b                     (Encrypt: Xhat_b = X_b + Mx_b)
//   output mask  My_b = P e_b = sum_j e_j PT[j, :] (Decrypt: Y_b = Yhat_b - My_b)
//   R_q = Gy e_q  and  u_q = e_q^T Q = sum_j e_j Q[j, :]
//                                                  (Verify: v_R = R_q . Yhat_b,
//                                                           v_L = u_q . Xhat_b)
// plus the two online element-wise steps and the stream flags that order a
// preparation stream against the online stream when both are captured in
// separate HIP graphs.
#include "count.h"
#include "field.h"
#include "masks.h"
#include "mvk_internal.h"
#include "syn_block.h"

namespace mvk {

namespace {

constexpr int kPrepThreads = 1024;     // syndrome workgroups hold a block of up to 16384 positions
constexpr int kQuarter = 256;          // gather items per workgroup: kPrepThreads / kQuarter
constexpr int kQuarters = kPrepThreads / kQuarter;
constexpr int kQGroups = kQuarter / 64;  // waves per item, each a share of the sparse terms
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kQBatch = 16;            // gathers in flight per thread

// Columns per gather item: one per lane, or with VEC four consecutive ones per
// lane (16-byte loads: a wave reads 1 KiB of a row per term).
constexpr uint32_t gather_cols(bool vec) { return vec ? 256u : 64u; }
// 64-bit partial sums of one item in LDS (a value per wave and column)
constexpr size_t gather_part(bool vec) { return (size_t)kQGroups * gather_cols(vec); }

// One gather item by a 256-thread quarter of the workgroup:
// out[i] = sum_s val[s] * M[idx[s], i] for the gather_cols(VEC) columns i from
// col0.  The four waves take a contiguous share of the terms each and add
// their partial sums in LDS (`part`, gather_part(VEC) values).  VEC: ld
// is a multiple of 4 and M 16-byte aligned, so a lane's four columns are all
// in the row or all past it.  Every quarter of the workgroup passes the one
// barrier here; a quarter with no item (live = false) issues no loads and
// writes nothing.  COHERENT: the results are stored device-coherently.
template <bool COHERENT, bool VEC>
__device__ __forceinline__ void gather_item(const uint32_t* __restrict__ M, uint32_t ld, uint32_t nrows,
                                            const uint32_t* __restrict__ idx, const uint32_t* __restrict__ val,
                                            uint32_t t, uint32_t* __restrict__ out, uint32_t col0, bool live,
                                            uint64_t* part) {
    constexpr int E = VEC ? 4 : 1;  // columns per lane
    const int ltid = threadIdx.x & (kQuarter - 1);
    const int lane = ltid & 63;
    const int g = __builtin_amdgcn_readfirstlane(ltid >> 6);
    const uint32_t i0 = col0 + (uint32_t)lane * E;
    const bool act = live && i0 < ld;
    const uint32_t is = act ? i0 : 0u;
    const uint32_t tt = live ? t : 0u;
    const uint32_t chunk = (tt + kQGroups - 1) / kQGroups;
    const uint32_t s_beg = (uint32_t)g * chunk;
    const uint32_t s_end = s_beg + chunk < tt ? s_beg + chunk : tt;
    uint64_t acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0;
    for (uint32_t s0 = s_beg; s0 < s_end; s0 += kQBatch) {
        // the batch's terms first: lane u loads term s0 + u (two loads, one
        // wait), and each term is read back from its lane as a wave-uniform
        // value; then every row load of the batch is issued before the first
        // is used (a row load never waits for a later term's index)
        const uint32_t lt = s0 + (uint32_t)(lane & (kQBatch - 1));
        const uint32_t lts = lt < s_end ? lt : s_beg;  // in-range term, value masked below
        const uint32_t jl = idx[lts], vl = val[lts];
        uint32_t mv[kQBatch][E], ww[kQBatch];
#pragma unroll
        for (int u = 0; u < kQBatch; ++u) {
            const bool ok = s0 + (uint32_t)u < s_end;
            uint32_t j = (uint32_t)__builtin_amdgcn_readlane((int)jl, u);
            j = j < nrows ? j : nrows - 1;
            ww[u] = ok ? (uint32_t)__builtin_amdgcn_readlane((int)vl, u) : 0u;
            const uint32_t* src = M + (size_t)j * ld + is;
            // non-temporal: every row segment is read once per launch
            if constexpr (VEC) {
                const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
                mv[u][0] = v.x;
                mv[u][1] = v.y;
                mv[u][2] = v.z;
                mv[u][3] = v.w;
            } else {
                mv[u][0] = __builtin_nontemporal_load(src);
            }
        }
#pragma unroll
        for (int u = 0; u < kQBatch; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] += ffold((uint64_t)ww[u] * mv[u][e]);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) part[(g * E + e) * 64 + lane] = acc[e];
    __syncthreads();
    if (g == 0 && act) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            uint64_t tot = 0;
#pragma unroll
            for (int h = 0; h < kQGroups; ++h) tot += part[(h * E + e) * 64 + lane];
            if (COHERENT)
                __hip_atomic_store(&out[i0 + e], fred64(tot), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            else
                out[i0 + e] = fred64(tot);
        }
    }
}

// Wide gather item for large preparations (VEC only): gather_item over
// kWideCols = 1024 columns, each lane loading four 16-byte pieces of a row
// (a wave reads 4 KiB of the row per term, the row segments of an item are
// four times as long as gather_item's, fewer DRAM pages opened per byte),
// kWideBatch terms per batch (the same 16 loads per lane in flight).
constexpr uint32_t kWideCols = 1024;
constexpr int kWidePieces = 4;  // 16-byte loads per lane and term
constexpr int kWideBatch = kQBatch / kWidePieces;
constexpr size_t gather_part_wide() { return (size_t)kQGroups * kWideCols; }

template <bool COHERENT>
__device__ __forceinline__ void gather_item_wide(const uint32_t* __restrict__ M, uint32_t ld, uint32_t nrows,
                                                 const uint32_t* __restrict__ idx,
                                                 const uint32_t* __restrict__ val, uint32_t t,
                                                 uint32_t* __restrict__ out, uint32_t col0, bool live,
                                                 uint64_t* part) {
    constexpr int E = 4 * kWidePieces;  // columns per lane
    const int ltid = threadIdx.x & (kQuarter - 1);
    const int lane = ltid & 63;
    const int g = __builtin_amdgcn_readfirstlane(ltid >> 6);
    // piece l of this lane: columns col0 + 256 l + 4 lane .. + 3
    bool act[kWidePieces];
    uint32_t is[kWidePieces];
#pragma unroll
    for (int l = 0; l < kWidePieces; ++l) {
        const uint32_t i0 = col0 + 256u * l + 4u * lane;
        act[l] = live && i0 < ld;
        is[l] = act[l] ? i0 : 0u;
    }
    const uint32_t tt = live ? t : 0u;
    const uint32_t chunk = (tt + kQGroups - 1) / kQGroups;
    const uint32_t s_beg = (uint32_t)g * chunk;
    const uint32_t s_end = s_beg + chunk < tt ? s_beg + chunk : tt;
    uint64_t acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0;
    for (uint32_t s0 = s_beg; s0 < s_end; s0 += kWideBatch) {
        // the batch's terms by lanes (as in gather_item), then every row load
        const uint32_t lt = s0 + (uint32_t)(lane & (kWideBatch - 1));
        const uint32_t lts = lt < s_end ? lt : s_beg;
        const uint32_t jl = idx[lts], vl = val[lts];
        uint32_t mv[kWideBatch][E], ww[kWideBatch];
#pragma unroll
        for (int u = 0; u < kWideBatch; ++u) {
            const bool ok = s0 + (uint32_t)u < s_end;
            uint32_t j = (uint32_t)__builtin_amdgcn_readlane((int)jl, u);
            j = j < nrows ? j : nrows - 1;
            ww[u] = ok ? (uint32_t)__builtin_amdgcn_readlane((int)vl, u) : 0u;
            const uint32_t* row = M + (size_t)j * ld;
#pragma unroll
            for (int l = 0; l < kWidePieces; ++l) {
                const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row + is[l]));
                mv[u][4 * l] = v.x;
                mv[u][4 * l + 1] = v.y;
                mv[u][4 * l + 2] = v.z;
                mv[u][4 * l + 3] = v.w;
            }
        }
#pragma unroll
        for (int u = 0; u < kWideBatch; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] += ffold((uint64_t)ww[u] * mv[u][e]);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) part[(g * E + e) * 64 + lane] = acc[e];
    __syncthreads();
    if (g == 0) {
#pragma unroll
        for (int l = 0; l < kWidePieces; ++l) {
            if (!act[l]) continue;
            uint32_t r[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                uint64_t tot = 0;
#pragma unroll
                for (int h = 0; h < kQGroups; ++h) tot += part[(h * E + 4 * l + e) * 64 + lane];
                r[e] = fred64(tot);
            }
            uint32_t* o = out + is[l];  // (word stores: the outputs need no 16-byte alignment)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (COHERENT)
                    __hip_atomic_store(&o[e], r[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                else
                    o[e] = r[e];
            }
        }
    }
}

template <int U>
constexpr size_t prep_lds_words() {
    constexpr size_t gather = (size_t)kQuarters * gather_part(true) * 2;
    if constexpr (U > 0)
        return syn::lds_words<U, kPrepThreads>() > gather ? syn::lds_words<U, kPrepThreads>() : gather;
    else
        return gather;
}

// One input of a preparation launch: count noise vectors e_b of t terms over
// the privacy code (block length r*n) and their input masks Mx (count x n).
struct PrepIn {
    const uint32_t *pi1, *pi2, *v1, *v2;
    const uint32_t *idx, *val;
    uint32_t* Mx;
    uint32_t n, r, t, count;
};
// One key of a preparation launch: the output masks My_b = P e_b of the noise
// of its input (index `in`), and count challenges e_q of t
// terms over its verification code (block length r*m) with R_q = Gy e_q and
// U_q = e_q^T Q.  (With no output masks items_x is 0 and `in` is not read.)
struct PrepProb {
    const uint32_t *pi1, *pi2, *v1, *v2;
    const uint32_t *idx, *val;
    const uint32_t *PT, *Q;
    uint32_t *My, *R, *U;
    uint32_t m, n, r, t, count, in;
    uint32_t nbm, nbn;  // gather_cols(VEC)-column blocks of m and n
    uint32_t items_x;   // My items: noise vectors of the input x nbm
};
struct PrepArgs {
    uint32_t NI, G;
    PrepIn in[kMaxPrep];
    PrepProb pr[kMaxPrep];
    // cumulative workgroup and item counts: noise syndromes of inputs < j + 1
    // (syndromes in this launch only), then challenge syndromes of keys
    // < g + 1 (after all noise syndromes), then gather items of keys < g + 1
    uint32_t sx_end[kMaxPrep], sy_end[kMaxPrep], it_end[kMaxPrep];
    uint32_t* counter;  // SIG: completion counters (count.h; zero before and after the launch)
    uint32_t slots;
    uint32_t* done[kMaxPrep];  // SIG: each set to done_value once every output is stored
    uint32_t ndone, done_value;
};

// Workgroups [0, sx_end[NI-1]): one noise syndrome each, input by input;
// then one challenge syndrome each, key by key (U > 0; the whole block in
// LDS; only the blocks short enough, the longer ones ran before); the rest:
// kQuarters gather items each, per key first the items of My (rows of its
// PT, the noise of its input), then those of U (rows of its Q).  VEC: every
// m and n a multiple of 4 and every PT, Q 16-byte aligned.  SIG: every output
// is stored device-coherently; each workgroup waits for its stores to complete
// (vmcnt 0) before the barrier and then counts itself done (count.h); the last
// one sets the done flags, so a kernel of another stream that sees a flag
// sees every output.  The descriptors are indexed by workgroup-uniform values,
// so they come through scalar loads from the kernel arguments.
template <int U, bool SIG, bool VEC>
__global__ __launch_bounds__(kPrepThreads) void client_prepare_kernel(PrepArgs a) {
    __shared__ __align__(16) uint32_t lds[prep_lds_words<U>()];
    uint32_t bid = blockIdx.x;
    bool gather = true;
    if constexpr (U > 0) {
        const uint32_t sx = a.NI ? a.sx_end[a.NI - 1] : 0u;
        const uint32_t sy = a.G ? a.sy_end[a.G - 1] : sx;
        if (bid < sx) {
            uint32_t j = 0;
            while (bid >= a.sx_end[j]) ++j;
            const PrepIn& in = a.in[j];
            syn::syn_block<true, U, kPrepThreads, SIG>(bid - (j ? a.sx_end[j - 1] : 0u), in.n, in.r, in.pi1, in.pi2,
                                                       in.v1, in.v2, nullptr, in.idx, in.val, in.t, nullptr, in.Mx,
                                                       lds);
            gather = false;
        } else if (bid < sy) {
            uint32_t g = 0;
            while (bid >= a.sy_end[g]) ++g;
            const PrepProb& pr = a.pr[g];
            syn::syn_block<true, U, kPrepThreads, SIG>(bid - (g ? a.sy_end[g - 1] : sx), pr.m, pr.r, pr.pi1, pr.pi2,
                                                       pr.v1, pr.v2, nullptr, pr.idx, pr.val, pr.t, nullptr, pr.R,
                                                       lds);
            gather = false;
        } else {
            bid -= sy;
        }
    }
    if (gather) {
        const int quarter = threadIdx.x / kQuarter;
        uint64_t* part = reinterpret_cast<uint64_t*>(lds) + quarter * gather_part(VEC);
        constexpr uint32_t cols = gather_cols(VEC);
        uint32_t item = bid * kQuarters + (uint32_t)quarter;
        uint32_t g = 0;
        while (g < a.G && item >= a.it_end[g]) ++g;
        if (g < a.G) {
            const PrepProb& pr = a.pr[g];
            item -= g ? a.it_end[g - 1] : 0u;
            if (item < pr.items_x) {
                const PrepIn& in = a.in[pr.in];
                const uint32_t b = item / pr.nbm, cb = item % pr.nbm;
                gather_item<SIG, VEC>(pr.PT, pr.m, in.r * in.n, in.idx + (size_t)b * in.t, in.val + (size_t)b * in.t,
                                      in.t, pr.My + (size_t)b * pr.m, cb * cols, true, part);
            } else {
                const uint32_t q = (item - pr.items_x) / pr.nbn, cb = (item - pr.items_x) % pr.nbn;
                gather_item<SIG, VEC>(pr.Q, pr.n, pr.r * pr.m, pr.idx + (size_t)q * pr.t, pr.val + (size_t)q * pr.t,
                                      pr.t, pr.U + (size_t)q * pr.n, cb * cols, true, part);
            }
        } else {
            gather_item<SIG, VEC>(nullptr, 0u, 1u, nullptr, nullptr, 0u, nullptr, 0u, false, part);
        }
    }
    if constexpr (SIG) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0 && count_last(a.counter, a.slots))
            for (uint32_t f = 0; f < a.ndone; ++f)
                __hip_atomic_store(a.done[f], a.done_value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The gathers of a preparation launch alone, one item per 256-thread
// workgroup (a quarter of client_prepare_kernel's), for launches with many
// items: small workgroups with a small LDS footprint share compute units with
// the kernels of other streams instead of taking whole ones.  The syndromes
// then run before, in client_prepare_kernel launched with their workgroups
// only.  SIG as in client_prepare_kernel.
template <bool SIG, bool VEC, bool WIDE>
__global__ __launch_bounds__(kQuarter) void client_gather_kernel(PrepArgs a) {
    static_assert(!WIDE || VEC, "wide items read 16 bytes per lane and piece");
    __shared__ __align__(16) uint64_t part[WIDE ? gather_part_wide() : gather_part(VEC)];
    constexpr uint32_t cols = WIDE ? kWideCols : gather_cols(VEC);
    uint32_t item = blockIdx.x;
    uint32_t g = 0;
    while (g < a.G && item >= a.it_end[g]) ++g;
    if (g < a.G) {
        const PrepProb& pr = a.pr[g];
        item -= g ? a.it_end[g - 1] : 0u;
        if (item < pr.items_x) {
            const PrepIn& in = a.in[pr.in];
            const uint32_t b = item / pr.nbm, cb = item % pr.nbm;
            if constexpr (WIDE)
                gather_item_wide<SIG>(pr.PT, pr.m, in.r * in.n, in.idx + (size_t)b * in.t, in.val + (size_t)b * in.t,
                                      in.t, pr.My + (size_t)b * pr.m, cb * cols, true, part);
            else
                gather_item<SIG, VEC>(pr.PT, pr.m, in.r * in.n, in.idx + (size_t)b * in.t, in.val + (size_t)b * in.t,
                                      in.t, pr.My + (size_t)b * pr.m, cb * cols, true, part);
        } else {
            const uint32_t q = (item - pr.items_x) / pr.nbn, cb = (item - pr.items_x) % pr.nbn;
            if constexpr (WIDE)
                gather_item_wide<SIG>(pr.Q, pr.n, pr.r * pr.m, pr.idx + (size_t)q * pr.t, pr.val + (size_t)q * pr.t,
                                      pr.t, pr.U + (size_t)q * pr.n, cb * cols, true, part);
            else
                gather_item<SIG, VEC>(pr.Q, pr.n, pr.r * pr.m, pr.idx + (size_t)q * pr.t, pr.val + (size_t)q * pr.t,
                                      pr.t, pr.U + (size_t)q * pr.n, cb * cols, true, part);
        }
    } else {
        if constexpr (WIDE)
            gather_item_wide<SIG>(nullptr, 0u, 1u, nullptr, nullptr, 0u, nullptr, 0u, false, part);
        else
            gather_item<SIG, VEC>(nullptr, 0u, 1u, nullptr, nullptr, 0u, nullptr, 0u, false, part);
    }
    if constexpr (SIG) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0 && count_last(a.counter, a.slots))
            for (uint32_t f = 0; f < a.ndone; ++f)
                __hip_atomic_store(a.done[f], a.done_value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}


// out[v][i] = sum_s val[v*t + s] * M[idx[v*t + s], i] for `count` sparse
// vectors v (M: nrows x ld): nb = ceil(ld / gather_cols(VEC)) items per
// vector, four per workgroup.
template <bool VEC>
__global__ __launch_bounds__(kPrepThreads) void gather_rows_kernel(const uint32_t* __restrict__ M, uint32_t ld,
                                                                   uint32_t nrows, const uint32_t* __restrict__ idx,
                                                                   const uint32_t* __restrict__ val, uint32_t t,
                                                                   uint32_t count, uint32_t nb,
                                                                   uint32_t* __restrict__ out) {
    __shared__ uint64_t part[kQuarters * gather_part(VEC)];
    const int quarter = threadIdx.x / kQuarter;
    const uint32_t item = blockIdx.x * kQuarters + (uint32_t)quarter;
    const bool live = item < count * nb;
    const uint32_t v = live ? item / nb : 0u, cb = live ? item % nb : 0u;
    gather_item<false, VEC>(M, ld, nrows, idx + (size_t)v * t, val + (size_t)v * t, t, out + (size_t)v * ld,
                            cb * gather_cols(VEC), live, part + quarter * gather_part(VEC));
}

template <bool WAIT, int PER>
__global__ __launch_bounds__(kAddThreads) void add_masks(const uint32_t* X, const uint32_t* __restrict__ Mx,
                                                         size_t count, uint32_t* Xhat, uint32_t* flag, uint32_t value,
                                                         uint64_t ticks, uint32_t* timed_out, uint32_t* counter) {
    add_masks_body<WAIT, PER>(blockIdx.x, gridDim.x, X, Mx, count, Xhat, flag, value, ticks, timed_out, counter);
}

__global__ void flag_signal_kernel(uint32_t* flag, uint32_t value) {
    if (threadIdx.x == 0) __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One thread polls the flag (device-coherent loads, a short sleep between
// polls) until it holds `value`, then clears it; after `ticks` of the constant
// wall clock it gives up, leaves the flag and sets *timed_out.
__global__ void flag_wait_kernel(uint32_t* flag, uint32_t value, uint64_t ticks, uint32_t* timed_out) {
    if (threadIdx.x != 0) return;
    if (!poll_flag(flag, value, ticks)) {
        if (timed_out) atomicOr(timed_out, 1u);
        return;
    }
    __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


// Syndrome tile per thread of a 1024-thread workgroup for block length N
// (0: above kSynScratchAbove, not in this launch).
uint32_t prep_u(uint64_t N) {
    for (uint32_t U : {4u, 8u, 12u, 16u})
        if (N <= (uint64_t)kPrepThreads * U) return U;
    return 0;
}

// Whether a syndrome of block length N runs inside the preparation launch.
bool prep_short(uint64_t N) { return prep_u(N) != 0; }

// Noise vectors behind the output masks of key g (those of its input).
uint32_t prob_nx(const PrepInputDesc* ins, const PrepProbDesc& p) {
    return p.in == kPrepNoInput ? 0u : ins[p.in].count;
}

// Whether the gathers of client_prepare_kernel read 16 bytes per lane: when
// the rows allow it and the 64-column items would need more than 256
// workgroups (a quarter as many wider items then still keep the chip busy;
// below, more and narrower items spread the gathers over more compute units:
// at 4096 x 4096 with one column the wider items cost a microsecond per step).
bool prep_vec(const PrepInputDesc* ins, const PrepProbDesc* probs, uint32_t G) {
    uint64_t items = 0;
    for (uint32_t g = 0; g < G; ++g) {
        const mvk_key& key = *probs[g].key;
        const uint32_t nx = prob_nx(ins, probs[g]), ny = probs[g].count;
        if (nx == 0 && ny == 0) continue;
        if (key.m % 4 != 0 || key.n % 4 != 0) return false;
        if (((uintptr_t)key.PT & 15) != 0 || ((uintptr_t)key.Q & 15) != 0) return false;
        items += (uint64_t)nx * ceil_div(key.m, gather_cols(false)) + (uint64_t)ny * ceil_div(key.n, gather_cols(false));
    }
    return items > 256u * kQuarters;
}

// The launch's arguments, syndrome tile and grid (workgroups: the syndromes
// short enough for one workgroup, then the gather items, kQuarters per
// workgroup).
struct PrepPlan {
    PrepArgs a;
    uint32_t U;
    bool vec;
    uint64_t grid;        // workgroups of the launch (of the gather launch when split)
    uint64_t syn_groups;  // syndrome workgroups
    bool split;           // syndromes and gathers in two launches (client_gather_kernel)
    bool wide;            // the gather launch's items are kWideCols columns wide
};

PrepPlan plan_with_cols(PrepPlan pl, const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G,
                        uint32_t cols);

PrepPlan prep_plan(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G) {
    PrepPlan pl{};
    PrepArgs& a = pl.a;
    a.NI = NI;
    a.G = G;
    pl.vec = prep_vec(ins, probs, G);
    return plan_with_cols(pl, ins, NI, probs, G, gather_cols(pl.vec));
}

// The plan's descriptors and counts for items of `cols` columns; a split
// plan with 16-byte rows that has at least 256 items of kWideCols columns
// takes those (client_gather_kernel's wide form).
PrepPlan plan_with_cols(PrepPlan pl, const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G,
                        uint32_t cols) {
    PrepArgs& a = pl.a;
    uint64_t sx = 0, sy = 0, items = 0;
    for (uint32_t j = 0; j < NI; ++j) {
        const PrepInputDesc& d = ins[j];
        PrepIn& in = a.in[j];
        const mvk_code* c = d.cx;
        in.pi1 = c->pi1, in.pi2 = c->pi2, in.v1 = c->v1, in.v2 = c->v2;
        in.idx = d.idx, in.val = d.val, in.Mx = d.Mx;
        in.n = c->k, in.r = c->r, in.t = d.t, in.count = d.count;
        const uint64_t N = (uint64_t)c->k * c->r;
        if (d.count && prep_short(N)) {
            sx += d.count;
            pl.U = prep_u(N) > pl.U ? prep_u(N) : pl.U;
        }
        a.sx_end[j] = (uint32_t)(sx < 0xffffffffu ? sx : 0xffffffffu);
    }
    sy = sx;
    for (uint32_t g = 0; g < G; ++g) {
        const PrepProbDesc& d = probs[g];
        const mvk_key& key = *d.key;
        PrepProb& pr = a.pr[g];
        pr.pi1 = key.cy.pi1, pr.pi2 = key.cy.pi2, pr.v1 = key.cy.v1, pr.v2 = key.cy.v2;
        pr.idx = d.idx, pr.val = d.val, pr.PT = key.PT, pr.Q = key.Q;
        pr.My = d.My, pr.R = d.R, pr.U = d.U;
        pr.m = key.m, pr.n = key.n, pr.r = key.cy.r, pr.t = d.t, pr.count = d.count;
        const uint32_t nx = prob_nx(ins, d);
        pr.in = nx ? d.in : 0u;
        pr.nbm = ceil_div(key.m, cols), pr.nbn = ceil_div(key.n, cols);
        const uint64_t ix = (uint64_t)nx * pr.nbm, iy = (uint64_t)d.count * pr.nbn;
        pr.items_x = (uint32_t)(ix < 0xffffffffu ? ix : 0xffffffffu);
        const uint64_t N = (uint64_t)key.m * key.cy.r;
        if (d.count && prep_short(N)) {
            sy += d.count;
            pl.U = prep_u(N) > pl.U ? prep_u(N) : pl.U;
        }
        a.sy_end[g] = (uint32_t)(sy < 0xffffffffu ? sy : 0xffffffffu);
        items += ix + iy;
        a.it_end[g] = (uint32_t)(items < 0xffffffffu ? items : 0xffffffffu);
    }
    // more gather workgroups than compute units: the gathers take their own
    // launch of small workgroups (client_gather_kernel), after the syndromes
    pl.syn_groups = sy;
    pl.split = (items + kQuarters - 1) / kQuarters > 256;
    pl.grid = pl.split ? items : sy + (items + kQuarters - 1) / kQuarters;
    pl.wide = cols == kWideCols;
    if (pl.split && pl.vec && !pl.wide) {
        const PrepPlan w = plan_with_cols(pl, ins, NI, probs, G, kWideCols);
        if (w.grid >= 256) return w;
    }
    return pl;
}

}  // namespace

size_t prep_ctrl_words(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G) {
    const uint64_t grid = prep_plan(ins, NI, probs, G).grid;
    return count_words(count_slots(grid > 0x7fffffffu ? 0x7fffffffu : (uint32_t)grid));
}

static_assert(2 * kMaxPrep <= kMaxSynSets, "one syndrome set per input and per key");

namespace {
// The syndromes too long for one workgroup: noise of the inputs, then
// challenges of the keys (one set each).
uint32_t long_sets(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G, SynSet* sets) {
    uint32_t S = 0;
    for (uint32_t j = 0; j < NI; ++j)
        if (ins[j].count && !prep_short((uint64_t)ins[j].cx->k * ins[j].cx->r))
            sets[S++] = SynSet{ins[j].cx, ins[j].idx, ins[j].val, ins[j].t, ins[j].count, ins[j].Mx};
    for (uint32_t g = 0; g < G; ++g)
        if (probs[g].count && !prep_short((uint64_t)probs[g].key->m * probs[g].key->cy.r))
            sets[S++] = SynSet{&probs[g].key->cy, probs[g].idx, probs[g].val, probs[g].t, probs[g].count, probs[g].R};
    return S;
}
}  // namespace

size_t prep_scratch_bytes(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G) {
    SynSet sets[2 * kMaxPrep];
    return syn_sets_scratch_bytes(sets, long_sets(ins, NI, probs, G, sets));
}

hipError_t launch_client_prepare_multi(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G,
                                       uint32_t* scratch, size_t scratch_bytes, uint32_t* counter,
                                       uint32_t* const* done, uint32_t ndone, uint32_t done_value, hipStream_t s) {
    if (NI > kMaxPrep || G == 0 || G > kMaxPrep || ndone > kMaxPrep) return hipErrorInvalidValue;
    // syndromes too long for one workgroup run first, all of them in one
    // sequence of segmented launches
    SynSet sets[2 * kMaxPrep];
    const uint32_t S = long_sets(ins, NI, probs, G, sets);
    if (S) {
        const hipError_t e = launch_syn_sets(sets, S, scratch, scratch_bytes, s);
        if (e != hipSuccess) return e;
    }
    PrepPlan pl = prep_plan(ins, NI, probs, G);
    if (pl.grid == 0) return hipSuccess;
    if (pl.grid > 0x7fffffffu) return hipErrorInvalidValue;
    PrepArgs& a = pl.a;
    if (pl.split && pl.syn_groups) {
        // the short syndromes: client_prepare_kernel with their workgroups only
        // (complete, and visible to the gather launch, when it ends)
        const dim3 sgrid((uint32_t)pl.syn_groups), sblock(kPrepThreads);
#define MVK_SYN_ONLY(UU) hipLaunchKernelGGL((client_prepare_kernel<UU, false, false>), sgrid, sblock, 0, s, a)
        if (pl.U == 4) { MVK_SYN_ONLY(4); }
        else if (pl.U == 8) { MVK_SYN_ONLY(8); }
        else if (pl.U == 12) { MVK_SYN_ONLY(12); }
        else { MVK_SYN_ONLY(16); }
#undef MVK_SYN_ONLY
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    a.counter = counter;
    a.slots = count_slots((uint32_t)pl.grid);
    a.ndone = done ? ndone : 0u;
    for (uint32_t f = 0; f < a.ndone; ++f) a.done[f] = done[f];
    a.done_value = done_value;
    const bool sig = a.ndone > 0;
    if (pl.split) {
        const dim3 ggrid((uint32_t)pl.grid), gblock(kQuarter);
        if (sig) {
            if (pl.wide) hipLaunchKernelGGL((client_gather_kernel<true, true, true>), ggrid, gblock, 0, s, a);
            else if (pl.vec) hipLaunchKernelGGL((client_gather_kernel<true, true, false>), ggrid, gblock, 0, s, a);
            else hipLaunchKernelGGL((client_gather_kernel<true, false, false>), ggrid, gblock, 0, s, a);
        } else {
            if (pl.wide) hipLaunchKernelGGL((client_gather_kernel<false, true, true>), ggrid, gblock, 0, s, a);
            else if (pl.vec) hipLaunchKernelGGL((client_gather_kernel<false, true, false>), ggrid, gblock, 0, s, a);
            else hipLaunchKernelGGL((client_gather_kernel<false, false, false>), ggrid, gblock, 0, s, a);
        }
        return hipGetLastError();
    }
    const dim3 grid((uint32_t)pl.grid), block(kPrepThreads);
#define MVK_PREP_V(UU, SIG)                                                                             \
    if (pl.vec)                                                                                         \
        hipLaunchKernelGGL((client_prepare_kernel<UU, SIG, true>), grid, block, 0, s, a);              \
    else                                                                                                \
        hipLaunchKernelGGL((client_prepare_kernel<UU, SIG, false>), grid, block, 0, s, a)
#define MVK_PREP(UU)          \
    if (sig) {                \
        MVK_PREP_V(UU, true);  \
    } else {                  \
        MVK_PREP_V(UU, false); \
    }
    if (pl.U == 0) { MVK_PREP(0); }
    else if (pl.U == 4) { MVK_PREP(4); }
    else if (pl.U == 8) { MVK_PREP(8); }
    else if (pl.U == 12) { MVK_PREP(12); }
    else { MVK_PREP(16); }
#undef MVK_PREP
#undef MVK_PREP_V
    return hipGetLastError();
}

namespace {
// The descriptors of G keys that share one input (the noise ex_idx/ex_val of
// nx vectors, mask Mx): the privacy code of the first key.
void group_descs(uint32_t G, const mvk_key* const* keys, const uint32_t* ex_idx, const uint32_t* ex_val,
                 uint32_t tx, uint32_t nx, const uint32_t* const* ey_idx, const uint32_t* const* ey_val, uint32_t ty,
                 uint32_t ny, uint32_t* Mx, uint32_t* const* My, uint32_t* const* R, uint32_t* const* Uq,
                 PrepInputDesc* in, PrepProbDesc* probs) {
    *in = PrepInputDesc{&keys[0]->cx, ex_idx, ex_val, tx, nx, Mx};
    for (uint32_t g = 0; g < G; ++g)
        // (the size queries pass no arrays: every array is read only where it exists)
        probs[g] = PrepProbDesc{keys[g], 0u, ny && ey_idx ? ey_idx[g] : nullptr, ny && ey_val ? ey_val[g] : nullptr,
                                ty, ny, nx && My ? My[g] : nullptr, ny && R ? R[g] : nullptr,
                                ny && Uq ? Uq[g] : nullptr};
}
}  // namespace

size_t prep_ctrl_words(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny) {
    if (G == 0 || G > kMaxPrep) return 0;
    PrepInputDesc in;
    PrepProbDesc probs[kMaxPrep];
    group_descs(G, keys, nullptr, nullptr, 0u, nx, nullptr, nullptr, 0u, ny, nullptr, nullptr, nullptr, nullptr, &in,
                probs);
    return prep_ctrl_words(&in, 1, probs, G);
}

size_t prep_scratch_bytes(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny) {
    if (G == 0 || G > kMaxPrep) return 0;
    PrepInputDesc in;
    PrepProbDesc probs[kMaxPrep];
    group_descs(G, keys, nullptr, nullptr, 0u, nx, nullptr, nullptr, 0u, ny, nullptr, nullptr, nullptr, nullptr, &in,
                probs);
    return prep_scratch_bytes(&in, 1, probs, G);
}

size_t prep_ctrl_words(const mvk_key& key, uint32_t nx, uint32_t ny) {
    const mvk_key* k = &key;
    return prep_ctrl_words(&k, 1, nx, ny);
}

hipError_t launch_client_prepare_group(uint32_t G, const mvk_key* const* keys, const uint32_t* ex_idx,
                                       const uint32_t* ex_val, uint32_t tx, uint32_t nx,
                                       const uint32_t* const* ey_idx, const uint32_t* const* ey_val, uint32_t ty,
                                       uint32_t ny, uint32_t* Mx, uint32_t* const* My, uint32_t* const* R,
                                       uint32_t* const* Uq, uint32_t* scratch, size_t scratch_bytes,
                                       uint32_t* counter, uint32_t* done, uint32_t done_value, hipStream_t s) {
    if (G == 0 || G > kMaxGroup) return hipErrorInvalidValue;
    PrepInputDesc in;
    PrepProbDesc probs[kMaxPrep];
    group_descs(G, keys, ex_idx, ex_val, tx, nx, ey_idx, ey_val, ty, ny, Mx, My, R, Uq, &in, probs);
    return launch_client_prepare_multi(&in, 1, probs, G, scratch, scratch_bytes, counter, done ? &done : nullptr,
                                       done ? 1u : 0u, done_value, s);
}

hipError_t launch_client_prepare(const mvk_key& key, const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx,
                                 uint32_t nx, const uint32_t* ey_idx, const uint32_t* ey_val, uint32_t ty,
                                 uint32_t ny, uint32_t* Mx, uint32_t* My, uint32_t* R, uint32_t* Uq,
                                 uint32_t* scratch, size_t scratch_bytes, uint32_t* counter, uint32_t* done,
                                 uint32_t done_value, hipStream_t s) {
    const mvk_key* k = &key;
    return launch_client_prepare_group(1, &k, ex_idx, ex_val, tx, nx, &ey_idx, &ey_val, ty, ny, Mx, &My, &R, &Uq,
                                       scratch, scratch_bytes, counter, done, done_value, s);
}

hipError_t launch_gather_rows(const uint32_t* M, uint32_t ld, uint32_t nrows, const uint32_t* idx,
                              const uint32_t* val, uint32_t t, uint32_t count, uint32_t* out, hipStream_t s) {
    if (count == 0 || ld == 0) return hipSuccess;
    // wider items as in client_prepare_kernel (prep_vec)
    const bool vec = ld % 4 == 0 && ((uintptr_t)M & 15) == 0 &&
                     (uint64_t)count * ceil_div(ld, gather_cols(false)) > 256u * kQuarters;
    const uint32_t nb = ceil_div(ld, gather_cols(vec));
    const uint64_t grid = ((uint64_t)count * nb + kQuarters - 1) / kQuarters;
    if (grid > 0x7fffffffu) return hipErrorInvalidValue;
    if (vec)
        hipLaunchKernelGGL(gather_rows_kernel<true>, dim3((uint32_t)grid), dim3(kPrepThreads), 0, s, M, ld, nrows,
                           idx, val, t, count, nb, out);
    else
        hipLaunchKernelGGL(gather_rows_kernel<false>, dim3((uint32_t)grid), dim3(kPrepThreads), 0, s, M, ld, nrows,
                           idx, val, t, count, nb, out);
    return hipGetLastError();
}

hipError_t launch_add_masks(const uint32_t* X, const uint32_t* Mx, size_t count, uint32_t* Xhat, uint32_t* flag,
                            uint32_t value, uint32_t timeout_us, uint32_t* timed_out, uint32_t* counter,
                            hipStream_t s) {
    if (count == 0 && !flag) return hipSuccess;
    // add_masks_per words per thread, one pass per workgroup up to 256
    // workgroups (a single workgroup clears the flag itself)
    const int per = add_masks_per(count);
    size_t blocks = (count + (size_t)per * kAddThreads - 1) / ((size_t)per * kAddThreads);
    if (blocks > 256) blocks = 256;
    if (blocks == 0) blocks = 1;
    uint64_t ticks = 0;
    if (flag) {
        const hipError_t e = wait_ticks(timeout_us, &ticks);
        if (e != hipSuccess) return e;
    }
#define MVK_ADD(W, P)                                                                                          \
    hipLaunchKernelGGL((add_masks<W, P>), dim3((uint32_t)blocks), dim3(kAddThreads), 0, s, X, Mx, count, Xhat, flag, \
                       value, ticks, timed_out, counter)
    if (per == 1) {
        if (flag) MVK_ADD(true, 1); else MVK_ADD(false, 1);
    } else if (per == 2) {
        if (flag) MVK_ADD(true, 2); else MVK_ADD(false, 2);
    } else {
        if (flag) MVK_ADD(true, 4); else MVK_ADD(false, 4);
    }
#undef MVK_ADD
    return hipGetLastError();
}

hipError_t launch_flag_signal(uint32_t* flag, uint32_t value, hipStream_t s) {
    hipLaunchKernelGGL(flag_signal_kernel, dim3(1), dim3(64), 0, s, flag, value);
    return hipGetLastError();
}

hipError_t launch_flag_wait(uint32_t* flag, uint32_t value, uint32_t timeout_us, uint32_t* timed_out,
                            hipStream_t s) {
    uint64_t ticks = 0;
    const hipError_t e = wait_ticks(timeout_us, &ticks);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(flag_wait_kernel, dim3(1), dim3(64), 0, s, flag, value, ticks, timed_out);
    return hipGetLastError();
}

}  // namespace mvk
