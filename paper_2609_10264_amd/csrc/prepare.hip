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
        uint32_t mv[kQBatch][E], ww[kQBatch];
#pragma unroll
        for (int u = 0; u < kQBatch; ++u) {
            const uint32_t sx = s0 + (uint32_t)u;
            const bool ok = sx < s_end;
            const uint32_t sl = ok ? sx : s_beg;  // in-range term, value masked below
            uint32_t j = idx[sl];
            j = j < nrows ? j : nrows - 1;
            ww[u] = ok ? val[sl] : 0u;
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

template <int U>
constexpr size_t prep_lds_words() {
    constexpr size_t gather = (size_t)kQuarters * gather_part(true) * 2;
    if constexpr (U > 0)
        return syn::lds_words<U, kPrepThreads>() > gather ? syn::lds_words<U, kPrepThreads>() : gather;
    else
        return gather;
}

struct PrepArgs {
    // G problems (keys of one shape and one privacy code) share the noise
    // vectors and their input mask Mx; each has its own verification code,
    // challenges, P^T, Q and outputs My, R, Uq.
    uint32_t G;
    // syndromes in this launch: nsx noise vectors of code x (Mx); nsy
    // challenges of code y per problem (R)
    uint32_t nsx, nsy;
    uint32_t n, rx, m, ry;
    const uint32_t *xpi1, *xpi2, *xv1, *xv2;
    const uint32_t *ypi1[kMaxGroup], *ypi2[kMaxGroup], *yv1[kMaxGroup], *yv2[kMaxGroup];
    const uint32_t *ex_idx, *ex_val;
    uint32_t tx, nx;  // nx noise vectors (My items), tx terms each
    const uint32_t *ey_idx[kMaxGroup], *ey_val[kMaxGroup];
    uint32_t ty, ny;  // ny challenges per problem (U items), ty terms each
    uint32_t nbm, nbn;  // gather_cols(VEC)-column blocks of m and n
    const uint32_t *PT[kMaxGroup], *Q[kMaxGroup];
    uint32_t* Mx;
    uint32_t* My[kMaxGroup];
    uint32_t* R[kMaxGroup];
    uint32_t* Uq[kMaxGroup];
    uint32_t* counter;  // SIG: completion counters (count.h; zero before and after the launch)
    uint32_t slots;
    uint32_t* done;     // SIG: set to done_value once every output is stored
    uint32_t done_value;
};

// Workgroups [0, nsx): one noise syndrome each; [nsx, nsx + G * nsy): one
// challenge syndrome each, problem by problem (U > 0; the whole block in
// LDS); the rest: kQuarters gather items each, per problem first the
// nx * nbm items of My (rows of its PT), then the ny * nbn items of U (rows
// of its Q).  VEC: m and n are multiples of 4 and every PT, Q 16-byte aligned.
// SIG: every output is stored device-coherently; each workgroup waits for its
// stores to complete (vmcnt 0) before the barrier and then counts itself done
// (count.h); the last one sets the done flag, so a kernel of another stream
// that sees the flag sees every output.
template <int U, bool SIG, bool VEC>
__global__ __launch_bounds__(kPrepThreads) void client_prepare_kernel(PrepArgs a) {
    __shared__ __align__(16) uint32_t lds[prep_lds_words<U>()];
    uint32_t bid = blockIdx.x;
    bool gather = true;
    if constexpr (U > 0) {
        if (bid < a.nsx) {
            syn::syn_block<true, U, kPrepThreads, SIG>(bid, a.n, a.rx, a.xpi1, a.xpi2, a.xv1, a.xv2, nullptr,
                                                       a.ex_idx, a.ex_val, a.tx, nullptr, a.Mx, lds);
            gather = false;
        } else if (bid < a.nsx + a.G * a.nsy) {
            const uint32_t k = bid - a.nsx, g = k / a.nsy;
            syn::syn_block<true, U, kPrepThreads, SIG>(k - g * a.nsy, a.m, a.ry, a.ypi1[g], a.ypi2[g], a.yv1[g],
                                                       a.yv2[g], nullptr, a.ey_idx[g], a.ey_val[g], a.ty, nullptr,
                                                       a.R[g], lds);
            gather = false;
        } else {
            bid -= a.nsx + a.G * a.nsy;
        }
    }
    if (gather) {
        const int quarter = threadIdx.x / kQuarter;
        uint64_t* part = reinterpret_cast<uint64_t*>(lds) + quarter * gather_part(VEC);
        constexpr uint32_t cols = gather_cols(VEC);
        uint32_t item = bid * kQuarters + (uint32_t)quarter;
        const uint32_t nbm = a.nbm, nbn = a.nbn;
        const uint32_t ix = a.nx * nbm, iy = a.ny * nbn, per = ix + iy;
        const uint32_t g = per ? item / per : a.G;
        item -= g < a.G ? g * per : 0u;
        if (g < a.G && item < ix) {
            const uint32_t b = item / nbm, cb = item % nbm;
            gather_item<SIG, VEC>(a.PT[g], a.m, a.rx * a.n, a.ex_idx + (size_t)b * a.tx,
                                  a.ex_val + (size_t)b * a.tx, a.tx, a.My[g] + (size_t)b * a.m, cb * cols, true, part);
        } else if (g < a.G) {
            const uint32_t q = (item - ix) / nbn, cb = (item - ix) % nbn;
            gather_item<SIG, VEC>(a.Q[g], a.n, a.ry * a.m, a.ey_idx[g] + (size_t)q * a.ty,
                                  a.ey_val[g] + (size_t)q * a.ty, a.ty, a.Uq[g] + (size_t)q * a.n, cb * cols, true,
                                  part);
        } else {
            gather_item<SIG, VEC>(nullptr, 0u, 1u, nullptr, nullptr, 0u, nullptr, 0u, false, part);
        }
    }
    if constexpr (SIG) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0 && count_last(a.counter, a.slots))
            __hip_atomic_store(a.done, a.done_value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Polls *flag (device-coherent loads, a short sleep between polls) from the
// calling thread until it holds `value`; false after `ticks` of the constant
// wall clock.
__device__ __forceinline__ bool poll_flag(const uint32_t* flag, uint32_t value, uint64_t ticks) {
    const uint64_t t0 = wall_clock64();
    while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != value) {
        if (wall_clock64() - t0 > ticks) return false;
        __builtin_amdgcn_s_sleep(4);
    }
    return true;
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

// Xhat = X + Mx, element-wise over count words, PER words per thread and
// pass with the pass's loads issued first.  WAIT: the loads of X (the query,
// not covered by the flag) are issued before thread 0 of each workgroup
// polls *flag for `value`; Mx is read device-coherently after it.  The flag
// is cleared by the only workgroup, or, with several, by the last one to
// finish (counted on `counter`, which it also clears).
constexpr int kAddThreads = 1024;
template <bool WAIT, int PER>
__global__ __launch_bounds__(kAddThreads) void add_masks(const uint32_t* X, const uint32_t* __restrict__ Mx,
                                                         size_t count, uint32_t* Xhat, uint32_t* flag, uint32_t value,
                                                         uint64_t ticks, uint32_t* timed_out, uint32_t* counter) {
    const size_t stride = (size_t)gridDim.x * kAddThreads, pass = stride * PER;
    const size_t g = (size_t)blockIdx.x * kAddThreads + threadIdx.x;
    bool polled = !WAIT;
    for (size_t base = 0; base < count; base += pass) {
        uint32_t xv[PER], mv[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const size_t i = base + g + stride * u;
            xv[u] = X[i < count ? i : count - 1];
        }
        if (WAIT && !polled) {  // first pass only (uniform)
            if (threadIdx.x == 0) {
                if (!poll_flag(flag, value, ticks)) {
                    if (timed_out) atomicOr(timed_out, 1u);
                } else if (gridDim.x == 1) {
                    __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            __syncthreads();
            polled = true;
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const size_t i = base + g + stride * u, is = i < count ? i : count - 1;
            mv[u] = WAIT ? __hip_atomic_load(&Mx[is], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : Mx[is];
        }
        uint32_t out[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            out[u] = fadd(xv[u], mv[u]);
            // pinned in a register before the guarded store, so that the
            // compiler does not sink the loads into the branch
            asm volatile("" : "+v"(out[u]));
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const size_t i = base + g + stride * u;
            if (i < count) Xhat[i] = out[u];
        }
    }
    if constexpr (WAIT) {
        if (!polled) {  // no pass at all (count == 0): still consume the flag
            if (threadIdx.x == 0 && !poll_flag(flag, value, ticks) && timed_out) atomicOr(timed_out, 1u);
            if (threadIdx.x == 0 && gridDim.x == 1)
                __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (gridDim.x > 1 && threadIdx.x == 0 && atomicAdd(counter, 1u) == gridDim.x - 1) {
            atomicExch(counter, 0u);
            __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
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

// Wall-clock ticks of timeout_us on the current device.
hipError_t wait_ticks(uint32_t timeout_us, uint64_t* ticks) {
    int dev = 0, khz = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return e;
    if (khz <= 0) return hipErrorInvalidValue;
    *ticks = (uint64_t)timeout_us * (uint64_t)khz / 1000u;
    return hipSuccess;
}

// Syndrome tile per thread of a 1024-thread workgroup for block length N
// (0: above kSynScratchAbove, not in this launch).
uint32_t prep_u(uint64_t N) {
    for (uint32_t U : {4u, 8u, 12u, 16u})
        if (N <= (uint64_t)kPrepThreads * U) return U;
    return 0;
}

// Whether the gathers of client_prepare_kernel read 16 bytes per lane: when
// the rows allow it and the 64-column items would need more than 256
// workgroups (a quarter as many wider items then still keep the chip busy;
// below, more and narrower items spread the gathers over more compute units:
// at 4096 x 4096 with one column the wider items cost a microsecond per step).
bool prep_vec(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny) {
    const mvk_key& key = *keys[0];
    if (key.m % 4 != 0 || key.n % 4 != 0) return false;
    for (uint32_t g = 0; g < G; ++g)
        if (((uintptr_t)keys[g]->PT & 15) != 0 || ((uintptr_t)keys[g]->Q & 15) != 0) return false;
    const uint64_t items = (uint64_t)G * ((uint64_t)nx * ceil_div(key.m, gather_cols(false)) +
                                          (uint64_t)ny * ceil_div(key.n, gather_cols(false)));
    return items > 256u * kQuarters;
}

// Workgroups of client_prepare_kernel: one per syndrome short enough for one
// workgroup, then the gather items, kQuarters per workgroup.
uint64_t prep_grid(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny) {
    const mvk_key& key = *keys[0];
    const uint64_t Nx = (uint64_t)key.cx.r * key.n, Ny = (uint64_t)key.cy.r * key.m;
    const uint32_t ux = nx ? prep_u(Nx) : 0u, uy = ny ? prep_u(Ny) : 0u;
    const uint32_t cols = gather_cols(prep_vec(keys, G, nx, ny));
    const uint64_t items = (uint64_t)G * ((uint64_t)nx * ceil_div(key.m, cols) + (uint64_t)ny * ceil_div(key.n, cols));
    return (ux ? nx : 0u) + (uy ? (uint64_t)G * ny : 0u) + (items + kQuarters - 1) / kQuarters;
}

}  // namespace

size_t prep_ctrl_words(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny) {
    const uint64_t grid = prep_grid(keys, G, nx, ny);
    return count_words(count_slots(grid > 0x7fffffffu ? 0x7fffffffu : (uint32_t)grid));
}

size_t prep_ctrl_words(const mvk_key& key, uint32_t nx, uint32_t ny) {
    const mvk_key* k = &key;
    return prep_ctrl_words(&k, 1, nx, ny);
}

hipError_t launch_client_prepare_group(uint32_t G, const mvk_key* const* keys, const uint32_t* ex_idx,
                                       const uint32_t* ex_val, uint32_t tx, uint32_t nx,
                                       const uint32_t* const* ey_idx, const uint32_t* const* ey_val, uint32_t ty,
                                       uint32_t ny, uint32_t* Mx, uint32_t* const* My, uint32_t* const* R,
                                       uint32_t* const* Uq, uint32_t* scratch, uint32_t* counter, uint32_t* done,
                                       uint32_t done_value, hipStream_t s) {
    if (G == 0 || G > kMaxGroup) return hipErrorInvalidValue;
    const mvk_key& key = *keys[0];
    const uint64_t Nx = (uint64_t)key.cx.r * key.n, Ny = (uint64_t)key.cy.r * key.m;
    const uint32_t ux = nx ? prep_u(Nx) : 0u, uy = ny ? prep_u(Ny) : 0u;
    // syndromes too long for one workgroup run in their own (segmented) launches first
    if (nx && !ux) {
        const hipError_t e = launch_syn_sparse(key.cx, ex_idx, ex_val, tx, nx, nullptr, scratch, Mx, s);
        if (e != hipSuccess) return e;
    }
    if (ny && !uy) {
        for (uint32_t g = 0; g < G; ++g) {
            const hipError_t e = launch_syn_sparse(keys[g]->cy, ey_idx[g], ey_val[g], ty, ny, nullptr, scratch, R[g], s);
            if (e != hipSuccess) return e;
        }
    }
    PrepArgs a{};
    a.G = G;
    a.nsx = ux ? nx : 0u;
    a.nsy = uy ? ny : 0u;
    a.n = key.n;
    a.rx = key.cx.r;
    a.m = key.m;
    a.ry = key.cy.r;
    a.xpi1 = key.cx.pi1, a.xpi2 = key.cx.pi2, a.xv1 = key.cx.v1, a.xv2 = key.cx.v2;
    a.ex_idx = ex_idx, a.ex_val = ex_val, a.tx = tx, a.nx = nx;
    a.ty = ty, a.ny = ny;
    for (uint32_t g = 0; g < G; ++g) {
        const mvk_code& cy = keys[g]->cy;
        a.ypi1[g] = cy.pi1, a.ypi2[g] = cy.pi2, a.yv1[g] = cy.v1, a.yv2[g] = cy.v2;
        a.ey_idx[g] = ny ? ey_idx[g] : nullptr, a.ey_val[g] = ny ? ey_val[g] : nullptr;
        a.PT[g] = keys[g]->PT, a.Q[g] = keys[g]->Q;
        a.My[g] = nx ? My[g] : nullptr, a.R[g] = ny ? R[g] : nullptr, a.Uq[g] = ny ? Uq[g] : nullptr;
    }
    const bool vec = prep_vec(keys, G, nx, ny);
    a.nbm = ceil_div(key.m, gather_cols(vec)), a.nbn = ceil_div(key.n, gather_cols(vec));
    a.Mx = Mx;
    a.counter = counter, a.done = done, a.done_value = done_value;
    const uint32_t U = ux > uy ? ux : uy;
    const uint64_t grid = prep_grid(keys, G, nx, ny);
    if (grid == 0) return hipSuccess;
    if (grid > 0x7fffffffu) return hipErrorInvalidValue;
    a.slots = count_slots((uint32_t)grid);
#define MVK_PREP_V(UU, SIG)                                                                                     \
    if (vec)                                                                                                    \
        hipLaunchKernelGGL((client_prepare_kernel<UU, SIG, true>), dim3((uint32_t)grid), dim3(kPrepThreads), 0, s, \
                           a);                                                                                  \
    else                                                                                                        \
        hipLaunchKernelGGL((client_prepare_kernel<UU, SIG, false>), dim3((uint32_t)grid), dim3(kPrepThreads), 0,   \
                           s, a)
#define MVK_PREP(UU)          \
    if (done) {               \
        MVK_PREP_V(UU, true);  \
    } else {                  \
        MVK_PREP_V(UU, false); \
    }
    if (U == 0) { MVK_PREP(0); }
    else if (U == 4) { MVK_PREP(4); }
    else if (U == 8) { MVK_PREP(8); }
    else if (U == 12) { MVK_PREP(12); }
    else { MVK_PREP(16); }
#undef MVK_PREP
#undef MVK_PREP_V
    return hipGetLastError();
}

hipError_t launch_client_prepare(const mvk_key& key, const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx,
                                 uint32_t nx, const uint32_t* ey_idx, const uint32_t* ey_val, uint32_t ty,
                                 uint32_t ny, uint32_t* Mx, uint32_t* My, uint32_t* R, uint32_t* Uq,
                                 uint32_t* scratch, uint32_t* counter, uint32_t* done, uint32_t done_value,
                                 hipStream_t s) {
    const mvk_key* k = &key;
    return launch_client_prepare_group(1, &k, ex_idx, ex_val, tx, nx, &ey_idx, &ey_val, ty, ny, Mx, &My, &R, &Uq,
                                       scratch, counter, done, done_value, s);
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
    // four words per thread, one pass per workgroup up to 256 workgroups (a
    // single workgroup up to 4096 words clears the flag itself)
    size_t blocks = (count + 4u * kAddThreads - 1) / (4u * kAddThreads);
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
    if (flag) MVK_ADD(true, 4); else MVK_ADD(false, 4);
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
