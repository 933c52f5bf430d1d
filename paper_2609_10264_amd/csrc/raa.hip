// RAA code maps (App. B) on gfx950.
//
//   encoding  G^T w = A^T V2 Pi2^T A^T V1 Pi1^T R^T w   (repeat, gather by pi1,
//             scale, prefix sum, gather by pi2, scale, prefix sum)
//   syndrome  G v   = R Pi1 V1 A Pi2 V2 A v             (suffix sum, scale,
//             scatter by pi2, suffix sum, scale, scatter by pi1, fold r)
//
// Two kernel shapes:
//  * enc_pass1/2: many vectors at once (Preprocess encodes every row and every
//    column of W).  One lane owns one vector within a segment of positions, so
//    each prefix sum is a running sum per lane plus a scan over segments, and
//    every access to the batch (vector index innermost) is a coalesced row.
//    The code arrays are indexed by the position only, which is uniform across
//    the workgroup, so they come through scalar loads.
//  * syn_wg: few vectors (Encrypt: one per query column; Verify: one per
//    repetition) of length up to 16384.  One 1024-thread workgroup owns one
//    vector; both work arrays stay in LDS.
//  * syn_p1/p2/p3: longer vectors, cut into segments over three launches.
#include "field.h"
#include "mvk_internal.h"
#include "syn_block.h"

namespace mvk {

namespace {

__device__ __forceinline__ uint32_t load_elem(const uint32_t* p, size_t i) { return p[i]; }
__device__ __forceinline__ uint32_t load_elem(const int8_t* p, size_t i) { return femb(p[i]); }

template <int RR>
__device__ __forceinline__ uint32_t div_r(uint32_t x, uint32_t r) {
    if constexpr (RR > 0)
        return x / RR;
    else
        return x / r;
}

// Batched encoding.  The N positions are cut into segments of L positions
// (L from enc_seg_len), and a one-wave workgroup takes one segment for 64*V
// vectors (V consecutive vectors per lane; vectors innermost in every array,
// so each position is one coalesced row).  Each prefix sum is a reduce, a
// scan over the segment sums, then a second pass that starts every segment
// from its offset (so no output is written twice):
//   sum 1     tot[s][v] = sum over segment s of v1[j] * w_v[pi1[j] / r]
//   scan      off[s][v] = sum of tot[s'][v] for s' < s
//   write 1   t3[j][v] = off[seg(j)][v] + running sum within the segment
//   sum 2, scan, write 2: the same with v2[j] * t3[pi2[j]][v] into out[j][v]
// Every output is the field sum of the same terms as one running sum over all N
// positions; field addition is exact, so the grouping does not change it.
constexpr int kEncLanes = 64;

// Segment length: the longest of 256, 128, 64 that still gives at least 2048
// workgroups (eight waves per compute unit) at four vectors per lane.
uint32_t enc_seg_len(size_t N, size_t nvec) {
    const size_t vg = (nvec + 4 * kEncLanes - 1) / (4 * kEncLanes);
    for (uint32_t L : {256u, 128u})
        if (((N + L - 1) / L) * vg >= 2048) return L;
    return 64u;
}

template <int V>
struct Lanes {
    uint32_t x[V];
};

// V elements (vectors vb .. vb+V-1, stride vs) of one position
template <int V>
__device__ __forceinline__ Lanes<V> load_lanes(const uint32_t* p, size_t vs) {
    Lanes<V> r;
    if constexpr (V == 4) {
        const uint4 q = *(const uint4*)p;
        r.x[0] = q.x, r.x[1] = q.y, r.x[2] = q.z, r.x[3] = q.w;
    } else {
#pragma unroll
        for (int q = 0; q < V; ++q) r.x[q] = p[q * vs];
    }
    return r;
}
template <int V>
__device__ __forceinline__ Lanes<V> load_lanes(const int8_t* p, size_t vs) {
    Lanes<V> r;
    if constexpr (V == 4) {
        const uint32_t w = *(const uint32_t*)p;
#pragma unroll
        for (int q = 0; q < 4; ++q) r.x[q] = femb((int8_t)(w >> (8 * q)));
    } else {
#pragma unroll
        for (int q = 0; q < V; ++q) r.x[q] = femb(p[q * vs]);
    }
    return r;
}
template <int V>
__device__ __forceinline__ void store_lanes(uint32_t* p, size_t vs, const Lanes<V>& v) {
    if constexpr (V == 4) {
        *(uint4*)p = make_uint4(v.x[0], v.x[1], v.x[2], v.x[3]);
    } else {
#pragma unroll
        for (int q = 0; q < V; ++q) p[q * vs] = v.x[q];
    }
}

// First prefix sum (over v1 .* Pi1^T R^T w).  WRITE = false: segment sums
// into tot; WRITE = true: t3 from the offsets in off.
template <typename T, int RR, int V, bool WRITE>
__global__ __launch_bounds__(kEncLanes) void enc_pass1(uint32_t N, uint32_t r, uint32_t L,
                                                       const uint32_t* __restrict__ pi1,
                                                       const uint32_t* __restrict__ v1, const T* __restrict__ in,
                                                       size_t ld_in, size_t vs_in, uint32_t nvec,
                                                       const uint32_t* __restrict__ off, uint32_t* __restrict__ t3,
                                                       uint32_t* __restrict__ tot) {
    const uint32_t seg = blockIdx.x, vb = (blockIdx.y * kEncLanes + threadIdx.x) * V;
    if (vb >= nvec) return;
    const T* src = in + (size_t)vb * vs_in;
    const uint32_t j0 = seg * L, j1 = j0 + L < N ? j0 + L : N;
    Lanes<V> acc;
    if (WRITE)
        acc = load_lanes<V>(off + (size_t)seg * nvec + vb, 1);
    else
#pragma unroll
        for (int q = 0; q < V; ++q) acc.x[q] = 0;
#pragma unroll 8
    for (uint32_t j = j0; j < j1; ++j) {
        uint32_t pj = pi1[j];
        if (pj >= N) pj = N - 1;
        const Lanes<V> x = load_lanes<V>(src + (size_t)div_r<RR>(pj, r) * ld_in, vs_in);
        const uint32_t c = v1[j];
#pragma unroll
        for (int q = 0; q < V; ++q) acc.x[q] = fadd(acc.x[q], fmul(c, x.x[q]));
        if (WRITE) store_lanes<V>(t3 + (size_t)j * nvec + vb, 1, acc);
    }
    if (!WRITE) store_lanes<V>(tot + (size_t)seg * nvec + vb, 1, acc);
}

// Second prefix sum (over v2 .* Pi2^T t3), the same two forms, into out.
template <int V, bool WRITE>
__global__ __launch_bounds__(kEncLanes) void enc_pass2(uint32_t N, uint32_t L, const uint32_t* __restrict__ pi2,
                                                       const uint32_t* __restrict__ v2,
                                                       const uint32_t* __restrict__ t3, uint32_t nvec,
                                                       const uint32_t* __restrict__ off, uint32_t* __restrict__ out,
                                                       size_t ld_out, size_t vs_out, uint32_t* __restrict__ tot) {
    const uint32_t seg = blockIdx.x, vb = (blockIdx.y * kEncLanes + threadIdx.x) * V;
    if (vb >= nvec) return;
    uint32_t* dst = out + (size_t)vb * vs_out;
    const uint32_t j0 = seg * L, j1 = j0 + L < N ? j0 + L : N;
    Lanes<V> acc;
    if (WRITE)
        acc = load_lanes<V>(off + (size_t)seg * nvec + vb, 1);
    else
#pragma unroll
        for (int q = 0; q < V; ++q) acc.x[q] = 0;
#pragma unroll 8
    for (uint32_t j = j0; j < j1; ++j) {
        uint32_t pj = pi2[j];
        if (pj >= N) pj = N - 1;
        const Lanes<V> a = load_lanes<V>(t3 + (size_t)pj * nvec + vb, 1);
        const uint32_t c = v2[j];
#pragma unroll
        for (int q = 0; q < V; ++q) acc.x[q] = fadd(acc.x[q], fmul(c, a.x[q]));
        if (WRITE) store_lanes<V>(dst + (size_t)j * ld_out, vs_out, acc);
    }
    if (!WRITE) store_lanes<V>(tot + (size_t)seg * nvec + vb, 1, acc);
}

// off[s][v] = sum_{s' < s} tot[s'][v] for every vector v (one thread each)
__global__ __launch_bounds__(256) void enc_scan(uint32_t nseg, uint32_t nvec, const uint32_t* __restrict__ tot,
                                                uint32_t* __restrict__ off) {
    const uint32_t v = blockIdx.x * 256 + threadIdx.x;
    if (v >= nvec) return;
    uint32_t run = 0;
#pragma unroll 8
    for (uint32_t sg = 0; sg < nseg; ++sg) {
        const uint32_t t = tot[(size_t)sg * nvec + v];
        off[(size_t)sg * nvec + v] = run;
        run = fadd(run, t);
    }
}

template <typename T, int RR, int V>
hipError_t launch_enc_v(const mvk_code& c, const T* in, size_t ld_in, size_t vs_in, uint32_t nvec, uint32_t* t3,
                        uint32_t* tot, uint32_t* off, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s) {
    const uint32_t N = c.k * c.r, L = enc_seg_len(N, nvec), nseg = ceil_div(N, L);
    const dim3 grid(nseg, ceil_div(nvec, kEncLanes * V)), block(kEncLanes), sgrid(ceil_div(nvec, 256u));
    hipLaunchKernelGGL((enc_pass1<T, RR, V, false>), grid, block, 0, s, N, c.r, L, c.pi1, c.v1, in, ld_in, vs_in,
                       nvec, nullptr, nullptr, tot);
    hipLaunchKernelGGL(enc_scan, sgrid, dim3(256), 0, s, nseg, nvec, tot, off);
    hipLaunchKernelGGL((enc_pass1<T, RR, V, true>), grid, block, 0, s, N, c.r, L, c.pi1, c.v1, in, ld_in, vs_in,
                       nvec, off, t3, nullptr);
    hipLaunchKernelGGL((enc_pass2<V, false>), grid, block, 0, s, N, L, c.pi2, c.v2, t3, nvec, nullptr, nullptr,
                       ld_out, vs_out, tot);
    hipLaunchKernelGGL(enc_scan, sgrid, dim3(256), 0, s, nseg, nvec, tot, off);
    hipLaunchKernelGGL((enc_pass2<V, true>), grid, block, 0, s, N, L, c.pi2, c.v2, t3, nvec, off, out, ld_out,
                       vs_out, nullptr);
    return hipGetLastError();
}

template <typename T, int RR>
hipError_t launch_enc_r(const mvk_code& c, const T* in, size_t ld_in, size_t vs_in, uint32_t nvec, uint32_t* t3,
                        uint32_t* tot, uint32_t* off, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s) {
    // four vectors per lane when every lane's four elements are adjacent and aligned
    const size_t al = 4 * sizeof(T);
    const bool v4 = nvec % 4 == 0 && vs_in == 1 && ld_in % 4 == 0 && (uintptr_t)in % al == 0 && vs_out == 1 &&
                    ld_out % 4 == 0 && (uintptr_t)out % 16 == 0 && (uintptr_t)t3 % 16 == 0 &&
                    (uintptr_t)tot % 16 == 0 && (uintptr_t)off % 16 == 0;
    if (v4) return launch_enc_v<T, RR, 4>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
    return launch_enc_v<T, RR, 1>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
}

template <typename T>
hipError_t launch_encT(const mvk_code& c, const T* in, size_t ld_in, size_t vs_in, uint32_t nvec, uint32_t* t3,
                       uint32_t* seg_scratch, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s) {
    if (nvec == 0) return hipSuccess;
    if (nvec > kMaxEncVectors) return hipErrorInvalidValue;
    const uint32_t N = c.k * c.r;
    uint32_t* tot = seg_scratch;
    uint32_t* off = seg_scratch + (size_t)ceil_div(N, enc_seg_len(N, nvec)) * nvec;
    switch (c.r) {
        case 1: return launch_enc_r<T, 1>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
        case 2: return launch_enc_r<T, 2>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
        case 3: return launch_enc_r<T, 3>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
        case 4: return launch_enc_r<T, 4>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
        case 8: return launch_enc_r<T, 8>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
        default: return launch_enc_r<T, 0>(c, in, ld_in, vs_in, nvec, t3, tot, off, out, ld_out, vs_out, s);
    }
}

// ---------------------------------------------------------------------------
// Syndrome of short blocks (N <= 16384): one 1024-thread workgroup per
// vector, the work arrays in LDS (syn_block.h).
// ---------------------------------------------------------------------------
constexpr int kSynThreads = 1024;
constexpr int kSynMaxU = 16;
static_assert((size_t)kSynThreads * kSynMaxU == kSynScratchAbove, "LDS syndrome covers the scratch-free range");
using syn::wave_incl_scan_dpp;

template <bool SPARSE, int U>
__global__ __launch_bounds__(kSynThreads) void syn_wg(uint32_t k, uint32_t r, const uint32_t* __restrict__ pi1,
                                                      const uint32_t* __restrict__ pi2,
                                                      const uint32_t* __restrict__ v1,
                                                      const uint32_t* __restrict__ v2,
                                                      const uint32_t* __restrict__ vin,
                                                      const uint32_t* __restrict__ idx,
                                                      const uint32_t* __restrict__ val, uint32_t t,
                                                      const uint32_t* __restrict__ X, uint32_t* __restrict__ out) {
    __shared__ uint32_t lds[syn::lds_words<U, kSynThreads>()];
    syn::syn_block<SPARSE, U, kSynThreads, false>(blockIdx.x, k, r, pi1, pi2, v1, v2, vin, idx, val, t, X, out, lds);
}

// ---------------------------------------------------------------------------
// Multi-workgroup syndrome for long blocks (several workgroups per vector).
// The length-N work array is cut into segments of kSegLen positions, one
// workgroup each, in three launches:
//   p1: a = suffix sum of the input (the carry into a segment is the sum of the
//       input beyond it: for sparse input a sum over the t terms, for dense
//       input a reduction of the tail), then b[pi2[j]] = v2[j] a[j]; p1 also
//       resets p2's look-back state
//   p2: c = suffix sum of b, then d[pi1[j]] = v1[j] c[j].  The carry into a
//       segment is the sum of the later segments' sums: every workgroup
//       publishes its segment's sum and reads the later ones (a single-pass
//       scan with look-back).  Segments are handed out by a ticket counter
//       from the last one down, so a workgroup only ever waits for segments
//       taken by workgroups that started before it.
//   p3: out[i] = (X[i] +) sum_{q<r} d[i r + q]
// b and d live in the global scratch (count x 2N words), followed by the
// look-back state: per vector one ticket word and one status word per segment
// (bit 32 set once the segment's sum, in the low 31 bits, is published).
// ---------------------------------------------------------------------------
constexpr int kSegThreads = 256;
constexpr int kSegPer = 4;
constexpr uint32_t kSegLen = kSegThreads * kSegPer;
static_assert(kSegLen == kSynSegLen, "segment length of the scratch layout");
// Bound on the polls of one look-back read (each followed by a short sleep):
// every awaited segment belongs to a workgroup that is already running, so the
// bound is only a guard that makes every wave exit.
constexpr uint32_t kLookSpinLimit = 1u << 22;

__device__ __forceinline__ unsigned long long* look_state(uint32_t* scratch, uint32_t count, uint32_t N, uint32_t c) {
    const uint32_t nseg = (N + kSegLen - 1) / kSegLen;
    return reinterpret_cast<unsigned long long*>(scratch + (size_t)count * 2 * N) + (size_t)c * (nseg + 1);
}

__device__ __forceinline__ uint64_t block_sum_u64_256(uint64_t v, uint64_t* red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, s);
        const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), s);
        v += ((uint64_t)hi << 32) | lo;
    }
    if (lane == 0) red[wave] = v;
    __syncthreads();
    const uint64_t t = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    return t;
}

// Inclusive suffix scan of the kSegPer consecutive values x[] owned by each of
// the 256 threads (thread t owns positions t*kSegPer ..), plus `carry`.
__device__ __forceinline__ void seg_suffix_scan(uint32_t (&x)[kSegPer], uint32_t carry, uint32_t* wsum) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int e = kSegPer - 2; e >= 0; --e) x[e] = fadd(x[e], x[e + 1]);
    const uint32_t incl = wave_incl_scan_dpp(x[0]);  // prefix over lanes of thread totals
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    const uint32_t w0 = wsum[0], w1 = wsum[1], w2 = wsum[2], w3 = wsum[3];
    __syncthreads();
    const uint32_t total = fadd(fadd(w0, w1), fadd(w2, w3));
    uint32_t before = 0;  // totals of earlier waves
    if (wave > 0) before = w0;
    if (wave > 1) before = fadd(before, w1);
    if (wave > 2) before = fadd(before, w2);
    // sum over later threads = total - (prefix through this thread)
    const uint32_t after = fsub(total, fadd(before, incl));
    const uint32_t off = fadd(after, carry);
#pragma unroll
    for (int e = 0; e < kSegPer; ++e) x[e] = fadd(x[e], off);
}

// Several syndromes of long blocks share each of the three launches: set i is
// count vectors over its own code, with its own work region (count x 2N words
// and the look-back state).  grid.y runs over the vectors of all sets, grid.x
// over the segments (p1, p2) or the fold chunks (p3) of the longest; the
// workgroups past a shorter set's end return at once (before p2's ticket).
struct SegSet {
    const uint32_t *pi1, *pi2, *v1, *v2;
    const uint32_t *vin, *idx, *val, *X;
    uint32_t* out;
    uint32_t* work;
    uint32_t k, r, t, count;
};
struct SegArgs {
    uint32_t S;
    uint32_t vend[kMaxSynSets];  // vectors of sets < i + 1
    SegSet set[kMaxSynSets];
};

// The set of global vector vy (grid.y) and the vector's index within it.
__device__ __forceinline__ const SegSet& seg_set(const SegArgs& a, uint32_t vy, uint32_t* c) {
    uint32_t i = 0;
    while (vy >= a.vend[i]) ++i;
    *c = vy - (i ? a.vend[i - 1] : 0u);
    return a.set[i];
}

template <bool SPARSE>
__global__ __launch_bounds__(kSegThreads) void syn_p1(const SegArgs a) {
    __shared__ uint32_t seg[kSegLen];
    __shared__ uint64_t red[4];
    __shared__ uint32_t wsum[4];
    uint32_t c;
    const SegSet& S = seg_set(a, blockIdx.y, &c);
    const uint32_t N = S.k * S.r, nseg = (N + kSegLen - 1) / kSegLen;
    if (blockIdx.x >= nseg) return;
    const uint32_t j0 = blockIdx.x * kSegLen, j1 = (j0 + kSegLen < N) ? j0 + kSegLen : N;
    const int tid = threadIdx.x;
    const uint32_t t = S.t;
    const uint32_t* __restrict__ idx = S.idx;
    const uint32_t* __restrict__ val = S.val;
    uint32_t* bbuf = S.work + (size_t)c * 2 * N;
    if (tid == 0) {
        // p2's look-back state: this segment's status word, and (segment 0) the ticket
        unsigned long long* st = look_state(S.work, S.count, N, c);
        st[1 + blockIdx.x] = 0ull;
        if (blockIdx.x == 0) st[0] = 0ull;
    }
    // code entries of this thread's positions (in flight during the carry)
    uint32_t p2[kSegPer], w2[kSegPer];
#pragma unroll
    for (int e = 0; e < kSegPer; ++e) {
        const uint32_t j = j0 + tid * kSegPer + e;
        const uint32_t js = j < j1 ? j : j0;
        p2[e] = S.pi2[js];
        w2[e] = S.v2[js];
    }
    uint64_t part = 0;
    if (SPARSE) {
        for (uint32_t q = tid; q < t; q += kSegThreads) {
            const uint32_t j = idx[(size_t)c * t + q];
            if (j >= j1 && j < N) part += val[(size_t)c * t + q];
        }
    } else {
        const uint32_t* src = S.vin + (size_t)c * N;
        for (uint32_t j = j1 + tid; j < N; j += kSegThreads) part += src[j];
    }
    const uint32_t carry = fred64(block_sum_u64_256(part, red));
    uint32_t x[kSegPer];
    if (SPARSE) {
#pragma unroll
        for (int e = 0; e < kSegPer; ++e) seg[tid * kSegPer + e] = 0u;
        __syncthreads();
        for (uint32_t q = tid; q < t; q += kSegThreads) {
            const uint32_t j = idx[(size_t)c * t + q];
            if (j >= j0 && j < j1) seg[j - j0] = val[(size_t)c * t + q];
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < kSegPer; ++e) x[e] = seg[tid * kSegPer + e];
    } else {
#pragma unroll
        for (int e = 0; e < kSegPer; ++e) {
            const uint32_t j = j0 + tid * kSegPer + e;
            x[e] = j < j1 ? S.vin[(size_t)c * N + j] : 0u;
        }
    }
    seg_suffix_scan(x, carry, wsum);  // A
#pragma unroll
    for (int e = 0; e < kSegPer; ++e) {
        const uint32_t j = j0 + tid * kSegPer + e;
        if (j < j1) bbuf[p2[e] < N ? p2[e] : N - 1] = fmul(w2[e], x[e]);  // V2, then Pi2 scatter
    }
}

__global__ __launch_bounds__(kSegThreads) void syn_p2(const SegArgs a) {
    __shared__ uint64_t red[4];
    __shared__ uint32_t wsum[4];
    __shared__ uint32_t sh_seg, sh_carry;
    uint32_t c;
    const SegSet& S = seg_set(a, blockIdx.y, &c);
    const uint32_t N = S.k * S.r, nseg = (N + kSegLen - 1) / kSegLen;
    if (blockIdx.x >= nseg) return;  // (uniform: no ticket taken)
    const int tid = threadIdx.x, lane = tid & 63;
    unsigned long long* st = look_state(S.work, S.count, N, c);
    if (tid == 0) {
        const uint32_t ticket = atomicAdd(reinterpret_cast<uint32_t*>(st), 1u);  // < nseg: one per workgroup
        sh_seg = ticket < nseg ? nseg - 1 - ticket : 0u;
    }
    __syncthreads();
    const uint32_t sg = sh_seg;
    const uint32_t j0 = sg * kSegLen, j1 = (j0 + kSegLen < N) ? j0 + kSegLen : N;
    const uint32_t* bbuf = S.work + (size_t)c * 2 * N;
    uint32_t* dbuf = S.work + (size_t)c * 2 * N + N;
    uint32_t p1[kSegPer], w1[kSegPer], x[kSegPer];
#pragma unroll
    for (int e = 0; e < kSegPer; ++e) {
        const uint32_t j = j0 + tid * kSegPer + e;
        const uint32_t js = j < j1 ? j : j0;
        p1[e] = S.pi1[js];
        w1[e] = S.v1[js];
        const uint32_t b = bbuf[js];
        x[e] = j < j1 ? b : 0u;
    }
    // publish this segment's sum
    const uint32_t own = fred64(block_sum_u64_256((uint64_t)x[0] + x[1] + x[2] + x[3], red));
    if (tid == 0) __hip_atomic_store(&st[1 + sg], (1ull << 32) | own, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // carry = sum of the later segments' sums, read 64 segments at a time
    if (tid < 64) {
        uint64_t acc = 0;
        for (uint32_t base = sg + 1; base < nseg; base += 64) {
            const uint32_t q = base + lane;
            if (q < nseg) {
                unsigned long long v = __hip_atomic_load(&st[1 + q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                for (uint32_t spin = 0; !(v >> 32) && spin < kLookSpinLimit; ++spin) {
                    __builtin_amdgcn_s_sleep(1);
                    v = __hip_atomic_load(&st[1 + q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                acc += (uint32_t)v;
            }
        }
#pragma unroll
        for (int sh = 32; sh >= 1; sh >>= 1) {
            const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)acc, sh);
            const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(acc >> 32), sh);
            acc += ((uint64_t)hi << 32) | lo;
        }
        if (tid == 0) sh_carry = fred64(acc);
    }
    __syncthreads();
    seg_suffix_scan(x, sh_carry, wsum);  // A
#pragma unroll
    for (int e = 0; e < kSegPer; ++e) {
        const uint32_t j = j0 + tid * kSegPer + e;
        if (j < j1) dbuf[p1[e] < N ? p1[e] : N - 1] = fmul(w1[e], x[e]);  // V1, then Pi1 scatter
    }
}

__global__ __launch_bounds__(256) void syn_p3(const SegArgs a) {
    uint32_t c;
    const SegSet& S = seg_set(a, blockIdx.y, &c);
    const uint32_t N = S.k * S.r;
    const uint32_t i = blockIdx.x * 256 + threadIdx.x;
    if (i >= S.k) return;
    const uint32_t* dbuf = S.work + (size_t)c * 2 * N + N;
    uint32_t s = 0;
    for (uint32_t q = 0; q < S.r; ++q) s = fadd(s, dbuf[(size_t)i * S.r + q]);  // R: fold blocks of r
    if (S.X) s = fadd(S.X[(size_t)c * S.k + i], s);
    S.out[(size_t)c * S.k + i] = s;
}

// The three launches over sets of one input kind (sparse or dense).
template <bool SPARSE>
hipError_t launch_seg_sets(const SegArgs& a, hipStream_t s) {
    uint32_t maxseg = 0, maxk = 0;
    for (uint32_t i = 0; i < a.S; ++i) {
        const size_t N = (size_t)a.set[i].k * a.set[i].r;
        const uint32_t nseg = (uint32_t)((N + kSegLen - 1) / kSegLen);
        maxseg = nseg > maxseg ? nseg : maxseg;
        maxk = a.set[i].k > maxk ? a.set[i].k : maxk;
    }
    const uint32_t nv = a.S ? a.vend[a.S - 1] : 0u;
    if (nv == 0) return hipSuccess;
    if (nv > 65535u) return hipErrorInvalidValue;
    const dim3 gseg(maxseg, nv);
    hipLaunchKernelGGL((syn_p1<SPARSE>), gseg, dim3(kSegThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(syn_p2, gseg, dim3(kSegThreads), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(syn_p3, dim3(ceil_div(maxk, 256u), nv), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <bool SPARSE>
hipError_t launch_syn(const mvk_code& c, const uint32_t* v, const uint32_t* idx, const uint32_t* val, uint32_t t,
                      uint32_t count, const uint32_t* X, uint32_t* scratch, uint32_t* out, hipStream_t s) {
    if (count == 0) return hipSuccess;
    const size_t N = (size_t)c.k * c.r;
    if (N <= (size_t)kSynThreads * kSynMaxU) {
        // short blocks: one workgroup per vector, everything in LDS
        const dim3 grid(count), block(kSynThreads);
        const size_t U = (N + kSynThreads - 1) / kSynThreads;
#define MVK_SYN(EV)                                                                                        \
    hipLaunchKernelGGL((syn_wg<SPARSE, EV>), grid, block, 0, s, c.k, c.r, c.pi1, c.pi2, c.v1, c.v2, v, idx, val, \
                       t, X, out)
        if (U <= 4) MVK_SYN(4);
        else if (U <= 8) MVK_SYN(8);
        else if (U <= 12) MVK_SYN(12);
        else MVK_SYN(16);
#undef MVK_SYN
        return hipGetLastError();
    }
    SegArgs a{};
    a.S = 1;
    a.vend[0] = count;
    a.set[0] = SegSet{c.pi1, c.pi2, c.v1, c.v2, v, idx, val, X, out, scratch, c.k, c.r, t, count};
    return launch_seg_sets<SPARSE>(a, s);
}

__global__ __launch_bounds__(256) void transpose_i8(const int8_t* __restrict__ W, uint32_t m, uint32_t n,
                                                    int8_t* __restrict__ WT) {
    __shared__ int8_t tile[64][65];
    const uint32_t r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const uint32_t r = r0 + i, c = c0 + tx;
        tile[i][tx] = (r < m && c < n) ? W[(size_t)r * n + c] : (int8_t)0;
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const uint32_t c = c0 + i, r = r0 + tx;  // WT[c][r] = W[r][c]
        if (c < n && r < m) WT[(size_t)c * m + r] = tile[tx][i];
    }
}

__global__ void fill_u32(uint32_t* p, size_t count, uint32_t value) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (size_t)gridDim.x * blockDim.x)
        p[i] = value;
}

}  // namespace

size_t encT_seg_words(size_t N, size_t nvec) {
    const size_t L = enc_seg_len(N, nvec);
    return 2 * ((N + L - 1) / L) * nvec;
}

hipError_t launch_encT_u32(const mvk_code& c, const uint32_t* in, size_t ld_in, size_t vs_in, uint32_t nvec,
                           uint32_t* t3, uint32_t* seg, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s) {
    return launch_encT<uint32_t>(c, in, ld_in, vs_in, nvec, t3, seg, out, ld_out, vs_out, s);
}

hipError_t launch_encT_i8(const mvk_code& c, const int8_t* in, size_t ld_in, size_t vs_in, uint32_t nvec,
                          uint32_t* t3, uint32_t* seg, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s) {
    return launch_encT<int8_t>(c, in, ld_in, vs_in, nvec, t3, seg, out, ld_out, vs_out, s);
}

size_t syn_sets_scratch_bytes(const SynSet* sets, uint32_t S) {
    size_t b = 0;
    for (uint32_t i = 0; i < S; ++i) b += (syn_scratch_bytes(sets[i].count, (size_t)sets[i].c->k * sets[i].c->r) + 255) & ~(size_t)255;
    return b;
}

hipError_t launch_syn_sets(const SynSet* sets, uint32_t S, uint32_t* scratch, size_t scratch_bytes, hipStream_t s) {
    if (S > kMaxSynSets) return hipErrorInvalidValue;
    // the sets' work regions lie one after another: the scratch must hold them all
    if (syn_sets_scratch_bytes(sets, S) > scratch_bytes) return hipErrorInvalidValue;
    SegArgs a{};
    uint32_t nv = 0;
    char* w = reinterpret_cast<char*>(scratch);
    for (uint32_t i = 0; i < S; ++i) {
        const SynSet& d = sets[i];
        const size_t N = (size_t)d.c->k * d.c->r;
        if (N <= kSynScratchAbove) return hipErrorInvalidValue;  // long blocks only
        if (d.count == 0) continue;
        a.set[a.S] = SegSet{d.c->pi1, d.c->pi2, d.c->v1, d.c->v2, nullptr, d.idx, d.val, nullptr, d.out,
                            reinterpret_cast<uint32_t*>(w), d.c->k, d.c->r, d.t, d.count};
        nv += d.count;
        a.vend[a.S++] = nv;
        w += (syn_scratch_bytes(d.count, N) + 255) & ~(size_t)255;
    }
    return launch_seg_sets<true>(a, s);
}

hipError_t launch_syn_dense(const mvk_code& c, const uint32_t* v, uint32_t count, uint32_t* scratch, uint32_t* out,
                            hipStream_t s) {
    return launch_syn<false>(c, v, nullptr, nullptr, 0u, count, nullptr, scratch, out, s);
}

hipError_t launch_syn_sparse(const mvk_code& c, const uint32_t* idx, const uint32_t* val, uint32_t t,
                             uint32_t count, const uint32_t* X, uint32_t* scratch, uint32_t* out, hipStream_t s) {
    return launch_syn<true>(c, nullptr, idx, val, t, count, X, scratch, out, s);
}

hipError_t launch_transpose_i8(const int8_t* W, uint32_t m, uint32_t n, int8_t* WT, hipStream_t s) {
    if (m == 0 || n == 0) return hipSuccess;
    hipLaunchKernelGGL(transpose_i8, dim3(ceil_div(n, 64), ceil_div(m, 64)), dim3(256), 0, s, W, m, n, WT);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, size_t count, uint32_t value, hipStream_t s) {
    if (count == 0) return hipSuccess;
    size_t blocks = (count + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_u32, dim3((uint32_t)blocks), dim3(256), 0, s, p, count, value);
    return hipGetLastError();
}

}  // namespace mvk
