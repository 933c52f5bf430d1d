// Syndrome G v (App. B: suffix sum, scale by V2, scatter by Pi2, suffix sum,
// scale by V1, scatter by Pi1, fold r) of one vector of length N = k*r by one
// workgroup of T threads, both work arrays in LDS.  Shared by the syndrome
// kernels and the fused decode/verify kernel.
//
// Layout: each work array is T rows of E+1 words; position j sits at word
// j + j/E, so row t holds positions [t*E, t*E + E) plus one pad word.  The
// suffix sums run over contiguous rows (thread t scans its own row, then the
// row totals are scanned across the workgroup); the odd row stride keeps those
// row accesses free of bank conflicts.  The code arrays are read with the
// position interleaved across threads (j = tid + T*u, coalesced) and are all
// in flight before the first LDS phase; the scatters of Pi2 and Pi1 use those
// registers.  The per-position loops are unconditional (positions >= N read a
// valid LDS word and write to the writer's own pad word, which no scan reads),
// so every LDS access of a loop is issued before the first wait.
#pragma once
#include "field.h"

namespace mvk {
namespace syn {

// Inclusive scan of one value per lane across the wave with DPP moves
// (row shifts inside each 16-lane row, then row broadcasts across rows).
__device__ __forceinline__ uint32_t wave_incl_scan_dpp(uint32_t x) {
    x = fadd(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true));  // row_shr:1
    x = fadd(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true));  // row_shr:2
    x = fadd(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true));  // row_shr:4
    x = fadd(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true));  // row_shr:8
    x = fadd(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false));  // row_bcast:15
    x = fadd(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false));  // row_bcast:31
    return x;
}

// Row length for U positions per thread: the power of two >= U.
template <int U>
constexpr int row_len() {
    return U <= 4 ? 4 : U <= 8 ? 8 : U <= 16 ? 16 : U <= 32 ? 32 : 64;
}

// LDS words syn_block<., U, T> needs: two work arrays and the scan scratch.
template <int U, int T>
constexpr size_t lds_words() {
    return (size_t)2 * T * (row_len<U>() + 1) + 2 * (T / 64) + 2;
}

template <int E>
__device__ __forceinline__ uint32_t pad_pos(uint32_t j) {
    static_assert((E & (E - 1)) == 0, "E is a power of two: the row index is a shift");
    return j + j / E;
}

// In-place inclusive suffix sum of the padded array `a` (all T*E positions;
// positions >= N hold zero).  The carry into a row is the sum of the totals
// of all later rows = grand total - inclusive prefix of totals.
template <int E, int T>
__device__ __forceinline__ void row_suffix_scan(uint32_t* a, uint32_t* wsum) {
    constexpr int NW = T / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    uint32_t* row = a + tid * (E + 1);
    uint32_t x[E];
#pragma unroll
    for (int e = 0; e < E; ++e) x[e] = row[e];
#pragma unroll
    for (int e = E - 2; e >= 0; --e) x[e] = fadd(x[e], x[e + 1]);
    const uint32_t incl = wave_incl_scan_dpp(x[0]);
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const uint32_t t = lane < NW ? wsum[lane] : 0u;
        const uint32_t ti = wave_incl_scan_dpp(t);
        if (lane < NW) wsum[NW + 1 + lane] = ti;  // inclusive prefix of wave totals
        if (lane == NW - 1) wsum[NW] = ti;        // grand total
    }
    __syncthreads();
    const uint32_t before = wave ? wsum[NW + wave] : 0u;  // totals of earlier waves
    const uint32_t carry = fsub(wsum[NW], fadd(before, incl));
#pragma unroll
    for (int e = 0; e < E; ++e) row[e] = fadd(x[e], carry);
    __syncthreads();
}

// dst[pi[j]] = v[j] * src[j] for this thread's positions j = tid + T*u (the
// writer's pad word for j >= N).  All reads are issued before the first
// write: the reads may alias the writes as far as the compiler knows, so
// reads interleaved with the writes would each wait for the LDS latency.
template <int U, int E, int T>
__device__ __forceinline__ void scale_scatter(const uint32_t* src, uint32_t* dst, const uint32_t (&pi)[U],
                                              const uint32_t (&v)[U], uint32_t N, uint32_t pad_slot) {
    const int tid = threadIdx.x;
    uint32_t a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = src[pad_pos<E>(tid + T * u)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t j = tid + T * u;
        const uint32_t to = j < N ? pad_pos<E>(pi[u] < N ? pi[u] : N - 1) : pad_slot;
        dst[to] = fmul(v[u], a[u]);
    }
}

// Vector c: sparse input (idx, val rows of t terms; SPARSE) or dense input
// (vin, count x N); out[c*k + i] = (X[c*k + i] +) (G v)[i].  N <= T*U.  With
// COHERENT the results are stored device-coherently (visible to other
// workgroups of the running kernel once the stores have completed).
template <bool SPARSE, int U, int T, bool COHERENT>
__device__ __forceinline__ void syn_block(uint32_t c, uint32_t k, uint32_t r, const uint32_t* __restrict__ pi1,
                                          const uint32_t* __restrict__ pi2, const uint32_t* __restrict__ v1,
                                          const uint32_t* __restrict__ v2, const uint32_t* __restrict__ vin,
                                          const uint32_t* __restrict__ idx, const uint32_t* __restrict__ val,
                                          uint32_t t, const uint32_t* __restrict__ X, uint32_t* out, uint32_t* lds) {
    constexpr int E = row_len<U>();
    constexpr int kRow = E + 1;
    constexpr int kXF = (U + 1) / 2;  // fold outputs per thread prefetched (all of them when r >= 2)
    uint32_t* A = lds;
    uint32_t* Bv = lds + T * kRow;
    uint32_t* wsum = lds + 2 * T * kRow;
    const int tid = threadIdx.x;
    const uint32_t N = k * r;
    const uint32_t pad_slot = (uint32_t)tid * kRow + E;  // this thread's pad word
    // Unconditional loads at an in-range position (j < N, else 0), so all of
    // them are in flight together; positions >= N are never used below.  The
    // first sparse term of this thread is loaded first: it is needed first.
    uint32_t sj = 0, sv = 0;
    if (SPARSE && t) {
        const uint32_t q = (uint32_t)tid < t ? (uint32_t)tid : 0u;
        sj = idx[(size_t)c * t + q];
        sv = val[(size_t)c * t + q];
    }
    // Pi2 and V2 (needed after the first suffix sum) now; Pi1 and V1 after the
    // first suffix sum, so that the initial burst of loads is half as long
    // (one compute unit issues them all) and the second half overlaps the
    // Pi2 phase.
    uint32_t p1[U], p2[U], w1[U], w2[U], xin[SPARSE ? 1 : U], xv[kXF];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t j = tid + T * u;
        const uint32_t js = j < N ? j : 0u;
        p2[u] = pi2[js];
        w2[u] = v2[js];
        if constexpr (!SPARSE) xin[u] = vin[(size_t)c * N + js];
    }
    if (X) {
#pragma unroll
        for (int f = 0; f < kXF; ++f) {
            const uint32_t i = tid + T * f;
            xv[f] = X[(size_t)c * k + (i < k ? i : 0u)];
        }
    }
    // A = input; Bv = 0 at positions >= N (the Pi2 scatter fills [0, N))
    {
        uint32_t* ra = A + tid * kRow;
        uint32_t* rb = Bv + tid * kRow;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (SPARSE) ra[e] = 0u;
            if ((uint32_t)tid * E + e >= N) rb[e] = 0u;
        }
    }
    if constexpr (SPARSE) {
        __syncthreads();
        if ((uint32_t)tid < t) A[pad_pos<E>(sj < N ? sj : N - 1)] = sv;
        for (uint32_t q = tid + T; q < t; q += T) {
            const uint32_t j = idx[(size_t)c * t + q];
            A[pad_pos<E>(j < N ? j : N - 1)] = val[(size_t)c * t + q];
        }
    } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t j = tid + T * u;
            A[pad_pos<E>(j)] = j < N ? xin[u] : 0u;
        }
        // rows past T*U (positions the loop above does not cover) start at zero
#pragma unroll
        for (int e = 0; e < E; ++e)
            if ((uint32_t)tid * E + e >= (uint32_t)T * U) A[tid * kRow + e] = 0u;
    }
    __syncthreads();
    row_suffix_scan<E, T>(A, wsum);  // A
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t j = tid + T * u;
        const uint32_t js = j < N ? j : 0u;
        p1[u] = pi1[js];
        w1[u] = v1[js];
    }
    scale_scatter<U, E, T>(A, Bv, p2, w2, N, pad_slot);  // V2, then Pi2
    __syncthreads();
    row_suffix_scan<E, T>(Bv, wsum);  // A
    scale_scatter<U, E, T>(Bv, A, p1, w1, N, pad_slot);  // V1, then Pi1
    __syncthreads();
    auto store = [&](uint32_t i, uint32_t s) {
        if (COHERENT)
            __hip_atomic_store(&out[(size_t)c * k + i], s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else
            out[(size_t)c * k + i] = s;
    };
    // R: fold blocks of r (+ X); reads at clamped positions, masked
    if (r <= 4) {  // every read of the fold issued before the first wait
        uint32_t d[kXF][4];
#pragma unroll
        for (int f = 0; f < kXF; ++f) {
            const uint32_t i = tid + T * f;
            const uint32_t is = i < k ? i : 0u;
#pragma unroll
            for (int v = 0; v < 4; ++v) d[f][v] = A[pad_pos<E>(is * r + ((uint32_t)v < r ? (uint32_t)v : r - 1))];
        }
#pragma unroll
        for (int f = 0; f < kXF; ++f) {
            const uint32_t i = tid + T * f;
            uint32_t s = X ? xv[f] : 0u;
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if ((uint32_t)v < r) s = fadd(s, d[f][v]);
            if (i < k) store(i, s);
        }
    } else {
#pragma unroll
        for (int f = 0; f < kXF; ++f) {
            const uint32_t i = tid + T * f;
            const uint32_t is = i < k ? i : 0u;
            uint32_t s = X ? xv[f] : 0u;
            for (uint32_t q0 = 0; q0 < r; q0 += 4) {
                uint32_t d[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const uint32_t q = q0 + v < r ? q0 + v : r - 1;
                    d[v] = A[pad_pos<E>(is * r + q)];
                }
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (q0 + v < r) s = fadd(s, d[v]);
            }
            if (i < k) store(i, s);
        }
    }
    for (uint32_t i = tid + T * kXF; i < k; i += T) {  // r = 1 only
        uint32_t s = X ? X[(size_t)c * k + i] : 0u;
        for (uint32_t q = 0; q < r; ++q) s = fadd(s, A[pad_pos<E>(i * r + q)]);
        store(i, s);
    }
}

}  // namespace syn
}  // namespace mvk
