// Server evaluation Yhat = W Xhat mod p (Protocol pvMVMD, server step) on the
// VALU with exact int8-limb arithmetic.
//
// Exactness.  Every query element x in [0, p) is replaced by its centred
// representative xc in [-(p-1)/2, (p-1)/2] and split into four balanced base-256
// digits d0..d3 in [-128, 127] with xc = sum_d 256^d d_d.  The int8 weights are
// then multiplied digit-plane by digit-plane with v_dot4_i32_i8 (four int8
// products summed into an int32).  For one output and one digit plane the
// exact sum over the whole row is bounded by n * 128 * 128 < 2^31 (n <=
// 131071), so every partial sum in any order fits an int32 and the
// accumulation is exact.  The four plane sums S_d are recombined as
// sum_d 2^(8d) S_d mod p.
//
// Digit split trick: with u = (uint32)(xc + 0x80808080), every byte b of u lies
// in [0, 255] and u ^ 0x80808080 holds the four balanced digits as int8 bytes
// (b - 128 == b ^ 0x80 as two's complement), lowest digit in byte 0.
//
// Layout.  W is read in its natural row-major form: a 256-thread workgroup owns
// R rows; thread t reads the 16-byte chunks t, t+256, ... of each row, so one
// wave reads 1 KiB contiguous per row and load instruction.  The thread keeps
// the digit planes of its 16 query elements in registers and reuses them for
// all R rows.  At the end the R*BQ*4 plane sums per thread are reduced across
// the wave by a transpose-reduction (each exchange step halves the number of
// live values) and across the four waves through LDS.
#include "field.h"
#include "mvk_internal.h"

namespace mvk {

namespace {

__device__ __forceinline__ uint32_t digit_word(uint32_t x) {
    const int32_t xc = x > (kP - 1) / 2 ? (int32_t)(x - kP) : (int32_t)x;
    return ((uint32_t)xc + 0x80808080u) ^ 0x80808080u;
}

// Four consecutive query elements -> four digit-plane words: pl[d] holds digit
// d of element e in byte e.
__device__ __forceinline__ void digit_planes(uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3,
                                             int32_t& p0, int32_t& p1, int32_t& p2, int32_t& p3) {
    const uint32_t u0 = digit_word(x0), u1 = digit_word(x1), u2 = digit_word(x2), u3 = digit_word(x3);
    // v_perm_b32(S0, S1, sel): selector bytes 0..3 pick bytes of S1, 4..7 bytes of S0.
    const uint32_t a_lo = __builtin_amdgcn_perm(u1, u0, 0x05010400u);  // u0.d0 u1.d0 u0.d1 u1.d1
    const uint32_t a_hi = __builtin_amdgcn_perm(u1, u0, 0x07030602u);  // u0.d2 u1.d2 u0.d3 u1.d3
    const uint32_t b_lo = __builtin_amdgcn_perm(u3, u2, 0x05010400u);
    const uint32_t b_hi = __builtin_amdgcn_perm(u3, u2, 0x07030602u);
    p0 = (int32_t)__builtin_amdgcn_perm(b_lo, a_lo, 0x05040100u);
    p1 = (int32_t)__builtin_amdgcn_perm(b_lo, a_lo, 0x07060302u);
    p2 = (int32_t)__builtin_amdgcn_perm(b_hi, a_hi, 0x05040100u);
    p3 = (int32_t)__builtin_amdgcn_perm(b_hi, a_hi, 0x07060302u);
}

__device__ __forceinline__ int32_t dot4(int32_t a, int32_t b, int32_t c) {
    return __builtin_amdgcn_sdot4(a, b, c, false);
}

// Transpose-reduction of V values per lane over the 64 lanes of a wave.
// Afterwards lane L holds the wave-wide sum of value index L >> (6 - log2 V).
template <int V>
__device__ __forceinline__ int32_t wave_xreduce(int32_t (&a)[V], int lane) {
    constexpr int LOGV = (V == 64) ? 6 : (V == 32) ? 5 : (V == 16) ? 4 : (V == 8) ? 3 : -1;
    static_assert(LOGV > 0, "V must be 8, 16, 32 or 64");
#pragma unroll
    for (int step = 0; step < LOGV; ++step) {
        const int s = 32 >> step;
        const int half = V >> (step + 1);
        const bool up = (lane & s) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
            const int32_t send = up ? a[i] : a[i + half];
            const int32_t keep = up ? a[i + half] : a[i];
            a[i] = keep + __shfl_xor(send, s);
        }
    }
    int32_t v = a[0];
#pragma unroll
    for (int s = 32 >> LOGV; s >= 1; s >>= 1) v += __shfl_xor(v, s);
    return v;
}

template <int R, int BQ, bool VEC>
__global__ __launch_bounds__(256) void server_eval_valu(const int8_t* __restrict__ W, uint32_t m, uint32_t n,
                                                        const uint32_t* __restrict__ X, uint32_t B,
                                                        uint32_t* __restrict__ Y) {
    constexpr int V = R * BQ * 4;
    const uint32_t row0 = blockIdx.x * R;
    const uint32_t q0 = blockIdx.y * BQ;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    int32_t acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0;

    const uint32_t nchunks = (n + 15) / 16;
    for (uint32_t c = tid; c < nchunks; c += 256) {
        const uint32_t k0 = c * 16;
        int32_t pl[BQ][4][4];  // [query][digit][group of 4 elements]
#pragma unroll
        for (int q = 0; q < BQ; ++q) {
            uint32_t x[16];
            if (q0 + q < B) {
                const uint32_t* xr = X + (size_t)(q0 + q) * n + k0;
                if (VEC) {
                    const uint4* xv = reinterpret_cast<const uint4*>(xr);
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const uint4 t = xv[g];
                        x[4 * g + 0] = t.x;
                        x[4 * g + 1] = t.y;
                        x[4 * g + 2] = t.z;
                        x[4 * g + 3] = t.w;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 16; ++e) x[e] = (k0 + e < n) ? xr[e] : 0u;
                }
            } else {
#pragma unroll
                for (int e = 0; e < 16; ++e) x[e] = 0u;
            }
#pragma unroll
            for (int g = 0; g < 4; ++g)
                digit_planes(x[4 * g], x[4 * g + 1], x[4 * g + 2], x[4 * g + 3], pl[q][0][g], pl[q][1][g],
                             pl[q][2][g], pl[q][3][g]);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint32_t row = row0 + r;
            int32_t w[4] = {0, 0, 0, 0};
            if (row < m) {
                const int8_t* wr = W + (size_t)row * n + k0;
                if (VEC) {
                    const int4 t = *reinterpret_cast<const int4*>(wr);
                    w[0] = t.x;
                    w[1] = t.y;
                    w[2] = t.z;
                    w[3] = t.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const uint32_t b = (k0 + e < n) ? (uint32_t)(uint8_t)wr[e] : 0u;
                        w[e >> 2] |= (int32_t)(b << (8 * (e & 3)));
                    }
                }
            }
#pragma unroll
            for (int q = 0; q < BQ; ++q)
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    int32_t a = acc[(r * BQ + q) * 4 + d];
                    a = dot4(w[0], pl[q][d][0], a);
                    a = dot4(w[1], pl[q][d][1], a);
                    a = dot4(w[2], pl[q][d][2], a);
                    a = dot4(w[3], pl[q][d][3], a);
                    acc[(r * BQ + q) * 4 + d] = a;
                }
        }
    }

    // Reduce over the wave, then over the four waves.
    constexpr int SH = (V == 64) ? 0 : (V == 32) ? 1 : (V == 16) ? 2 : 3;
    __shared__ int32_t red[4][V];
    const int32_t wsum = wave_xreduce<V>(acc, lane);
    if ((lane & ((1 << SH) - 1)) == 0) red[wave][lane >> SH] = wsum;
    __syncthreads();
    if (tid < 64) {
        // thread t handles value index t % V (lanes >= V duplicate and do not store)
        const int vi = tid % V;
        const int32_t S = red[0][vi] + red[1][vi] + red[2][vi] + red[3][vi];
        const int d = vi & 3;
        uint32_t part = fred_s64((int64_t)S << (8 * d));
        part = fadd(part, (uint32_t)__shfl_xor((int)part, 1));
        part = fadd(part, (uint32_t)__shfl_xor((int)part, 2));
        const int rq = vi >> 2;
        const int r = rq / BQ;
        const int q = rq % BQ;
        const uint32_t row = row0 + r;
        if (tid < V && d == 0 && row < m && q0 + q < B) Y[(size_t)(q0 + q) * m + row] = part;
    }
}

typedef int32_t v4i __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Matrix-core path for up to four query columns per launch group.
//
// The contraction C = D * W^T is done by v_mfma_i32_16x16x64_i8 with
//   A operand (16 rows)  = digit planes of the queries: row i = 4*q + d holds
//                          digit d of query q (four queries per tile),
//   B operand (16 cols)  = 16 rows of W, taken straight from HBM,
// so C[4q + d][j] = sum_k digit_d(x_q[k]) * W[row0 + j][k] is the int32 plane
// sum S_d of query q and row j (same exactness bound as the VALU path).  In
// the 16x16 accumulator layout lane l holds C[4*(l/16) + v][l % 16], v = 0..3:
// one lane ends with all four plane sums of one (query, row) pair, so no
// cross-lane reduction is needed; the matrix core performs it.
//
// A workgroup of KW waves owns 16 rows of W; the waves split K into blocks of
// 64.  Per K chunk each wave first issues the loads of its W blocks (all in
// flight at once), then the workgroup converts the query chunk into digit
// planes in LDS (overlapping the W latency), then each wave runs its MFMAs.
// The KW partial accumulators are summed through LDS at the end.
//
// Both operands use the same lane -> k assignment (lane group l/16 supplies the
// 16 consecutive k of its quarter of the 64-block), so the k order inside the
// instruction does not affect the sum.
// ---------------------------------------------------------------------------
template <int QB, int KW, int KBW, bool VEC>
__global__ __launch_bounds__(KW * 64) void server_eval_mfma_small(const int8_t* __restrict__ W, uint32_t m,
                                                                  uint32_t n, const uint32_t* __restrict__ X,
                                                                  uint32_t B, uint32_t* __restrict__ Y) {
    constexpr int KC = 64 * KBW * KW;  // k per chunk
    constexpr int STRIDE = KC + 16;    // padded LDS row (bytes)
    constexpr int ROWS = 4 * QB;
    __shared__ __align__(16) uint8_t dig[ROWS * STRIDE];
    __shared__ v4i red[KW][64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t row0 = blockIdx.x * 16;
    const uint32_t q0 = blockIdx.y * QB;
    const uint32_t wrow = row0 + (lane & 15);
    const int kg = lane >> 4;
    const int arow = lane & 15;
    const int8_t* wbase = W + (size_t)(wrow < m ? wrow : 0) * n;

    v4i acc = {0, 0, 0, 0};
    for (uint32_t kc0 = 0; kc0 < n; kc0 += KC) {
        v4i bw[KBW];
#pragma unroll
        for (int j = 0; j < KBW; ++j) {
            const uint32_t k = kc0 + (uint32_t)(wave * KBW + j) * 64 + kg * 16;
            v4i t = {0, 0, 0, 0};
            if (wrow < m && k < n) {
                if (VEC) {
                    t = *reinterpret_cast<const v4i*>(wbase + k);
                } else {
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const uint32_t b = (k + e < n) ? (uint32_t)(uint8_t)wbase[k + e] : 0u;
                        t[e >> 2] |= (int32_t)(b << (8 * (e & 3)));
                    }
                }
            }
            bw[j] = t;
        }
        for (int idx = tid; idx < QB * (KC / 4); idx += KW * 64) {
            const int q = idx / (KC / 4);
            const int k4 = idx % (KC / 4);
            const uint32_t k = kc0 + 4 * k4;
            uint32_t x[4] = {0u, 0u, 0u, 0u};
            if (q0 + q < B && k < n) {
                const uint32_t* xr = X + (size_t)(q0 + q) * n + k;
                if (VEC) {
                    const uint4 t = *reinterpret_cast<const uint4*>(xr);
                    x[0] = t.x;
                    x[1] = t.y;
                    x[2] = t.z;
                    x[3] = t.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) x[e] = (k + e < n) ? xr[e] : 0u;
                }
            }
            int32_t p[4];
            digit_planes(x[0], x[1], x[2], x[3], p[0], p[1], p[2], p[3]);
#pragma unroll
            for (int d = 0; d < 4; ++d) *reinterpret_cast<int32_t*>(dig + (q * 4 + d) * STRIDE + 4 * k4) = p[d];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < KBW; ++j) {
            const int kbl = wave * KBW + j;
            if (kc0 + (uint32_t)kbl * 64 < n) {
                v4i a = {0, 0, 0, 0};
                if (arow < ROWS) a = *reinterpret_cast<const v4i*>(dig + arow * STRIDE + kbl * 64 + kg * 16);
                acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, bw[j], acc, 0, 0, 0);
            }
        }
        __syncthreads();
    }
    red[wave][lane] = acc;
    __syncthreads();
    if (wave == 0) {
        v4i sum = red[0][lane];
#pragma unroll
        for (int w = 1; w < KW; ++w) sum += red[w][lane];
        const int q = lane >> 4;
        if (q < QB && q0 + q < B && wrow < m) {
            int64_t v = (int64_t)sum[0] + ((int64_t)sum[1] << 8) + ((int64_t)sum[2] << 16) + ((int64_t)sum[3] << 24);
            Y[(size_t)(q0 + q) * m + wrow] = fred_s64(v);
        }
    }
}

template <int QB, int KW, int KBW>
hipError_t launch_mfma_small(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t B, uint32_t* Y,
                             hipStream_t s) {
    const dim3 grid(ceil_div(m, 16), ceil_div(B, QB));
    const bool vec = (n % 16 == 0) && ((uintptr_t)W % 16 == 0) && ((uintptr_t)X % 16 == 0);
    if (vec)
        hipLaunchKernelGGL((server_eval_mfma_small<QB, KW, KBW, true>), grid, dim3(KW * 64), 0, s, W, m, n, X, B, Y);
    else
        hipLaunchKernelGGL((server_eval_mfma_small<QB, KW, KBW, false>), grid, dim3(KW * 64), 0, s, W, m, n, X, B,
                           Y);
    return hipGetLastError();
}

template <int R, int BQ>
hipError_t launch_cfg(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t B, uint32_t* Y,
                      hipStream_t s) {
    const dim3 grid(ceil_div(m, R), ceil_div(B, BQ));
    const bool vec = (n % 16 == 0) && ((uintptr_t)W % 16 == 0) && ((uintptr_t)X % 16 == 0);
    if (vec)
        hipLaunchKernelGGL((server_eval_valu<R, BQ, true>), grid, dim3(256), 0, s, W, m, n, X, B, Y);
    else
        hipLaunchKernelGGL((server_eval_valu<R, BQ, false>), grid, dim3(256), 0, s, W, m, n, X, B, Y);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_server_eval(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t B,
                              uint32_t* Y, int path, hipStream_t s) {
    if (path == MVK_PATH_VALU) {
        if (B == 1) return launch_cfg<16, 1>(W, m, n, X, B, Y, s);
        if (B == 2) return launch_cfg<8, 2>(W, m, n, X, B, Y, s);
        return launch_cfg<4, 4>(W, m, n, X, B, Y, s);
    }
    if (B == 1) return launch_mfma_small<1, 8, 8>(W, m, n, X, B, Y, s);
    if (B == 2) return launch_mfma_small<2, 8, 8>(W, m, n, X, B, Y, s);
    return launch_mfma_small<4, 8, 4>(W, m, n, X, B, Y, s);
}

}  // namespace mvk
