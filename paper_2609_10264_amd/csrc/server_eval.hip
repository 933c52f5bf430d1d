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

// Where a launch writes its results.  The launch walks m = G * mg rows: the
// row stack of G matrices of mg rows each (G = 1: one matrix); row r of the
// stack is row r % mg of output r / mg, and output g is B x mg (query q at
// y[g] + q * mg).
struct YOut {
    uint32_t* y[kMaxGroup];
    uint32_t mg;
    __device__ __forceinline__ uint32_t* at(uint32_t q, uint32_t row) const {
        const uint32_t g = row / mg;
        return y[g] + (size_t)q * mg + (row - g * mg);
    }
};

// The outputs of queries b0.. of every matrix of the stack.
inline YOut yout_shift(YOut o, uint32_t b0) {
    for (int g = 0; g < kMaxGroup; ++g)
        if (o.y[g]) o.y[g] += (size_t)b0 * o.mg;
    return o;
}

// 16 bytes of W, a non-temporal load: W is streamed once per launch, so its
// lines are not kept in the caches (measured on MI355X: the single-query
// launch at 4096 x 4096 from 5.2 to 4.9 us, at 16384 x 16384 from 46 to 41 us).
__device__ __forceinline__ v4i load_w16(const int8_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const v4i*>(p));
}

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
// W operand sources: row-major W read 16 bytes at a time (rows of whole 16-byte
// granules, 16-byte aligned), row-major W read byte by byte, or W packed in
// MFMA operand order (see pack_w_kernel).
enum WLayout { kWRowVec = 0, kWRowScalar = 1, kWPacked = 2 };

template <int QB, int KW, int KBW, bool VEC, int WL>
__global__ __launch_bounds__(KW * 64) void server_eval_mfma_small(const int8_t* __restrict__ W, uint32_t m,
                                                                  uint32_t n, const uint32_t* __restrict__ X,
                                                                  uint32_t B, const YOut Y) {
    constexpr int KC = 64 * KBW * KW;  // k per chunk
    constexpr int STRIDE = KC + 16;    // padded LDS row (bytes)
    constexpr int ROWS = 4 * QB;
    constexpr int NT = (ROWS + 15) / 16;  // A tiles of 16 digit rows (four queries each)
    __shared__ __align__(16) uint8_t dig[ROWS * STRIDE];
    __shared__ v4i red[KW][NT][64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t row0 = blockIdx.x * 16;
    const uint32_t q0 = blockIdx.y * QB;
    const uint32_t wrow = row0 + (lane & 15);
    const int kg = lane >> 4;
    const int arow = lane & 15;
    const int8_t* wbase = W + (size_t)(wrow < m ? wrow : 0) * n;

    // Query elements converted per thread and chunk (four consecutive k each).
    constexpr int NXG = QB * (KC / 4) / (KW * 64);
    static_assert(NXG * KW * 64 == QB * (KC / 4), "chunk must split evenly over the workgroup");
    v4i acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = v4i{0, 0, 0, 0};
    for (uint32_t kc0 = 0; kc0 < n; kc0 += KC) {
        // 1. query loads first (needed first), 2. W loads (in flight during the
        // conversion), 3. convert the query chunk into LDS digit planes.
        uint32_t xq[NXG][4];
        uint32_t xok[NXG];  // bit e set: element e of the group is in range
#pragma unroll
        for (int it = 0; it < NXG; ++it) {
            const int idx = tid + it * KW * 64;
            const int q = idx / (KC / 4);
            const int k4 = idx % (KC / 4);
            const uint32_t k = kc0 + 4 * k4;
            const bool okq = q0 + q < B;
            const uint32_t* xr = X + (size_t)(okq ? q0 + q : 0) * n;
            if (VEC) {
                const uint4 t = *reinterpret_cast<const uint4*>(xr + (k < n ? k : 0));
                xok[it] = (okq && k < n) ? 0xfu : 0u;
                xq[it][0] = t.x;
                xq[it][1] = t.y;
                xq[it][2] = t.z;
                xq[it][3] = t.w;
            } else {
                xok[it] = 0u;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bool ok = okq && k + e < n;
                    xok[it] |= ok ? (1u << e) : 0u;
                    xq[it][e] = xr[ok ? k + e : 0];
                }
            }
        }
        // Keep the query loads ahead of the W loads in the instruction stream:
        // the conversion below then waits only for them, not for W.
        __builtin_amdgcn_sched_barrier(0);
        v4i bw[KBW];
        int32_t wmask[KBW];
#pragma unroll
        for (int j = 0; j < KBW; ++j) {
            // Unconditional load at an in-range address, masked at use: no
            // branches, so the waits can count outstanding loads.
            const uint32_t k = kc0 + (uint32_t)(wave * KBW + j) * 64 + kg * 16;
            v4i t = {0, 0, 0, 0};
            if (WL == kWPacked) {
                // tile (row block, k-block) is 1 KiB in operand order, zero padded
                const uint32_t kb = kc0 / 64 + (uint32_t)(wave * KBW + j);
                const uint32_t nkb = (n + 63) / 64;
                const bool okw = kb < nkb;
                wmask[j] = okw ? -1 : 0;
                t = load_w16(W + (((size_t)blockIdx.x * nkb + (okw ? kb : 0u)) * 64 + lane) * 16);
                bw[j] = t;
                continue;
            }
            const bool okw = wrow < m && k < n;
            wmask[j] = okw ? -1 : 0;
            if (WL == kWRowVec) {
                t = load_w16(wbase + (okw ? k : 0u));
            } else {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const bool ok = okw && k + e < n;
                    const uint32_t b = (uint32_t)(uint8_t)wbase[ok ? k + e : 0u];
                    t[e >> 2] |= (int32_t)((ok ? b : 0u) << (8 * (e & 3)));
                }
            }
            bw[j] = t;
        }
        __builtin_amdgcn_sched_barrier(0);  // all W loads issued before the conversion starts
#pragma unroll
        for (int it = 0; it < NXG; ++it) {
            const int idx = tid + it * KW * 64;
            const int q = idx / (KC / 4);
            const int k4 = idx % (KC / 4);
            int32_t p[4];
            const uint32_t x0 = (xok[it] & 1u) ? xq[it][0] : 0u, x1 = (xok[it] & 2u) ? xq[it][1] : 0u;
            const uint32_t x2 = (xok[it] & 4u) ? xq[it][2] : 0u, x3 = (xok[it] & 8u) ? xq[it][3] : 0u;
            digit_planes(x0, x1, x2, x3, p[0], p[1], p[2], p[3]);
#pragma unroll
            for (int d = 0; d < 4; ++d) *reinterpret_cast<int32_t*>(dig + (q * 4 + d) * STRIDE + 4 * k4) = p[d];
        }
        __syncthreads();
        // Blocks past the end of the row hold zeros on both operands and add
        // nothing, so every MFMA runs unconditionally.
#pragma unroll
        for (int j = 0; j < KBW; ++j) {
            const int kbl = wave * KBW + j;
            v4i w;
            w[0] = bw[j][0] & wmask[j];
            w[1] = bw[j][1] & wmask[j];
            w[2] = bw[j][2] & wmask[j];
            w[3] = bw[j][3] & wmask[j];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int r = t * 16 + arow;  // digit row: 4 * query + digit
                const v4i araw = *reinterpret_cast<const v4i*>(dig + (r < ROWS ? r : 0) * STRIDE + kbl * 64 + kg * 16);
                const int32_t msk = r < ROWS ? -1 : 0;
                v4i a;
                a[0] = araw[0] & msk;
                a[1] = araw[1] & msk;
                a[2] = araw[2] & msk;
                a[3] = araw[3] & msk;
                acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, w, acc[t], 0, 0, 0);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) red[wave][t][lane] = acc[t];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i sum = red[0][t][lane];
#pragma unroll
            for (int w = 1; w < KW; ++w) sum += red[w][t][lane];
            const int q = t * 4 + (lane >> 4);
            if (q < QB && q0 + q < B && wrow < m) {
                int64_t v = (int64_t)sum[0] + ((int64_t)sum[1] << 8) + ((int64_t)sum[2] << 16) +
                            ((int64_t)sum[3] << 24);
                *Y.at(q0 + q, wrow) = fred_s64(v);
            }
        }
    }
}

template <int QB, int KW, int KBW>
hipError_t launch_mfma_small(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t B, const YOut& Y,
                             bool packed, hipStream_t s) {
    const dim3 grid(ceil_div(m, 16), ceil_div(B, QB));
    const bool xvec = (n % 16 == 0) && ((uintptr_t)X % 16 == 0);
    const bool wvec = (n % 16 == 0) && ((uintptr_t)W % 16 == 0);
#define MVK_SMALL(XV, WLV) \
    hipLaunchKernelGGL((server_eval_mfma_small<QB, KW, KBW, XV, WLV>), grid, dim3(KW * 64), 0, s, W, m, n, X, B, Y)
    if (packed) {
        if (xvec) MVK_SMALL(true, kWPacked);
        else MVK_SMALL(false, kWPacked);
    } else if (xvec && wvec) {
        MVK_SMALL(true, kWRowVec);
    } else {
        MVK_SMALL(false, kWRowScalar);
    }
#undef MVK_SMALL
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Matrix-core GEMM path for batches of query columns (B > 4).
//
// C = D W^T, D the digit matrix of the queries (digit row 4q + d = plane d of
// query q, padded with zero rows to QT*16), W read from HBM exactly once.
// digits_tiled_kernel stores D in MFMA operand order: granule (kb, qt, l) is
// the 16 bytes that lane l supplies for digit tile qt and k-block kb (64 k),
// i.e. digit row 16*qt + l%16 at k = 64*kb + 16*(l/16) + [0, 16).
//
// A workgroup of eight waves (two per SIMD) owns a block of W rows and all QT
// digit tiles, over one of `ksplit` equal ranges of k-blocks; the waves form a
// grid over (digit tiles) x (W tiles).  Operands travel HBM/L2 -> LDS with
// global_load_lds_dwordx4 (lane i's 16 bytes land at base + 16*i), so no
// registers hold data in flight and the prefetch depth is set by the ring
// size S: k-block kb uses ring slot kb % S, which holds the block's W tiles
// and digit tiles, each loaded by one wave (or two, with identical bytes).
// Iteration kb: wait until this wave's loads of k-block kb have landed (the
// S-1 later k-blocks may still be in flight), barrier (everyone's landed),
// read the operands from LDS and run the MFMAs, barrier (every wave has read
// the slot), refill the slot with k-block kb+S.  Every operand read is a
// ds_read_b128 at 16*lane: conflict free.
//
// Workgroups are placed so that the eight consecutive workgroup ids (one per
// XCD under round-robin dispatch) of one group take 8/ksplit row blocks and
// all ksplit k-ranges, each XCD always the same k-range: an XCD's L2 then
// holds one k-range of D only.
//
// Epilogue: lane l of C tile (qt, t) holds the four digit sums of query
// 4*qt + l/16 for W row 16*t + l%16, recombined in-lane to a value mod p.
// With ksplit > 1 the k-ranges of a row block are added by the workgroup that
// finishes last (see the end of the kernel).
// ---------------------------------------------------------------------------
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    // s_waitcnt with expcnt and lgkmcnt at their maxima (no wait on them);
    // vmcnt is split over bits [3:0] and [15:14]
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xf) | (0x7 << 4) | (0xf << 8) | (((N >> 4) & 3) << 14));
}

// global_load_lds_dwordx4: lane i's 16 bytes at `src` land at LDS address
// M0 + 16*i.  Issued as inline assembly so that the compiler does not add its
// own (conservative, whole-queue) waits before later LDS reads; the ring
// waits are explicit wait_vmcnt calls.  Vector-memory loads complete in
// order, so loads the compiler does not know about can only make its own
// waits longer, never shorter.
__device__ __forceinline__ void dma16(const void* src, int8_t* lds_base) {
    const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int8_t*)lds_base;
    uint32_t saved;  // M0 is restored right after the issue (the load reads it at issue)
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "global_load_lds_dwordx4 %2, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds), "v"(src)
        : "memory");
}

// One thread per (k-block kb, query q, 16-element quarter kq): reads the 16
// query elements once and writes the four granules of digits 0..3, which are
// consecutive (digit row 4q + d -> lane (4q + d) % 16 + 16*kq of tile q/4).
// Padded queries (q >= B) and elements past n are zero.
template <bool VEC>
__global__ __launch_bounds__(256) void digits_tiled_kernel(const uint32_t* __restrict__ X, uint32_t n, uint32_t B,
                                                           uint32_t QT, uint32_t nkb, int8_t* __restrict__ Dt) {
    const uint32_t g = blockIdx.x * 256 + threadIdx.x;
    const uint32_t nq = QT * 4;
    if (g >= nkb * nq * 4) return;
    const uint32_t kq = g % 4, q = (g / 4) % nq, kb = g / (4 * nq);
    const uint32_t k0 = kb * 64 + kq * 16;
    uint32_t x[16];
    const bool okq = q < B;
    const uint32_t* xr = X + (size_t)(okq ? q : 0u) * n;
    if (VEC) {  // n % 16 == 0 and X 16-byte aligned: the quarter is wholly in or out
        const bool ok = okq && k0 < n;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const uint4 t = *reinterpret_cast<const uint4*>(xr + (ok ? k0 : 0u) + 4 * v);
            x[4 * v] = ok ? t.x : 0u;
            x[4 * v + 1] = ok ? t.y : 0u;
            x[4 * v + 2] = ok ? t.z : 0u;
            x[4 * v + 3] = ok ? t.w : 0u;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const bool ok = okq && k0 + e < n;
            const uint32_t t = xr[ok ? k0 + e : 0u];
            x[e] = ok ? t : 0u;
        }
    }
    int32_t pl[4][4];  // pl[d][w]: digit plane d of elements 4w .. 4w+3
#pragma unroll
    for (int w = 0; w < 4; ++w)
        digit_planes(x[4 * w], x[4 * w + 1], x[4 * w + 2], x[4 * w + 3], pl[0][w], pl[1][w], pl[2][w], pl[3][w]);
    const uint32_t l0 = 4 * (q % 4) + 16 * kq;
    int8_t* dst = Dt + ((size_t)(kb * QT + q / 4) * 64 + l0) * 16;
#pragma unroll
    for (int d = 0; d < 4; ++d)
        *reinterpret_cast<int4*>(dst + 16 * d) = make_int4(pl[d][0], pl[d][1], pl[d][2], pl[d][3]);
}

// sum_d 2^(8d) S_d mod p for the four signed digit-plane sums of one output.
__device__ __forceinline__ uint32_t digits_to_field(v4i sum) { return fdigits4(sum[0], sum[1], sum[2], sum[3]); }

// Epilogue of the streamed kernels: lane `lane` of wave `wave` holds the
// accumulator tiles acc[i][t] of queries qbase + 4i and rows rowbase + 16t.
// With one k-range the values go to Y.  With several, every workgroup stores
// its values with device-coherent stores (written through the XCD's L2),
// waits for them, and counts itself on its row block's counter; the workgroup
// that arrives last reads the other ranges' values with device-coherent loads,
// adds them, writes Y and resets the counter.  No cache-wide flush or
// invalidate is needed.  The values are exchanged in accumulator-tile order
// (64 consecutive words per tile, one per lane), so every store and load
// covers whole cache lines.  `flag` is a word of idle LDS.
template <int QW, int TWW, int NW>
__device__ __forceinline__ void store_tiles(const v4i (&acc)[QW][TWW], uint32_t m, uint32_t B,
                                            const YOut& Y, uint32_t* part, uint32_t* counters,
                                            uint32_t rb, uint32_t nrb, uint32_t ks, uint32_t ksplit, int wave,
                                            int lane, uint32_t rowbase, uint32_t qbase, uint32_t* flag) {
    if (ksplit == 1) {
#pragma unroll
        for (int i = 0; i < QW; ++i)
#pragma unroll
            for (int t = 0; t < TWW; ++t) {
                const uint32_t q = qbase + 4 * i, row = rowbase + 16 * t;
                if (q < B && row < m) *Y.at(q, row) = digits_to_field(acc[i][t]);
            }
        return;
    }
    auto slot = [&](uint32_t o, int i, int t) {
        return ((((size_t)o * nrb + rb) * NW + wave) * (QW * TWW) + i * TWW + t) * 64 + lane;
    };
#pragma unroll
    for (int i = 0; i < QW; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t)
            __hip_atomic_store(&part[slot(ks, i, t)], digits_to_field(acc[i][t]), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's stores are complete
    __syncthreads();
    if (threadIdx.x == 0) *flag = (atomicAdd(&counters[rb], 1u) == ksplit - 1) ? 1u : 0u;
    __syncthreads();
    if (!*flag) return;
    uint32_t v[QW][TWW];
#pragma unroll
    for (int i = 0; i < QW; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t) v[i][t] = digits_to_field(acc[i][t]);
    for (uint32_t o = 0; o < ksplit; ++o) {  // one round of independent loads per range
        if (o == ks) continue;
#pragma unroll
        for (int i = 0; i < QW; ++i)
#pragma unroll
            for (int t = 0; t < TWW; ++t)
                v[i][t] = fadd(v[i][t], __hip_atomic_load(&part[slot(o, i, t)], __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_AGENT));
    }
#pragma unroll
    for (int i = 0; i < QW; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t) {
            const uint32_t q = qbase + 4 * i, row = rowbase + 16 * t;
            if (q < B && row < m) *Y.at(q, row) = v[i][t];
        }
    if (threadIdx.x == 0) atomicExch(&counters[rb], 0u);
}

// Split-k exchange of the digits-stationary kernel: one 64-bit atomic add
// per value into a per-value accumulator (this k-range's value mod p in the
// low 40 bits, a count of arrived k-ranges from bit 40).  The add that
// completes the count (it returns ksplit - 1 arrivals) holds the whole sum:
// that lane writes Y and resets the accumulator, so every launch leaves the
// accumulators at zero.  One round trip to the memory side, and no
// per-row-block counter.  The accumulators are indexed like the kernel's
// value layout: (row block, wave, digit tile, W tile, lane).
template <int QW, int TWW, int NW>
__device__ __forceinline__ void store_tiles_atomic(const v4i (&acc)[QW][TWW], uint32_t m, uint32_t B,
                                                   const YOut& Y, unsigned long long* accum, uint32_t rb,
                                                   uint32_t ksplit, int wave, int lane, uint32_t rowbase,
                                                   uint32_t qbase) {
    unsigned long long old[QW][TWW];
    uint32_t v[QW][TWW];
    const size_t base = ((size_t)rb * NW + wave) * (QW * TWW);
#pragma unroll
    for (int i = 0; i < QW; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t) {
            v[i][t] = digits_to_field(acc[i][t]);
            old[i][t] = atomicAdd(&accum[(base + i * TWW + t) * 64 + lane], (1ull << 40) | (unsigned long long)v[i][t]);
        }
#pragma unroll
    for (int i = 0; i < QW; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t) {
            if ((uint32_t)(old[i][t] >> 40) != ksplit - 1) continue;
            const uint32_t q = qbase + 4 * i, row = rowbase + 16 * t;
            if (q < B && row < m) *Y.at(q, row) = fred64((old[i][t] & ((1ull << 40) - 1)) + v[i][t]);
            __hip_atomic_store(&accum[(base + i * TWW + t) * 64 + lane], 0ull, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
}

// global_load_dwordx4 into a register quad, as inline assembly like dma16 so
// that the explicit wait_vmcnt calls count it; the value may only be used
// after a wait that covers it and a pin_vgpr that orders the use after that
// wait.
__device__ __forceinline__ void load16(v4i& dst, const void* src) {
    asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(dst) : "v"(src) : "memory");
}
__device__ __forceinline__ void pin_vgpr(v4i& x) { asm volatile("" : "+v"(x)); }

// QT digit tiles and NWT = (NW/WQ)*TWW W tiles per workgroup; the NW waves
// form a WQ x (NW/WQ) grid: wave w computes digit tiles [(w%WQ)*QT/WQ, ...)
// against W tiles [(w/WQ)*TWW, ...).  W tiles, shared by the WQ waves of a
// row group, travel HBM -> LDS by global_load_lds into an S-slot ring, every
// wave issuing AW of a k-block's tiles; each wave loads its own QW digit
// tiles (16 bytes per lane, already in operand order) straight into
// registers, S k-blocks ahead, so the DMA path carries W only.  One wait per
// k-block covers both: the loads complete in order, and S blocks are in
// flight.
template <int QT, int NW, int WQ, int TWW, int S, bool PACKED>
__global__ __launch_bounds__(NW * 64) void server_eval_mfma_stream(
    const int8_t* __restrict__ W, uint32_t m, uint32_t n, const int8_t* __restrict__ Dt, uint32_t nkb,
    uint32_t ksplit, uint32_t B, const YOut Y, uint32_t* part, uint32_t* counters) {
    constexpr int WR = NW / WQ;               // waves along the row dimension
    constexpr int NWT = WR * TWW;             // W tiles per workgroup
    constexpr int QW = QT / WQ;               // digit tiles per wave
    constexpr int AW = (NWT + NW - 1) / NW;   // W tiles a wave loads per k-block
    constexpr int PER = AW + QW;              // loads per wave per k-block
    static_assert(WQ * WR == NW && QW * WQ == QT, "tile split");
    static_assert(S * PER <= 63, "vmcnt range");
    static_assert(S >= 2, "ring depth");
    constexpr uint32_t kRows = NWT * 16;
    __shared__ __align__(16) int8_t Wring[S][NWT][1024];
    // workgroup -> (row block, k-range), see above
    const uint32_t xcd = blockIdx.x % 8, per_group = 8 / ksplit;
    const uint32_t rb = (blockIdx.x / 8) * per_group + xcd / ksplit;
    const uint32_t ks = xcd % ksplit;
    if (rb * kRows >= m) return;  // padding workgroup of the last group
    const uint32_t kb_per = (nkb + ksplit - 1) / ksplit;
    const uint32_t kb0 = ks * kb_per;
    const uint32_t kb1 = kb0 + kb_per < nkb ? kb0 + kb_per : nkb;
    const uint32_t nk = kb1 > kb0 ? kb1 - kb0 : 0u;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wq = wave % WQ, wr = wave / WQ;
    const uint32_t kl = (lane >> 4) * 16;
    const int8_t* wptr[AW];  // rows this wave loads (row-major W)
#pragma unroll
    for (int a = 0; a < AW; ++a) {
        const uint32_t row = rb * kRows + ((wave * AW + a) % NWT) * 16 + (lane & 15);
        wptr[a] = W + (size_t)(row < m ? row : m - 1) * n;
    }
    // In-range global k-block of local block j: blocks past the end of the
    // range (and every block of an empty range) re-read an in-range block that
    // is never consumed.
    auto kblock = [&](uint32_t j) {
        const uint32_t kbj = kb0 + (j < nk ? j : (nk ? nk - 1 : 0u));
        return kbj < nkb ? kbj : nkb - 1;
    };
    // Row-major W: columns >= n are read at column 0 (they meet zero digits).
    // Packed W: tile (row tile, k-block) is 1 KiB in operand order, zero padded;
    // row tiles past the end re-read the last one (their rows are not stored).
    // When NWT is not a multiple of NW some tiles are loaded twice (same bytes).
    const uint32_t nrt = (m + 15) / 16;
    v4i dreg[S][QW];
    auto issue = [&](uint32_t j, int slot) {
        const uint32_t kbe = kblock(j);
#pragma unroll
        for (int a = 0; a < AW; ++a) {
            const int tile = (wave * AW + a) % NWT;
            if (PACKED) {
                const uint32_t rt = rb * (kRows / 16) + tile;
                dma16(W + (((size_t)(rt < nrt ? rt : nrt - 1) * nkb + kbe) * 64 + lane) * 16, &Wring[slot][tile][0]);
            } else {
                const uint32_t k = kbe * 64 + kl;
                dma16(wptr[a] + (k < n ? k : 0u), &Wring[slot][tile][0]);
            }
        }
#pragma unroll
        for (int i = 0; i < QW; ++i)
            load16(dreg[slot][i], Dt + ((size_t)(kbe * QT + wq * QW + i) * 64 + lane) * 16);
    };
    v4i acc[QW][TWW];
#pragma unroll
    for (int i = 0; i < QW; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t) acc[i][t] = v4i{0, 0, 0, 0};

#pragma unroll
    for (int j = 0; j < S; ++j) issue(j, j);
    // k-blocks in groups of S so that the ring slot (and the register set of
    // the digit tiles) is a compile-time index
    for (uint32_t j0 = 0; j0 < nk; j0 += S) {
#pragma unroll
        for (int sl = 0; sl < S; ++sl) {
            const uint32_t j = j0 + sl;
            if (j < nk) {
                wait_vmcnt<(S - 1) * PER>();  // this wave's loads of k-block j landed
#pragma unroll
                for (int i = 0; i < QW; ++i) pin_vgpr(dreg[sl][i]);
                __syncthreads();  // everyone's W tiles landed
                v4i cb[TWW];
#pragma unroll
                for (int t = 0; t < TWW; ++t)
                    cb[t] = *reinterpret_cast<const v4i*>(&Wring[sl][wr * TWW + t][16 * lane]);
#pragma unroll
                for (int i = 0; i < QW; ++i)
#pragma unroll
                    for (int t = 0; t < TWW; ++t)
                        acc[i][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(dreg[sl][i], cb[t], acc[i][t], 0, 0, 0);
                __syncthreads();  // every wave has read the slot: refill it
                issue(j + S, sl);
            }
        }
    }
    wait_vmcnt<0>();  // drain the trailing prefetches before the registers are reused or the workgroup exits
#pragma unroll
    for (int sl = 0; sl < S; ++sl)
#pragma unroll
        for (int i = 0; i < QW; ++i) pin_vgpr(dreg[sl][i]);

    const uint32_t rowbase = rb * kRows + wr * (TWW * 16) + (lane & 15);
    const uint32_t qbase = wq * QW * 4 + (lane >> 4);
    store_tiles<QW, TWW, NW>(acc, m, B, Y, part, counters, rb, (m + kRows - 1) / kRows, ks, ksplit, wave, lane,
                             rowbase, qbase, reinterpret_cast<uint32_t*>(&Wring[0][0][0]));
}

// Digits-stationary variant for small batches (QT <= 4, i.e. B <= 16): the
// digit matrix of the workgroup's k-range (QT*16 digit rows x at most KBM
// k-blocks) is computed from the queries by the workgroup itself, once,
// straight into LDS; it is read-only afterwards, so the main loop has no
// barriers.  W needs no sharing between waves (each wave owns TWW row tiles),
// so it travels HBM -> registers with ordinary loads: chunks of C k-blocks,
// the next chunk's loads issued before the current chunk's MFMAs (two
// register sets used in turn).  NW waves (eight as launched: four measured
// no better); rows 16*NW*TWW per workgroup.
template <int QT, int TWW, int KBM, int C, bool PACKED, int NW>
__global__ __launch_bounds__(NW * 64) void server_eval_mfma_dstat(const int8_t* __restrict__ W, uint32_t m,
                                                                  uint32_t n, const uint32_t* __restrict__ X,
                                                                  uint32_t nkb, uint32_t ksplit, uint32_t B,
                                                                  const YOut Y, unsigned long long* accum,
                                                                  uint32_t rot_mul) {
    constexpr uint32_t kRows = NW * TWW * 16;
    __shared__ __align__(16) int8_t Dst[KBM][QT][1024];
    const uint32_t xcd = blockIdx.x % 8, per_group = 8 / ksplit;
    const uint32_t rb = (blockIdx.x / 8) * per_group + xcd / ksplit;
    const uint32_t ks = xcd % ksplit;
    if (rb * kRows >= m) return;  // padding workgroup of the last group
    const uint32_t kb_per = (nkb + ksplit - 1) / ksplit;  // <= KBM (checked by the launcher)
    const uint32_t kb0 = ks * kb_per;
    const uint32_t kb1 = kb0 + kb_per < nkb ? kb0 + kb_per : nkb;
    const uint32_t nk = kb1 > kb0 ? kb1 - kb0 : 0u;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t kl = (lane >> 4) * 16;
    const uint32_t nrt = (m + 15) / 16;
    const int8_t* wptr[TWW];
#pragma unroll
    for (int t = 0; t < TWW; ++t) {
        const uint32_t row = rb * kRows + (wave * TWW + t) * 16 + (lane & 15);
        wptr[t] = W + (size_t)(row < m ? row : m - 1) * n;
    }
    // Each wave walks its k-range from its own starting block (row tile *
    // rot_mul, cyclically): the sum does not depend on the order, and waves
    // of neighbouring row tiles then do not read the same k-offset at once.
    const uint32_t rot = nk ? ((rb * (kRows / 16) + (uint32_t)wave * TWW) * rot_mul) % nk : 0u;
    auto rotj = [&](uint32_t j) { return j + rot < nk ? j + rot : j + rot - nk; };  // j < nk
    // B operand of row tile t at local k-block j (in range: blocks past the
    // end re-read the last block of the range, masked out below)
    auto load_w = [&](uint32_t j, int t) -> v4i {
        const uint32_t kbj = kb0 + (j < nk ? rotj(j) : (nk ? rotj(nk - 1) : 0u));
        const uint32_t kbe = kbj < nkb ? kbj : nkb - 1;
        if (PACKED) {
            const uint32_t rt = rb * (kRows / 16) + wave * TWW + t;
            return load_w16(W + (((size_t)(rt < nrt ? rt : nrt - 1) * nkb + kbe) * 64 + lane) * 16);
        }
        const uint32_t k = kbe * 64 + kl;
        return load_w16(wptr[t] + (k < n ? k : 0u));  // columns >= n meet zero digits
    };
    // Digit tiles of this k-range into LDS: unit (local k-block, query,
    // 16-element quarter) -> the four granules of digits 0..3 (consecutive lanes
    // (4q + d) % 16 + 16*kq of tile q/4); queries >= B and elements past n are
    // zero.  A thread has at most kUnits units; their query loads are issued
    // first (needed first), then the first W chunk, then the conversion (which
    // waits for the query loads only).
    constexpr int kThreads = NW * 64;
    constexpr int kUnits = (KBM * QT * 16 + kThreads - 1) / kThreads;
    const uint32_t nunits = nk * QT * 16;
    const bool xvec = (n % 16 == 0) && (((uintptr_t)X & 15) == 0);
    uint32_t x[kUnits][16];
#pragma unroll
    for (int r = 0; r < kUnits; ++r) {
        const uint32_t u = threadIdx.x + (uint32_t)kThreads * r;
        const uint32_t kq = u % 4, q = (u / 4) % (QT * 4), kbl = u / (QT * 16);
        const uint32_t k0 = (kb0 + kbl) * 64 + kq * 16;
        const bool okq = u < nunits && q < B;
        const uint32_t* xr = X + (size_t)(okq ? q : 0u) * n;
        if (xvec) {
            const bool ok = okq && k0 < n;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const uint4 t = *reinterpret_cast<const uint4*>(xr + (ok ? k0 : 0u) + 4 * v);
                x[r][4 * v] = ok ? t.x : 0u;
                x[r][4 * v + 1] = ok ? t.y : 0u;
                x[r][4 * v + 2] = ok ? t.z : 0u;
                x[r][4 * v + 3] = ok ? t.w : 0u;
            }
        } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const bool ok = okq && k0 + e < n;
                const uint32_t t = xr[ok ? k0 + e : 0u];
                x[r][e] = ok ? t : 0u;
            }
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    v4i wa[C][TWW], wb[C][TWW];
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int t = 0; t < TWW; ++t) wa[c][t] = load_w(c, t);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int r = 0; r < kUnits; ++r) {
        const uint32_t u = threadIdx.x + (uint32_t)kThreads * r;
        if (u >= nunits) break;
        const uint32_t kq = u % 4, q = (u / 4) % (QT * 4), kbl = u / (QT * 16);
        int32_t pl[4][4];
#pragma unroll
        for (int w = 0; w < 4; ++w)
            digit_planes(x[r][4 * w], x[r][4 * w + 1], x[r][4 * w + 2], x[r][4 * w + 3], pl[0][w], pl[1][w],
                         pl[2][w], pl[3][w]);
        int8_t* dst = &Dst[kbl][q / 4][16 * (4 * (q % 4) + 16 * kq)];
#pragma unroll
        for (int d = 0; d < 4; ++d)
            *reinterpret_cast<int4*>(dst + 16 * d) = make_int4(pl[d][0], pl[d][1], pl[d][2], pl[d][3]);
    }
    __syncthreads();  // digit tiles written; read-only from here on
    v4i acc[QT][TWW];
#pragma unroll
    for (int i = 0; i < QT; ++i)
#pragma unroll
        for (int t = 0; t < TWW; ++t) acc[i][t] = v4i{0, 0, 0, 0};
    // MFMAs of the chunk starting at local k-block j0 with W operands w
    // (blocks >= nk contribute nothing: their W operand is masked to zero)
    auto compute = [&](uint32_t j0, const v4i (&w)[C][TWW]) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const uint32_t j = j0 + c;
            const int32_t msk = j < nk ? -1 : 0;
            const uint32_t jd = j < nk ? rotj(j) : 0u;
            v4i ca[QT];
#pragma unroll
            for (int i = 0; i < QT; ++i) ca[i] = *reinterpret_cast<const v4i*>(&Dst[jd][i][16 * lane]);
#pragma unroll
            for (int t = 0; t < TWW; ++t) {
                const v4i bw = w[c][t] & msk;
#pragma unroll
                for (int i = 0; i < QT; ++i)
                    acc[i][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ca[i], bw, acc[i][t], 0, 0, 0);
            }
        }
    };
    // (a chunk is loaded only if it holds a block of the range: no loads past
    // the end that nothing uses)
    for (uint32_t j0 = 0; j0 < nk; j0 += 2 * C) {
        if (j0 + C < nk) {
#pragma unroll
            for (int c = 0; c < C; ++c)
#pragma unroll
                for (int t = 0; t < TWW; ++t) wb[c][t] = load_w(j0 + C + c, t);
        }
        compute(j0, wa);
        if (j0 + C >= nk) break;
        if (j0 + 2 * C < nk) {
#pragma unroll
            for (int c = 0; c < C; ++c)
#pragma unroll
                for (int t = 0; t < TWW; ++t) wa[c][t] = load_w(j0 + 2 * C + c, t);
        }
        compute(j0 + C, wb);
    }
    const uint32_t rowbase = rb * kRows + wave * (TWW * 16) + (lane & 15);
    const uint32_t qbase = (uint32_t)(lane >> 4);
    if (ksplit > 1) {
        store_tiles_atomic<QT, TWW, NW>(acc, m, B, Y, accum, rb, ksplit, wave, lane, rowbase, qbase);
        return;
    }
    __syncthreads();  // every wave is past its last digit-tile read
    store_tiles<QT, TWW, NW>(acc, m, B, Y, nullptr, nullptr, rb, (m + kRows - 1) / kRows, ks, 1u, wave, lane,
                             rowbase, qbase, reinterpret_cast<uint32_t*>(&Dst[0][0][0]));
}

// Streamed-path configurations by digit tiles per launch group (QT): eight
// waves (two per SIMD, so one wave's LDS reads overlap the other's MFMAs),
// wave grid, W tiles per wave, ring slots; at most 28 accumulator tiles per
// wave.  QT = 16: 4 x 2 waves, 7 W tiles each (224 rows); QT = 8: 2 x 4
// waves, 4 W tiles (256 rows); QT <= 4: 1 x 8 waves, 2 W tiles (256 rows).
constexpr int kStreamWaves = 8;
constexpr int kStreamSlots = 4;  // k-blocks in flight (W ring slots and digit register sets)
uint32_t stream_rows(uint32_t qt) { return qt == 16 ? 224u : 256u; }
uint32_t stream_slots(uint32_t) { return kStreamSlots; }

// k-range split: the split (1, 2, 4 or 8) that minimises the estimated time
// ceil(workgroups / 256) * (k-blocks per range + pipeline fill), the smaller
// on ties, keeping at least 4 k-blocks per range.
uint32_t stream_ksplit(uint32_t m, uint32_t n, uint32_t qt) {
    const uint32_t nrb = ceil_div(m, stream_rows(qt)), nkb = ceil_div(n, 64);
    const uint32_t fill = stream_slots(qt) + 2;
    // storing and re-reading the partial values of a split costs about
    // 4*B / 64 = qt k-blocks of W traffic per workgroup
    uint32_t best = 1, best_cost = 0xffffffffu;
    for (uint32_t ks = 1; ks <= 8; ks *= 2) {
        if (ks > 1 && nkb < 4 * ks) break;
        const uint32_t cost = ceil_div(nrb * ks, 256) * (ceil_div(nkb, ks) + fill + (ks > 1 ? qt : 0u));
        if (cost < best_cost) {
            best_cost = cost;
            best = ks;
        }
    }
    return best;
}

// ---------------------------------------------------------------------------
// Wide-tile path for 17..32 queries per launch group on packed W, built on
// v_mfma_i32_32x32x32_i8: one instruction multiplies a 32 x 32 digit tile by
// a 32 x 32 W tile, twice the work of a 16x16x64 instruction for the same 2
// KiB of operands, so every operand byte brought into registers (W from HBM,
// digits from LDS) does twice the work.  Operand order of the instruction
// (checked on the hardware): lane l supplies row (or column) l % 32 at k
// bytes 16*(l/32) .. +16 of the 32-wide k-slice; lane l's sixteen results
// are column l % 32, rows 8*(j/4) + 4*(l/32) + j%4 (j < 16).
//
// digits32_kernel stores the digit matrix D (digit row 4q + d = plane d of
// query q) in that order: tile (kb, dt, h) is the 1 KiB that the 64 lanes
// supply for digit rows 32*dt .. +32 and k = 64*kb + 32*h .. +32.  A k-block
// holds 2*DT tiles (DT = query slots / 8).
//
// server_eval_mfma_x32: NW waves, each owning 32 W rows (two packed row
// tiles) over all of k, so a workgroup owns 32*NW rows and no k is split.
// Per k-block the digit tiles (shared by the waves) travel L2 -> LDS by
// global_load_lds into an S-slot ring, each wave issuing its share, and each
// wave loads its own two W operands (the two 32-wide k-slices of its rows,
// 16 bytes per lane, gathered from the packed 16-row tiles) straight into
// registers with non-temporal loads, S k-blocks ahead.  One wait per k-block
// covers both (loads complete in issue order).  A wave's DT accumulator
// tiles hold the four digit sums of 2*DT*4 queries per lane, recombined in
// the lane to values mod p.
// ---------------------------------------------------------------------------
template <bool VEC>
__global__ __launch_bounds__(256) void digits32_kernel(const uint32_t* __restrict__ X, uint32_t n, uint32_t B,
                                                       uint32_t DT, uint32_t nkb, int8_t* __restrict__ Dt) {
    // one thread per (k-block kb, query q, 16-element quarter kq)
    const uint32_t g = blockIdx.x * 256 + threadIdx.x;
    const uint32_t nq = DT * 8;
    if (g >= nkb * nq * 4) return;
    const uint32_t kq = g % 4, q = (g / 4) % nq, kb = g / (4 * nq);
    const uint32_t k0 = kb * 64 + kq * 16;
    uint32_t x[16];
    const bool okq = q < B;
    const uint32_t* xr = X + (size_t)(okq ? q : 0u) * n;
    if (VEC) {  // n % 16 == 0 and X 16-byte aligned: the quarter is wholly in or out
        const bool ok = okq && k0 < n;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const uint4 t = *reinterpret_cast<const uint4*>(xr + (ok ? k0 : 0u) + 4 * v);
            x[4 * v] = ok ? t.x : 0u;
            x[4 * v + 1] = ok ? t.y : 0u;
            x[4 * v + 2] = ok ? t.z : 0u;
            x[4 * v + 3] = ok ? t.w : 0u;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const bool ok = okq && k0 + e < n;
            const uint32_t t = xr[ok ? k0 + e : 0u];
            x[e] = ok ? t : 0u;
        }
    }
    int32_t pl[4][4];  // pl[d][w]: digit plane d of elements 4w .. 4w+3
#pragma unroll
    for (int w = 0; w < 4; ++w)
        digit_planes(x[4 * w], x[4 * w + 1], x[4 * w + 2], x[4 * w + 3], pl[0][w], pl[1][w], pl[2][w], pl[3][w]);
    // digit rows 4q .. 4q+3 are lanes (4q % 32) .. +3 of tile (kb, q / 8, kq / 2),
    // k-half kq % 2 of the slice: 64 consecutive bytes
    const uint32_t lane0 = (4 * q) % 32 + 32 * (kq % 2);
    int8_t* dst = Dt + (((size_t)kb * DT + q / 8) * 2 + kq / 2) * 1024 + (size_t)lane0 * 16;
#pragma unroll
    for (int d = 0; d < 4; ++d)
        *reinterpret_cast<int4*>(dst + 16 * d) = make_int4(pl[d][0], pl[d][1], pl[d][2], pl[d][3]);
}

// global_load_dwordx4 with the non-temporal hint, as inline assembly (see
// load16): W is streamed once per launch.
__device__ __forceinline__ void load16_nt(v4i& dst, const void* src) {
    asm volatile("global_load_dwordx4 %0, %1, off nt" : "=v"(dst) : "v"(src) : "memory");
}

typedef int v16i __attribute__((ext_vector_type(16)));

template <int DT, int NR, int WQ, int S>
__global__ __launch_bounds__(NR * WQ * 64) void server_eval_mfma_x32(const int8_t* __restrict__ W, uint32_t m,
                                                                     uint32_t n, const int8_t* __restrict__ Dt,
                                                                     uint32_t nkb, uint32_t B, const YOut Y) {
    // NR row groups x WQ digit groups of waves: wave (wr, wq) multiplies the
    // 32 rows of row group wr by digit tiles [wq*DW, (wq+1)*DW)
    constexpr int NW = NR * WQ, DW = DT / WQ;
    constexpr int NT = 2 * DT;                  // digit tiles per k-block
    constexpr int AD = (NT + NW - 1) / NW;      // digit tiles a wave loads per k-block
    constexpr int PER = AD + 2;                 // loads per wave per k-block
    static_assert(DW * WQ == DT, "digit split");
    static_assert(S * PER <= 63, "vmcnt range");
    static_assert(S >= 2, "ring depth");
    __shared__ __align__(16) int8_t Dring[S][NT][1024];
    const uint32_t rb = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wr = wave / WQ, wq = wave % WQ;
    // this lane's W row: 32 rows per row group, row tile (lane % 32) / 16 of the pair
    const uint32_t nrt = (m + 15) / 16;
    const uint32_t rt = (rb * NR + wr) * 2 + ((lane & 31) >> 4);
    const uint32_t rtc = rt < nrt ? rt : nrt - 1;  // rows past the end re-read the last tile (not stored)
    const int8_t* wrow = W + (size_t)rtc * nkb * 1024 + (size_t)((lane & 15) + 16 * (lane >> 5)) * 16;
    v4i wreg[S][2];
    // k-block j into ring slot `slot` (blocks past the end re-read the last
    // one, never consumed)
    auto issue = [&](uint32_t j, int slot) {
        const uint32_t kb = j < nkb ? j : nkb - 1;
#pragma unroll
        for (int a = 0; a < AD; ++a) {
            const int tile = (wave * AD + a) % NT;
            dma16(Dt + ((size_t)kb * NT + tile) * 1024 + (size_t)lane * 16, &Dring[slot][tile][0]);
        }
        // k-slice h of the block: 16-byte chunks 2h and 2h+1 of the packed tile
#pragma unroll
        for (int h = 0; h < 2; ++h) load16_nt(wreg[slot][h], wrow + (size_t)kb * 1024 + (size_t)h * 512);
    };
    v16i acc[DW];
#pragma unroll
    for (int d = 0; d < DW; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[d][e] = 0;
#pragma unroll
    for (int j = 0; j < S; ++j) issue(j, j);
    for (uint32_t j0 = 0; j0 < nkb; j0 += S) {
#pragma unroll
        for (int sl = 0; sl < S; ++sl) {
            const uint32_t j = j0 + sl;
            if (j < nkb) {
                wait_vmcnt<(S - 1) * PER>();  // this wave's loads of k-block j landed
                pin_vgpr(wreg[sl][0]);
                pin_vgpr(wreg[sl][1]);
                __syncthreads();  // every wave's digit tiles of k-block j landed
                // all of the block's digit operands are read before the first
                // MFMA (one LDS latency per block instead of one per MFMA)
                v4i a[2][DW];
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int d = 0; d < DW; ++d)
                        a[h][d] = *reinterpret_cast<const v4i*>(&Dring[sl][2 * (wq * DW + d) + h][16 * lane]);
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int d = 0; d < DW; ++d) pin_vgpr(a[h][d]);
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int d = 0; d < DW; ++d)
                        acc[d] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[h][d], wreg[sl][h], acc[d], 0, 0, 0);
                __syncthreads();  // every wave has read the slot: refill it
                issue(j + S, sl);
            }
        }
    }
    wait_vmcnt<0>();  // drain the trailing prefetches before the registers are reused or the workgroup exits
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
        pin_vgpr(wreg[sl][0]);
        pin_vgpr(wreg[sl][1]);
    }
    const uint32_t row = (rb * NR + wr) * 32 + (lane & 31);
#pragma unroll
    for (int d = 0; d < DW; ++d)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const uint32_t q = 8 * (wq * DW + d) + 2 * g + (uint32_t)(lane >> 5);
            const v4i s4 = {acc[d][4 * g], acc[d][4 * g + 1], acc[d][4 * g + 2], acc[d][4 * g + 3]};
            if (q < B && row < m) *Y.at(q, row) = digits_to_field(s4);
        }
}

// server_eval_mfma_x32 for a launch group of 17..32 queries (qt = 8 digit
// tiles of 16 rows, four 32-row digit tiles): digits32_kernel into Dt, then
// one workgroup per 128 rows.  (Measured at 28672 x 8192: 32 queries 57 us
// against 65 us for the streamed kernel; with 64 queries, eight 32-row digit
// tiles per wave, 89 us against 78, so those stay on the streamed kernel.)
constexpr int kX32RowGroups = 4, kX32Slots = 4;
constexpr uint32_t kX32Rows = 32 * kX32RowGroups;
hipError_t launch_x32(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t nkb, uint32_t B,
                      const YOut& Y, int8_t* Dt, hipStream_t s) {
    constexpr uint32_t DT = 4;
    if (B > DT * 8) return hipErrorInvalidValue;
    const uint32_t threads = nkb * DT * 8 * 4;
    if (n % 16 == 0 && (uintptr_t)X % 16 == 0)
        hipLaunchKernelGGL(digits32_kernel<true>, dim3(ceil_div(threads, 256)), dim3(256), 0, s, X, n, B, DT, nkb,
                           Dt);
    else
        hipLaunchKernelGGL(digits32_kernel<false>, dim3(ceil_div(threads, 256)), dim3(256), 0, s, X, n, B, DT, nkb,
                           Dt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((server_eval_mfma_x32<DT, kX32RowGroups, 1, kX32Slots>), dim3(ceil_div(m, kX32Rows)),
                       dim3(kX32RowGroups * 64), 0, s, W, m, n, Dt, nkb, B, Y);
    return hipGetLastError();
}

// The wide-tile kernel takes a launch group of packed W with 17..32 queries
// when its row blocks alone fill the chip (no k is split).
bool takes_x32(uint32_t m, uint32_t qt, bool packed) {
    return packed && qt == 8 && ceil_div(m, kX32Rows) >= 192;
}

template <int QT, int WQ, int TWW, int S>
hipError_t launch_stream_cfg(const int8_t* W, uint32_t m, uint32_t n, const int8_t* Dt, uint32_t nkb, uint32_t B,
                             const YOut& Y, uint32_t ksplit, uint32_t* part, uint32_t* counters, bool packed,
                             hipStream_t s) {
    constexpr uint32_t rows = (kStreamWaves / WQ) * TWW * 16;
    const uint32_t nrb = ceil_div(m, rows), per_group = 8 / ksplit;
    const dim3 grid(ceil_div(nrb, per_group) * 8);
    if (packed)
        hipLaunchKernelGGL((server_eval_mfma_stream<QT, kStreamWaves, WQ, TWW, S, true>), grid,
                           dim3(kStreamWaves * 64), 0, s, W, m, n, Dt, nkb, ksplit, B, Y, part, counters);
    else
        hipLaunchKernelGGL((server_eval_mfma_stream<QT, kStreamWaves, WQ, TWW, S, false>), grid,
                           dim3(kStreamWaves * 64), 0, s, W, m, n, Dt, nkb, ksplit, B, Y, part, counters);
    return hipGetLastError();
}

// Packed W: granule (rt, kb, l) = the 16 bytes lane l supplies as the B
// operand for rows 16*rt .. 16*rt + 15 and k-block kb, i.e. row 16*rt + l%16 at
// k = 64*kb + 16*(l/16) + [0, 16); rows >= m and k >= n are zero.
__global__ __launch_bounds__(256) void pack_w_kernel(const int8_t* __restrict__ W, uint32_t m, uint32_t n,
                                                     uint32_t nkb, size_t granules, int8_t* __restrict__ Wp) {
    const size_t g = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (g >= granules) return;
    const uint32_t l = (uint32_t)(g % 64), kb = (uint32_t)((g / 64) % nkb);
    const uint32_t rt = (uint32_t)(g / (64 * (size_t)nkb));
    const uint32_t row = rt * 16 + (l & 15), k0 = kb * 64 + (l >> 4) * 16;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (row < m) {
        const int8_t* src = W + (size_t)row * n;
        if (k0 + 16 <= n && (((uintptr_t)(src + k0)) & 15) == 0) {
            const uint4 t = *reinterpret_cast<const uint4*>(src + k0);
            w[0] = t.x;
            w[1] = t.y;
            w[2] = t.z;
            w[3] = t.w;
        } else {
            for (uint32_t e = 0; e < 16 && k0 + e < n; ++e)
                w[e >> 2] |= (uint32_t)(uint8_t)src[k0 + e] << (8 * (e & 3));
        }
    }
    *reinterpret_cast<uint4*>(Wp + g * 16) = make_uint4(w[0], w[1], w[2], w[3]);
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

namespace {
uint32_t group_qt(uint32_t nb) { return nb <= 8 ? 2 : nb <= 16 ? 4 : nb <= 32 ? 8 : 16; }
}  // namespace

size_t packed_w_bytes(uint32_t m, uint32_t n) { return (size_t)ceil_div(m, 16) * ceil_div(n, 64) * 1024; }

hipError_t launch_pack_w(const int8_t* W, uint32_t m, uint32_t n, int8_t* Wp, hipStream_t s) {
    const uint32_t nkb = ceil_div(n, 64);
    const size_t granules = (size_t)ceil_div(m, 16) * nkb * 64;
    hipLaunchKernelGGL(pack_w_kernel, dim3((uint32_t)((granules + 255) / 256)), dim3(256), 0, s, W, m, n, nkb,
                       granules, Wp);
    return hipGetLastError();
}

namespace {
// How one launch group of nb queries (4 < nb <= 64) is evaluated.
struct GroupPlan {
    bool dstat;     // digits-stationary kernel (else digit matrix + streamed kernel)
    uint32_t qt;    // digit tiles
    uint32_t tww;   // W tiles per wave (digits-stationary kernel)
    uint32_t rows;  // rows per workgroup
    uint32_t ks;    // k-ranges
    uint32_t kbm;   // k-blocks of digit tiles the LDS holds (digits-stationary kernel)
};

constexpr uint32_t kDstatKbm4 = 32, kDstatKbm2 = 64;  // k-blocks of digit tiles in 128 KiB of LDS

// LDS of the digits-stationary kernel sized to the k-range: the next power of
// two of its k-blocks, at least 8.  (A 16-query launch at 4096 x 4096 with four
// ranges of 16 k-blocks: 9.9 us with 64 KiB of LDS against 11.8 us with 128 KiB.)
uint32_t dstat_kbm(uint32_t kb_per) {
    uint32_t k = 8;
    while (k < kb_per) k *= 2;
    return k;
}

GroupPlan group_plan(uint32_t m, uint32_t n, uint32_t nb) {
    const uint32_t qt = group_qt(nb), nkb = ceil_div(n, 64);
    GroupPlan g{false, qt, 0, stream_rows(qt), stream_ksplit(m, n, qt), 0};
    if (qt > 4) return g;
    // digits-stationary: rows 128*tww, each k-range's digit tiles fit in LDS;
    // estimated time ceil(workgroups / 256) * (W k-blocks per workgroup in units
    // of 128 rows + fill + exchange of the split values, which the last
    // workgroup of a row block reads from the ks - 1 others)
    const uint32_t kbm = qt == 4 ? kDstatKbm4 : kDstatKbm2;
    uint32_t best = 0xffffffffu;
    for (uint32_t tww = 1; tww <= 2; ++tww)
        for (uint32_t ks = 1; ks <= 8; ks *= 2) {
            const uint32_t kb_per = ceil_div(nkb, ks);
            if (kb_per > kbm) continue;
            const uint32_t rows = 128 * tww, nwg = ceil_div(m, rows) * ks;
            const uint32_t cost = ceil_div(nwg, 256) * (kb_per * tww + 6 + qt * (ks - 1));
            if (cost < best) {
                best = cost;
                g = GroupPlan{true, qt, tww, rows, ks, dstat_kbm(kb_per)};
            }
        }
    return g;
}

template <int QT, int TWW, int KBM, int C, int NW>
hipError_t launch_dstat_cfg(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t nkb, uint32_t B,
                            const YOut& Y, uint32_t ksplit, unsigned long long* accum, bool packed,
                            hipStream_t s);

// Starting-block step of the digits-stationary kernel's k-walk per row tile
// (odd, so the starting blocks of a power-of-two k-range all differ).
// Measured on MI355X, the 128 server calls of a stack pass replayed
// alternately in one process: 1.736 ms without, 1.713 ms with step 7 (5:
// 1.716, 13: 1.726, 1: 1.737).
uint32_t dstat_rotation() { return 7u; }

// launch_dstat_cfg for the plan's LDS size (kbm a power of two in [8, KBM max])
template <int QT, int TWW, int NW>
hipError_t launch_dstat_kbm(uint32_t kbm, const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t nkb,
                            uint32_t B, const YOut& Y, uint32_t ksplit, unsigned long long* accum,
                            bool packed, hipStream_t s) {
    constexpr uint32_t kMax = QT == 4 ? kDstatKbm4 : kDstatKbm2;
    if (kbm == 8) return launch_dstat_cfg<QT, TWW, 8, 8, NW>(W, m, n, X, nkb, B, Y, ksplit, accum, packed, s);
    if (kbm == 16) return launch_dstat_cfg<QT, TWW, 16, 8, NW>(W, m, n, X, nkb, B, Y, ksplit, accum, packed, s);
    if (kbm == 32) return launch_dstat_cfg<QT, TWW, 32, 8, NW>(W, m, n, X, nkb, B, Y, ksplit, accum, packed, s);
    if constexpr (kMax >= 64)
        if (kbm == 64)
            return launch_dstat_cfg<QT, TWW, 64, 8, NW>(W, m, n, X, nkb, B, Y, ksplit, accum, packed, s);
    return hipErrorInvalidValue;
}

template <int QT, int TWW, int KBM, int C, int NW>
hipError_t launch_dstat_cfg(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t nkb, uint32_t B,
                            const YOut& Y, uint32_t ksplit, unsigned long long* accum, bool packed,
                            hipStream_t s) {
    if (ksplit == 0 || ceil_div(nkb, ksplit) > (uint32_t)KBM) return hipErrorInvalidValue;  // LDS holds the range
    if (ksplit > 1 && !accum) return hipErrorInvalidValue;
    const uint32_t nrb = ceil_div(m, 16 * NW * TWW), per_group = 8 / ksplit;
    const dim3 grid(ceil_div(nrb, per_group) * 8);
    const uint32_t rot = dstat_rotation();
    if (packed)
        hipLaunchKernelGGL((server_eval_mfma_dstat<QT, TWW, KBM, C, true, NW>), grid, dim3(NW * 64), 0, s, W, m, n,
                           X, nkb, ksplit, B, Y, accum, rot);
    else
        hipLaunchKernelGGL((server_eval_mfma_dstat<QT, TWW, KBM, C, false, NW>), grid, dim3(NW * 64), 0, s, W, m, n,
                           X, nkb, ksplit, B, Y, accum, rot);
    return hipGetLastError();
}
}  // namespace

ServerEvalPlan server_eval_plan(uint32_t m, uint32_t n, uint32_t B, int path, bool packed) {
    ServerEvalPlan pl{0, 0};
    if (path == MVK_PATH_VALU || B <= 4 || (!packed && n % 16 != 0)) return pl;
    const size_t nkb = ceil_div(n, 64);
    size_t dt_bytes = 0, part_bytes = 0;
    // launch groups hold 64 queries, the last one B % 64 (if nonzero)
    const uint32_t sizes[2] = {B < 64 ? B : 64u, B > 64 ? B % 64 : 0u};
    for (uint32_t nb : sizes) {
        if (nb == 0) continue;
        const GroupPlan g = group_plan(m, n, nb);
        if (!g.dstat) {
            const size_t db = (nkb * g.qt * 64 * 16 + 255) & ~(size_t)255;
            dt_bytes = db > dt_bytes ? db : dt_bytes;
        }
        if (g.ks > 1) {
            const size_t nrb = ceil_div(m, g.rows);
            if (g.dstat) {
                // one 64-bit accumulator per value of the row blocks (zero between launches)
                const size_t aw = nrb * g.rows * g.qt * 4 * 2;
                pl.ctrl_words = aw > pl.ctrl_words ? aw : pl.ctrl_words;
            } else {
                const size_t pb = (size_t)g.ks * nrb * g.rows * g.qt * 4 * 4;
                part_bytes = pb > part_bytes ? pb : part_bytes;
                pl.ctrl_words = nrb > pl.ctrl_words ? nrb : pl.ctrl_words;
            }
        }
    }
    pl.ws_bytes = dt_bytes + part_bytes;
    return pl;
}

hipError_t launch_server_eval_group(const int8_t* W, uint32_t G, uint32_t mg, uint32_t n, const uint32_t* X,
                                    uint32_t B, uint32_t* const* Ys, int path, bool packed, void* ws,
                                    uint32_t* counters, hipStream_t s) {
    if (G == 0 || G > kMaxGroup || (G > 1 && (!packed || path == MVK_PATH_VALU))) return hipErrorInvalidValue;
    YOut out{};
    for (uint32_t g = 0; g < G; ++g) out.y[g] = Ys[g];
    out.mg = mg;
    const uint32_t m = G * mg;  // rows of the stack
    uint32_t* const Y = Ys[0];
    if (path == MVK_PATH_VALU) {
        if (B == 1) return launch_cfg<16, 1>(W, m, n, X, B, Y, s);
        if (B == 2) return launch_cfg<8, 2>(W, m, n, X, B, Y, s);
        return launch_cfg<4, 4>(W, m, n, X, B, Y, s);
    }
    if (B == 1) return launch_mfma_small<1, 8, 8>(W, m, n, X, B, out, packed, s);
    if (B == 2) return launch_mfma_small<2, 8, 8>(W, m, n, X, B, out, packed, s);
    if (B <= 4) return launch_mfma_small<4, 8, 4>(W, m, n, X, B, out, packed, s);
    if (!packed && (n % 16 != 0 || (uintptr_t)W % 16 != 0)) {
        // Rows that are not whole 16-byte granules: the streamed path would read
        // past the end of W on the last row; use the small path per 4 queries.
        for (uint32_t b0 = 0; b0 < B; b0 += 4) {
            const uint32_t nb = (B - b0) < 4 ? (B - b0) : 4;
            const hipError_t e =
                launch_mfma_small<4, 8, 4>(W, m, n, X + (size_t)b0 * n, nb, yout_shift(out, b0), false, s);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    // Up to 64 queries per launch group; W is streamed once per group.
    const uint32_t nkb = ceil_div(n, 64);
    size_t dt_bytes = 0;
    for (uint32_t b0 = 0; b0 < B; b0 += 64) {
        const GroupPlan g = group_plan(m, n, (B - b0) < 64 ? (B - b0) : 64);
        if (!g.dstat) {
            const size_t db = (nkb * g.qt * 64 * 16 + 255) & ~(size_t)255;
            dt_bytes = db > dt_bytes ? db : dt_bytes;
        }
    }
    int8_t* Dt = (int8_t*)ws;
    // the digits-stationary kernel's split-k accumulators share the control
    // words with the streamed kernel's counters (each launch leaves them zero)
    unsigned long long* accum = reinterpret_cast<unsigned long long*>(counters);
    uint32_t* part = (uint32_t*)((char*)ws + dt_bytes);
    for (uint32_t b0 = 0; b0 < B; b0 += 64) {
        const uint32_t nb = (B - b0) < 64 ? (B - b0) : 64;
        const GroupPlan g = group_plan(m, n, nb);
        const uint32_t* Xb = X + (size_t)b0 * n;
        const YOut Yb = yout_shift(out, b0);
        hipError_t e = hipSuccess;
        if (g.dstat) {
            if (g.qt == 4)
                e = g.tww == 1 ? launch_dstat_kbm<4, 1, 8>(g.kbm, W, m, n, Xb, nkb, nb, Yb, g.ks, accum,
                                                           packed, s)
                               : launch_dstat_kbm<4, 2, 8>(g.kbm, W, m, n, Xb, nkb, nb, Yb, g.ks, accum,
                                                           packed, s);
            else
                e = g.tww == 1 ? launch_dstat_kbm<2, 1, 8>(g.kbm, W, m, n, Xb, nkb, nb, Yb, g.ks, accum,
                                                           packed, s)
                               : launch_dstat_kbm<2, 2, 8>(g.kbm, W, m, n, Xb, nkb, nb, Yb, g.ks, accum,
                                                           packed, s);
            if (e != hipSuccess) return e;
            continue;
        }
        const uint32_t qt = g.qt, ks = g.ks;
        if (takes_x32(m, qt, packed)) {
            e = launch_x32(W, m, n, Xb, nkb, nb, Yb, Dt, s);
            if (e != hipSuccess) return e;
            continue;
        }
        const uint32_t threads = nkb * qt * 16;
        if (n % 16 == 0 && (uintptr_t)Xb % 16 == 0)
            hipLaunchKernelGGL(digits_tiled_kernel<true>, dim3(ceil_div(threads, 256)), dim3(256), 0, s, Xb, n, nb,
                               qt, nkb, Dt);
        else
            hipLaunchKernelGGL(digits_tiled_kernel<false>, dim3(ceil_div(threads, 256)), dim3(256), 0, s, Xb, n, nb,
                               qt, nkb, Dt);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (qt == 2)
            e = launch_stream_cfg<2, 1, 2, kStreamSlots>(W, m, n, Dt, nkb, nb, Yb, ks, part, counters, packed, s);
        else if (qt == 4)
            e = launch_stream_cfg<4, 1, 2, kStreamSlots>(W, m, n, Dt, nkb, nb, Yb, ks, part, counters, packed, s);
        else if (qt == 8)
            e = launch_stream_cfg<8, 2, 4, kStreamSlots>(W, m, n, Dt, nkb, nb, Yb, ks, part, counters, packed, s);
        else
            e = launch_stream_cfg<16, 4, 7, kStreamSlots>(W, m, n, Dt, nkb, nb, Yb, ks, part, counters, packed, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_server_eval(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t B,
                              uint32_t* Y, int path, bool packed, void* ws, uint32_t* counters, hipStream_t s) {
    return launch_server_eval_group(W, 1, m, n, X, B, &Y, path, packed, ws, counters, s);
}

}  // namespace mvk
