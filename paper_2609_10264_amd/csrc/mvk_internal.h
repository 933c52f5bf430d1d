// Internal launch interface between the C-ABI layer (api.hip) and the kernel
// translation units.  Every launcher only enqueues work on `s` and returns the
// status of hipGetLastError().
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mvk.h"

namespace mvk {

// server_eval.hip
// What launch_server_eval needs besides its arguments: ws_bytes of workspace
// and ctrl_words of counters that are zero before the launch (every launch
// leaves them at zero).
struct ServerEvalPlan {
    size_t ws_bytes;
    size_t ctrl_words;
};
ServerEvalPlan server_eval_plan(uint32_t m, uint32_t n, uint32_t B, int path, bool packed);
// W: row-major m x n, or (packed) the layout written by launch_pack_w.
hipError_t launch_server_eval(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* X, uint32_t B,
                              uint32_t* Y, int path, bool packed, void* ws, uint32_t* counters, hipStream_t s);
// G (<= kMaxGroup) matrices of mg x n sharing the queries X: W is the packed
// layout of their row stack (G * mg rows; mg a multiple of 16 when G > 1) and
// Ys[g] (B x mg) receives matrix g's product.  Plan with m = G * mg.
constexpr uint32_t kMaxGroup = MVK_MAX_GROUP;
hipError_t launch_server_eval_group(const int8_t* W, uint32_t G, uint32_t mg, uint32_t n, const uint32_t* X,
                                    uint32_t B, uint32_t* const* Ys, int path, bool packed, void* ws,
                                    uint32_t* counters, hipStream_t s);
// Packed W: ceil(m/16) * ceil(n/64) tiles of 1 KiB in MFMA operand order.
size_t packed_w_bytes(uint32_t m, uint32_t n);
hipError_t launch_pack_w(const int8_t* W, uint32_t m, uint32_t n, int8_t* Wp, hipStream_t s);

// raa.hip -------------------------------------------------------------------
// G^T applied to `nvec` vectors whose element i of vector v sits at
// in[i*ld_in + v*vs_in]; result element j of vector v goes to
// out[j*ld_out + v*vs_out].  t3: scratch of N*nvec uint32 (N = r*k); seg:
// scratch of encT_seg_words(N, nvec) uint32.
size_t encT_seg_words(size_t N, size_t nvec);
// Vectors per call of the batched encoder (at least 64 per workgroup row, 65535 rows).
constexpr uint32_t kMaxEncVectors = 65535u * 64u;
hipError_t launch_encT_u32(const mvk_code& c, const uint32_t* in, size_t ld_in, size_t vs_in, uint32_t nvec,
                           uint32_t* t3, uint32_t* seg, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s);
hipError_t launch_encT_i8(const mvk_code& c, const int8_t* in, size_t ld_in, size_t vs_in, uint32_t nvec,
                          uint32_t* t3, uint32_t* seg, uint32_t* out, size_t ld_out, size_t vs_out, hipStream_t s);
// Block lengths above this value run the syndrome in segments of kSynSegLen
// positions (several workgroups per vector) and need syn_scratch_bytes(count,
// N) bytes of scratch; up to it the syndrome runs in LDS and needs none.
constexpr size_t kSynScratchAbove = 16384;
constexpr size_t kSynSegLen = 1024;
// Two work arrays of N words per vector, then per vector a ticket word and one
// status word per segment (64-bit each).
inline size_t syn_scratch_bytes(size_t count, size_t N) {
    if (N <= kSynScratchAbove) return 0;
    const size_t nseg = (N + kSynSegLen - 1) / kSynSegLen;
    return count * (2 * N * sizeof(uint32_t) + (nseg + 1) * sizeof(uint64_t));
}
// G v for `count` vectors: dense (v: count x N) or sparse (idx/val: count x t).
// If X != nullptr the result is added to X (out = X + G v), as in Encrypt.
// scratch: syn_scratch_bytes(count, N), 8-byte aligned.
hipError_t launch_syn_dense(const mvk_code& c, const uint32_t* v, uint32_t count, uint32_t* scratch,
                            uint32_t* out, hipStream_t s);
hipError_t launch_syn_sparse(const mvk_code& c, const uint32_t* idx, const uint32_t* val, uint32_t t,
                             uint32_t count, const uint32_t* X, uint32_t* scratch, uint32_t* out,
                             hipStream_t s);
// Sparse syndromes of long blocks (N > kSynScratchAbove) of several codes in
// one sequence of three launches: set i is `count` vectors (idx/val: count x
// t) over code *c, results into out (count x c->k).  scratch: scratch_bytes
// of at least syn_sets_scratch_bytes(sets, S), 256-byte aligned (else
// hipErrorInvalidValue and nothing is launched).
struct SynSet {
    const mvk_code* c;
    const uint32_t *idx, *val;
    uint32_t t, count;
    uint32_t* out;
};
constexpr uint32_t kMaxSynSets = 16;
size_t syn_sets_scratch_bytes(const SynSet* sets, uint32_t S);
hipError_t launch_syn_sets(const SynSet* sets, uint32_t S, uint32_t* scratch, size_t scratch_bytes, hipStream_t s);
// W (m x n int8) -> WT (n x m int8)
hipError_t launch_transpose_i8(const int8_t* W, uint32_t m, uint32_t n, int8_t* WT, hipStream_t s);
hipError_t launch_fill_u32(uint32_t* p, size_t count, uint32_t value, hipStream_t s);

// client.hip ----------------------------------------------------------------
constexpr uint32_t kClientBlock = 256;  // threads per workgroup of the gather kernels
constexpr uint32_t kClientCols = 64;    // output columns per workgroup of the gather kernels
// Decrypt + Verify in one launch (see client.hip).  r: ell x m words,
// r_q = Gy e_q.  ctrl: dv_ctrl_bytes(m, n, B, ell) bytes of control region
// (completion counters, then the 64-bit accumulators), zero before the first
// launch and left at zero by every launch of the three decode/verify kernels.
// ell <= kMaxEll.
constexpr uint32_t kMaxEll = 16;
size_t dv_ctrl_bytes(uint32_t m, uint32_t n, uint32_t B, uint32_t ell);
hipError_t launch_decode_verify(const uint32_t* PT, const uint32_t* Q, uint32_t m, uint32_t n, uint32_t Nx,
                                uint32_t Ny, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx, const uint32_t* ey_idx,
                                const uint32_t* ey_val, uint32_t ty, uint32_t ell, const uint32_t* r, uint32_t* Y,
                                uint32_t* ctrl, uint32_t* vL, uint32_t* vR, uint32_t* accept, hipStream_t s);

// The same with the challenge syndromes r_q = Gy e_q computed in the launch
// (written to r, ell x m words) by 512-thread workgroups that hold a whole
// block of Ny = cyr * m positions in LDS.  ctrl as above; its words 1 and 2
// hold the syndrome completion count and the wait time-out flag.
// dv_decode_cols: output columns per lane of the decode role these launches
// pick (4 when m % 4 == 0, PT, Yhat, Y and r are 16-byte aligned and the
// B * ceil(m / 256) decode workgroups fill the chip, else 1).
// dv_syn_fits: the launch applies (Ny small enough, every workgroup resident
// at once on the current device), for the decode width E = dv_decode_cols.
constexpr uint32_t kDvSynThreads = 512;
uint32_t dv_syn_u(uint32_t Ny);
uint32_t dv_decode_cols(uint32_t m, uint32_t B, const void* PT, const void* Yhat, const void* Y, const void* r);
bool dv_syn_fits(uint32_t m, uint32_t n, uint32_t Ny, uint32_t B, uint32_t ell, uint32_t E);
hipError_t launch_decode_verify_syn(const uint32_t* PT, const uint32_t* Q, uint32_t m, uint32_t n, uint32_t Nx,
                                    uint32_t Ny, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                    const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx,
                                    const uint32_t* ey_idx, const uint32_t* ey_val, uint32_t ty, uint32_t ell,
                                    uint32_t cyr, const uint32_t* pi1, const uint32_t* pi2, const uint32_t* v1,
                                    const uint32_t* v2, uint32_t* r, uint32_t* Y, uint32_t* ctrl, uint32_t* vL,
                                    uint32_t* vR, uint32_t* accept, hipStream_t s);

// decode_verify with the output masks My (B x m) and the vectors u_q (U,
// ell x n) from client_prepare in place of the gathers.
hipError_t launch_decode_verify_masked(uint32_t m, uint32_t n, const uint32_t* Xhat, const uint32_t* Yhat,
                                       uint32_t B, const uint32_t* My, uint32_t ell, const uint32_t* r,
                                       const uint32_t* U, uint32_t* Y, uint32_t* ctrl, uint32_t* vL, uint32_t* vR,
                                       uint32_t* accept, hipStream_t s);

// The same for G <= kMaxGroup problems sharing Xhat (one launch where the
// problem takes the wide kernel, else one per problem); ctrl: G control
// regions of dv_group_ctrl_stride words each.  vL, vR may be null.
size_t dv_group_ctrl_stride(uint32_t m, uint32_t n, uint32_t B, uint32_t ell);
// The decode/verify of one response and the masked encode of the next,
// independent query in one launch where the decode/verify takes its small
// form (else two launches); ctrl as launch_decode_verify_masked, add_counter
// as launch_add_masks (distinct words).
hipError_t launch_client_turn(uint32_t m, uint32_t n, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                              const uint32_t* My, uint32_t ell, const uint32_t* r, const uint32_t* U, uint32_t* Y,
                              uint32_t* ctrl, uint32_t* vL, uint32_t* vR, uint32_t* accept, const uint32_t* Xn,
                              const uint32_t* Mxn, size_t countn, uint32_t* Xhatn, uint32_t* flag, uint32_t value,
                              uint32_t timeout_us, uint32_t* timed_out, uint32_t* add_counter, hipStream_t s);
hipError_t launch_decode_verify_masked_group(uint32_t G, uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B,
                                             const uint32_t* const* Yhat, const uint32_t* const* My, uint32_t ell,
                                             const uint32_t* const* R, const uint32_t* const* U, uint32_t* const* Y,
                                             uint32_t* const* vL, uint32_t* const* vR, uint32_t* const* accept,
                                             uint32_t* ctrl, hipStream_t s);

// prepare.hip ---------------------------------------------------------------
// Mx, My for nx noise vectors and R, U for ny challenges (either count may
// be 0).  scratch: scratch_bytes of at least prep_scratch_bytes (the work
// regions of the syndromes longer than kSynScratchAbove, one after another).  done (may be null): set to
// done_value once every output is stored and visible device-wide; counter:
// prep_ctrl_words(key, nx, ny) words of completion counters (count.h), zero
// before the launch (left zero).
size_t prep_ctrl_words(const mvk_key& key, uint32_t nx, uint32_t ny);
// Several inputs and the keys they feed in one launch (at most kMaxPrep of
// each): input j holds `count` noise vectors of `t` terms over the privacy
// code cx (Mx: count x cx->k); key g the output masks My of the noise of input
// `in` (kPrepNoInput: none) and `count` challenges with R, U.  Syndromes
// longer than kSynScratchAbove run first in their own launches (scratch of
// prep_scratch_bytes); done: ndone device words, each set to done_value once
// every output is stored and visible device-wide; counter: prep_ctrl_words
// words, zero before the launch (left zero).
constexpr uint32_t kMaxPrep = MVK_MAX_PREP;
constexpr uint32_t kPrepNoInput = 0xffffffffu;
struct PrepInputDesc {
    const mvk_code* cx;
    const uint32_t *idx, *val;
    uint32_t t, count;
    uint32_t* Mx;
};
struct PrepProbDesc {
    const mvk_key* key;
    uint32_t in;
    const uint32_t *idx, *val;
    uint32_t t, count;
    uint32_t *My, *R, *U;
};
size_t prep_ctrl_words(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G);
size_t prep_scratch_bytes(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G);
// the same for G keys sharing one input of nx noise vectors, ny challenges each
size_t prep_scratch_bytes(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny);
hipError_t launch_client_prepare_multi(const PrepInputDesc* ins, uint32_t NI, const PrepProbDesc* probs, uint32_t G,
                                       uint32_t* scratch, size_t scratch_bytes, uint32_t* counter,
                                       uint32_t* const* done, uint32_t ndone, uint32_t done_value, hipStream_t s);
size_t prep_ctrl_words(const mvk_key* const* keys, uint32_t G, uint32_t nx, uint32_t ny);
// The same for G <= kMaxGroup keys of one shape and one privacy code that share
// the noise vectors (Mx once; My[g], R[g], Uq[g] per key, with the challenges
// ey_idx[g], ey_val[g]).
hipError_t launch_client_prepare_group(uint32_t G, const mvk_key* const* keys, const uint32_t* ex_idx,
                                       const uint32_t* ex_val, uint32_t tx, uint32_t nx,
                                       const uint32_t* const* ey_idx, const uint32_t* const* ey_val, uint32_t ty,
                                       uint32_t ny, uint32_t* Mx, uint32_t* const* My, uint32_t* const* R,
                                       uint32_t* const* Uq, uint32_t* scratch, size_t scratch_bytes,
                                       uint32_t* counter, uint32_t* done, uint32_t done_value, hipStream_t s);
hipError_t launch_client_prepare(const mvk_key& key, const uint32_t* ex_idx, const uint32_t* ex_val, uint32_t tx,
                                 uint32_t nx, const uint32_t* ey_idx, const uint32_t* ey_val, uint32_t ty,
                                 uint32_t ny, uint32_t* Mx, uint32_t* My, uint32_t* R, uint32_t* Uq,
                                 uint32_t* scratch, size_t scratch_bytes, uint32_t* counter, uint32_t* done,
                                 uint32_t done_value, hipStream_t s);
// Xhat = X + Mx; with a flag, after waiting for *flag == value (which the
// launch then clears; counter as above).
hipError_t launch_add_masks(const uint32_t* X, const uint32_t* Mx, size_t count, uint32_t* Xhat, uint32_t* flag,
                            uint32_t value, uint32_t timeout_us, uint32_t* timed_out, uint32_t* counter,
                            hipStream_t s);
// out[v][:] = sum_s val[v*t+s] * M[idx[v*t+s], :] for `count` sparse vectors
// (M: nrows x ld, row-major).
hipError_t launch_gather_rows(const uint32_t* M, uint32_t ld, uint32_t nrows, const uint32_t* idx,
                              const uint32_t* val, uint32_t t, uint32_t count, uint32_t* out, hipStream_t s);
hipError_t launch_flag_signal(uint32_t* flag, uint32_t value, hipStream_t s);
hipError_t launch_flag_wait(uint32_t* flag, uint32_t value, uint32_t timeout_us, uint32_t* timed_out,
                            hipStream_t s);

// batch.hip -----------------------------------------------------------------
// Client checks of batch verification.  R: ell x m primary syndromes G e_q;
// Rs: ell2 x Bn secondary syndromes G' e'_j; ctrl: batch_ctrl_bytes(...) of
// control region.
hipError_t launch_batch_check(uint32_t m, uint32_t n, uint32_t B, const uint32_t* X, const uint32_t* Y,
                              const uint32_t* Ut, const uint32_t* R, const uint32_t* Rs, const uint32_t* Qaux,
                              uint32_t N, uint32_t N2, const uint32_t* e_idx, const uint32_t* e_val, uint32_t t,
                              uint32_t ell, const uint32_t* e2_idx, const uint32_t* e2_val, uint32_t t2,
                              uint32_t ell2, uint32_t* ctrl, uint32_t* vL, uint32_t* vR, uint32_t* sL, uint32_t* sR,
                              uint32_t* accept, hipStream_t s);
// Control bytes of launch_batch_check (completion counters, then the 64-bit
// accumulators), zero before the launch and left at zero.
size_t batch_ctrl_bytes(uint32_t m, uint32_t n, uint32_t B, uint32_t ell, uint32_t ell2);

// validate.hip --------------------------------------------------------------
// Adds to *out the number of words of a[0, count) that are >= p.
hipError_t launch_count_noncanonical(const uint32_t* a, size_t count, uint32_t* out, hipStream_t s);

// calib.hip -----------------------------------------------------------------
// Streaming read of bytes (a multiple of 16) at data; sink: sink_words words
// (at least 256), their XOR is the XOR of the buffer's words.
hipError_t launch_stream_read(const void* data, size_t bytes, uint32_t* sink, uint32_t sink_words, hipStream_t s);

// seeded.hip ----------------------------------------------------------------
// The sampling specification of sample.h.  Host: a code's four arrays (N = k*r
// words each) and `count` sparse vectors (count x t each, t <= N).  Device:
// the same sparse vectors, one lane per vector.
void sample_code_host(uint32_t k, uint32_t r, uint64_t seed, uint64_t tag, uint32_t* pi1, uint32_t* pi2,
                      uint32_t* v1, uint32_t* v2);
void sample_sparse_host(uint32_t count, uint32_t N, uint32_t t, uint64_t seed, uint64_t tag, uint32_t* idx,
                        uint32_t* val);
hipError_t launch_sample_sparse(uint64_t seed, uint64_t tag, uint32_t count, uint32_t N, uint32_t t, uint32_t* idx,
                                uint32_t* val, hipStream_t s);

inline uint32_t ceil_div(uint32_t a, uint32_t b) { return (a + b - 1) / b; }

}  // namespace mvk
