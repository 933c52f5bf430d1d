/*
 * mvk.h -- C ABI of the MI355X (gfx950) library for the data-parallel hot path
 * of private and verifiable matrix-vector multiplication delegation (pvMVMD,
 * "Maverick", arxiv 2609.10264).
 *
 * Field: F_p.  Two builds of the same sources implement this ABI, one per
 * field: libmvk.so over p = 2^31 - 1 (MVK_PRIME) and libmvk_bb.so over the
 * BabyBear prime q = 15 * 2^27 + 1 (MVK_PRIME_BABYBEAR), the field of the
 * paper's evaluation (Sec. 7.1).  mvk_field_modulus() names the build's p;
 * everything below holds for either.  A "field array" is uint32 in canonical
 * form [0, p).  The public matrix W is int8 (each entry w is the field element
 * w mod p; Sec. 7.2 embeds quantised signed integers into the field).
 *
 * Conventions shared by every call
 *  - Pointers marked "device" are HIP device pointers (any allocator); the
 *    caller owns every buffer it passes and must keep it alive until the work
 *    enqueued on `stream` has completed.  Pointers marked "host" are ordinary
 *    host memory read during the call.
 *  - `stream` is a hipStream_t passed as void*; NULL means the default stream.
 *    All calls only enqueue work on `stream` and return without waiting for it.
 *  - Matrices are row-major.  A batch of B vectors of length L is B x L (vector b
 *    starts at element b*L).
 *  - Return value: MVK_OK, or a negative mvk_status.  On an error nothing has
 *    been enqueued unless the status is MVK_EHIP (a launch failed; the stream
 *    may hold part of the work and the outputs are undefined).
 *  - Inputs are not validated on the device: field inputs must be < p and
 *    permutations / sparse positions must be in range, or the outputs are
 *    undefined (out-of-range indices are clamped, never dereferenced).
 *    With MVK_VALIDATE=1 in the environment, mvk_server_eval*, mvk_encode,
 *    mvk_decode_verify*, mvk_verify, mvk_encode_masked and
 *    mvk_decode_verify_masked first check that their field inputs are
 *    canonical, waiting for the stream, and return MVK_ERANGE (nothing else
 *    enqueued) if one is not; a debugging mode, not for graph capture.
 *  - The library keeps a per-(device, stream) workspace that grows on demand
 *    (hipMalloc at first use and when a larger size is needed); calls enqueued
 *    on two different streams never share workspace memory.  A buffer that a
 *    growth replaces is retired, not freed, so HIP graphs captured earlier on
 *    the stream (which hold its address) stay valid; mvk_workspace_release
 *    frees the retired buffers.  A call whose stream is capturing a graph and
 *    that would need a larger workspace returns MVK_ECAPTURE (run it once
 *    outside the capture first).  Calls on one stream from several host
 *    threads at once are not supported: give each thread its own stream.
 */
#ifndef MVK_H_
#define MVK_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MVK_PRIME 2147483647u
#define MVK_PRIME_BABYBEAR 2013265921u
#define MVK_ABI_VERSION 9

typedef int32_t mvk_status;
#define MVK_OK 0
#define MVK_EINVAL (-1) /* missing pointer, zero or inconsistent size */
#define MVK_ERANGE (-2) /* a size beyond the exactness limit of a kernel, or (MVK_VALIDATE) a field input >= p */
#define MVK_ENOMEM (-3) /* workspace allocation failed */
#define MVK_EHIP (-4)   /* a HIP runtime call or kernel launch failed */
#define MVK_ERANDOM (-5)   /* the operating system's random source failed (MVK_SEED_FRESH) */
#define MVK_ECAPTURE (-6)  /* the workspace would have to grow while the stream captures a graph */

/* Largest column count n of W for which server_eval's int8-limb accumulation
 * is exact: n * 128 * 128 < 2^31. */
#define MVK_MAX_N 131071u

/*
 * Description of an RAA code (App. B): G = R Pi1 V1 A Pi2 V2 A in F^{k x N},
 * N = r*k.  R repeats every entry r times (positions i*r .. i*r+r-1 hold entry
 * i), Pi has Pi[i][j] = 1 iff pi(j) = i, V = diag(v), A is upper triangular
 * all-ones.  pi1, pi2: device, N uint32 each, permutations of [0, N).
 * v1, v2: device, N uint32 each, values in [1, p-1].
 */
typedef struct mvk_code {
    uint32_t k;
    uint32_t r;
    const uint32_t *pi1;
    const uint32_t *pi2;
    const uint32_t *v1;
    const uint32_t *v2;
} mvk_code;

/*
 * Public parameters pp of Protocol pvMVMD (Preprocess):
 *   cx : privacy code, k = n, block length Nx = cx.r * n
 *   cy : verification code, k = m, block length Ny = cy.r * m
 *   PT : device, Nx x m field array, PT[j*m + i] = P[i][j] with P = W Gx
 *   Q  : device, Ny x n field array, Q = Gy^T W
 * PT and Q are written by mvk_keygen and read by mvk_decode_verify.
 */
typedef struct mvk_key {
    uint32_t m;
    uint32_t n;
    mvk_code cx;
    mvk_code cy;
    uint32_t *PT;
    uint32_t *Q;
} mvk_key;

/*
 * `count` sparse vectors of E_t^N (Sec. 3 notation: exactly t nonzeros).
 * idx, val: device, count x t uint32.  Row c lists the t distinct positions
 * (< N) and their nonzero values (in [1, p-1]) of vector c.
 */
typedef struct mvk_sparse {
    const uint32_t *idx;
    const uint32_t *val;
    uint32_t t;
    uint32_t count;
} mvk_sparse;

/* Human-readable name of a status code (static string). */
const char *mvk_status_str(mvk_status s);

/* MVK_ABI_VERSION of the loaded library. */
int32_t mvk_abi_version(void);

/* The prime p of the loaded build: MVK_PRIME or MVK_PRIME_BABYBEAR. */
uint32_t mvk_field_modulus(void);

/*
 * Server evaluation (Protocol pvMVMD: the server's only work is the field
 * matrix-vector product y^ = M x^, once per query column).
 *   W    : device, m x n int8, row-major (row i at W + i*n)
 *   Xhat : device, B x n field array (the masked queries)
 *   Yhat : device, B x m field array, written: Yhat[b][i] = sum_k W[i][k] Xhat[b][k] mod p
 * m == 0 or B == 0: no work.  n == 0: Yhat is zeroed.
 * Errors: MVK_EINVAL (null pointer), MVK_ERANGE (n > MVK_MAX_N, m or B at
 * least 2^31, W or Yhat above 2^62 bytes).
 */
mvk_status mvk_server_eval(const int8_t *W, uint32_t m, uint32_t n, const uint32_t *Xhat,
                           uint32_t B, uint32_t *Yhat, void *stream);

/* Kernel family for mvk_server_eval_path. */
#define MVK_PATH_AUTO 0 /* the library's choice (matrix-core path) */
#define MVK_PATH_VALU 1 /* v_dot4_i32_i8 on the vector ALUs, cross-lane reduction in software */
#define MVK_PATH_MFMA 2 /* v_mfma_i32_16x16x64_i8 on the matrix cores */

/*
 * mvk_server_eval with an explicit kernel family (same result bit for bit;
 * used to compare the two designs).  path: one of MVK_PATH_*.
 * Errors: as mvk_server_eval, plus MVK_EINVAL for an unknown path.
 */
mvk_status mvk_server_eval_path(const int8_t *W, uint32_t m, uint32_t n, const uint32_t *Xhat,
                                uint32_t B, uint32_t *Yhat, int32_t path, void *stream);

/*
 * Server-side weight layout.  The server may store W once in MFMA operand
 * order ("packed") instead of row-major: ceil(m/16) * ceil(n/64) tiles of
 * 1 KiB, tile (rt, kb) holding rows 16*rt .. 16*rt+15 and columns
 * 64*kb .. 64*kb+63 (zero beyond m and n), so that every W read of the server
 * product is a contiguous 1 KiB run.  The product is the same field matrix-vector
 * product as mvk_server_eval (Protocol pvMVMD, server step), bit for bit.
 *
 * mvk_packed_weight_bytes: size of the packed buffer (0 if m or n is 0).
 * mvk_pack_weights: W (device, m x n int8, row-major) -> Wp (device, caller
 *   allocated, mvk_packed_weight_bytes(m, n) bytes, 16-byte aligned).
 * mvk_server_eval_packed: as mvk_server_eval with W given packed.
 * Errors: MVK_EINVAL (null or misaligned pointer), MVK_ERANGE (n > MVK_MAX_N).
 */
size_t mvk_packed_weight_bytes(uint32_t m, uint32_t n);
mvk_status mvk_pack_weights(const int8_t *W, uint32_t m, uint32_t n, int8_t *Wp, void *stream);
mvk_status mvk_server_eval_packed(const int8_t *Wp, uint32_t m, uint32_t n, const uint32_t *Xhat,
                                  uint32_t B, uint32_t *Yhat, void *stream);

/*
 * Several matrices of one shape applied to the same queries in one launch
 * (for example the q, k and v projections of a decoder layer, which share
 * their input): Yhat[g] = W_g Xhat mod p for g < G, bit for bit the products
 * G calls of mvk_server_eval_packed would give (Protocol pvMVMD, server step,
 * once per matrix).  The server stores the G matrices as the packed layout of
 * their row stack [W_0; W_1; ...] ((G*m) x n): mvk_pack_weights of the stacked
 * matrix, or G packed buffers of mvk_packed_weight_bytes(m, n) bytes placed
 * back to back (the same bytes when m is a multiple of 16).
 *   Wp   : device, packed (G*m) x n, 16-byte aligned
 *   G    : 1..MVK_MAX_GROUP; m must be a multiple of 16 when G > 1
 *   Xhat : device, B x n field array
 *   Yhat : host array of G device pointers, each B x m, written
 * Errors: MVK_EINVAL (null or misaligned pointer, G out of range, m not a
 * multiple of 16), MVK_ERANGE (as mvk_server_eval for m*G rows).
 */
#define MVK_MAX_GROUP 4u
mvk_status mvk_server_eval_packed_group(const int8_t *Wp, uint32_t G, uint32_t m, uint32_t n,
                                        const uint32_t *Xhat, uint32_t B, uint32_t *const *Yhat, void *stream);

/*
 * mvk_server_eval_packed for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same product, bit for bit, whose kernels keep their scratch
 * (the batched kernels' digit matrix, split-k partial sums and accumulators,
 * row-block counters) in a device array of the library of
 * MVK_STATIC_SCRATCH_BYTES + 64 KiB (control words first, at least 64 KiB of
 * them, then the data), held on every GPU the library runs on until the
 * process ends.  It calls no hipMalloc or hipFree.  The control words are
 * cleared by a kernel at every call.  Every call on one GPU shares that GPU's
 * array: calls that overlap in time on one GPU (two streams, two threads)
 * race and must be ordered by the caller.
 * Errors: as mvk_server_eval_packed, plus MVK_ERANGE when the shape's scratch
 * exceeds the array (28672 x 8192 with 64 queries needs about 16.7 MB).
 */
#define MVK_STATIC_SCRATCH_BYTES (32u << 20)
mvk_status mvk_server_eval_packed_static(const int8_t *Wp, uint32_t m, uint32_t n, const uint32_t *Xhat,
                                         uint32_t B, uint32_t *Yhat, void *stream);

/*
 * Preprocess (Protocol pvMVMD): writes key->PT = (W Gx)^T and key->Q = Gy^T W
 * (m encodings of the rows and n encodings of the columns of W, Sec. 6.3).
 *   key : host struct; key->m, key->n, the two codes and the PT, Q buffers
 *         must be set (cx.k == n, cy.k == m)
 *   W   : device, m x n int8
 * Uses a workspace of about m*n + max(Nx*m, Ny*n)*4 bytes (plus 2/256 of that
 * for the segment sums of the prefix scans).
 * Errors: MVK_EINVAL, MVK_ERANGE (a buffer size above 2^62 bytes, m or n above
 * 65535 * 64), MVK_ENOMEM.
 */
mvk_status mvk_keygen(const mvk_key *key, const int8_t *W, void *stream);

/*
 * Encrypt (Protocol pvMVMD): for every column b, x'_b = Gx e_b and
 * Xhat_b = X_b + x'_b, where e_b is sparse vector b of `ex`
 * (ex->count == B, positions < Nx).  The caller keeps `ex` as the secret
 * state st for decode.
 *   X    : device, B x n field array (plaintext queries)
 *   Xhat : device, B x n field array, written
 * Errors: MVK_EINVAL, MVK_ERANGE (B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_encode(const mvk_key *key, const uint32_t *X, uint32_t B, const mvk_sparse *ex,
                      uint32_t *Xhat, void *stream);

/*
 * Verify + Decrypt (Protocol pvMVMD) for B columns.
 *   Verify: for each repetition q < ey->count (= ell) with challenge e_q in
 *     E_ty^Ny (positions < Ny), v_L = (e_q^T Q) Xhat_b and
 *     v_R = e_q^T (Gy^T Yhat_b); column b is accepted iff v_L == v_R for every q.
 *     One challenge per repetition is shared by all columns (Sec. 5.4).
 *     The server must not learn the challenges before its responses are fixed.
 *   Decrypt: Y_b = Yhat_b - P e_b with e_b sparse vector b of `ex`
 *     (the state returned by encode).
 *   Xhat   : device, B x n;  Yhat : device, B x m (the server's responses)
 *   Y      : device, B x m, written (must be discarded where accept is 0)
 *   vL, vR : device, ell x B, written; may be NULL
 *   accept : device, B uint32, written 1 (accept) or 0 (reject)
 * A rejection is a result, not an error.  ell = ey->count must be 1..16.
 * Errors: MVK_EINVAL, MVK_ERANGE (ell > 16 or B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_decode_verify(const mvk_key *key, const uint32_t *Xhat, const uint32_t *Yhat,
                             uint32_t B, const mvk_sparse *ex, const mvk_sparse *ey,
                             uint32_t *Y, uint32_t *vL, uint32_t *vR, uint32_t *accept,
                             void *stream);

/*
 * Verify alone (Protocol vMVMD, Sec. 5.1; the verification-only mode of
 * Sec. 7): for plaintext queries X (B x n) and claimed results Y (B x m) of
 * the key's matrix, v_L = (e_q^T Q) x_b and v_R = (Gy e_q)^T y_b for every
 * repetition q; accept[b] = 1 iff they agree for every q.  The same check as
 * mvk_decode_verify without the decryption (the key's privacy code and PT are
 * not used).  vL, vR: device, ell x B, may be NULL.
 * Errors: MVK_EINVAL, MVK_ERANGE (ell > 16 or B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_verify(const mvk_key *key, const uint32_t *X, const uint32_t *Y, uint32_t B,
                      const mvk_sparse *ey, uint32_t *vL, uint32_t *vR, uint32_t *accept, void *stream);

/*
 * Verify, first half: the challenge syndromes R[q*m + i] = (Gy e_q)[i] for
 * every repetition q < ey->count (R_q is the vector whose inner product with a
 * response gives v_R = e_q^T (Gy^T Yhat_b), the transposition identity of
 * App. B).  R depends only on the challenges, so a client may compute it
 * before or while the server evaluates; the challenges must stay hidden from
 * the server until the responses are fixed.
 *   ey : ell = ey->count (1 <= ell <= 16) challenges of t_y positions < Ny
 *   R  : device, ell x m field array, written
 * Errors: MVK_EINVAL, MVK_ERANGE (ell > 16), MVK_ENOMEM.
 */
mvk_status mvk_verify_prepare(const mvk_key *key, const mvk_sparse *ey, uint32_t *R, void *stream);

/*
 * mvk_decode_verify with the challenge syndromes R computed beforehand by
 * mvk_verify_prepare for the same key and the same ey (R is read, device,
 * ell x m).  Same outputs, bit for bit.
 * Errors: as mvk_decode_verify.
 */
mvk_status mvk_decode_verify_prepared(const mvk_key *key, const uint32_t *Xhat,
                                      const uint32_t *Yhat, uint32_t B, const mvk_sparse *ex,
                                      const mvk_sparse *ey, const uint32_t *R, uint32_t *Y,
                                      uint32_t *vL, uint32_t *vR, uint32_t *accept, void *stream);

/*
 * Client preparation: every part of Encrypt, Decrypt and Verify that depends
 * on neither the query nor the server's response (Sec. 7 "boost mode": masks
 * generated ahead of time; its standard mode pipelines the same work for the
 * next query while the server evaluates the current one).
 *   ex (may be NULL or count 0): B = ex->count noise vectors e_b of t_x
 *       positions < Nx (the secret state of Encrypt/Decrypt);
 *       Mx : device, B x n, written, input masks   Mx_b = Gx e_b
 *       My : device, B x m, written, output masks  My_b = P e_b = W Mx_b
 *   ey (may be NULL or count 0): ell = ey->count (1..16) challenges e_q of
 *       t_y positions < Ny;
 *       R  : device, ell x m, written, R_q = Gy e_q (as mvk_verify_prepare)
 *       U  : device, ell x n, written, U_q = e_q^T Q
 * The outputs are secret to the client (they determine e); the challenges
 * never leave the client, so they may be drawn before the responses exist.
 * One launch when Nx and Ny are at most 16384 (syndromes and row gathers side
 * by side), else the longer syndromes run first in their own launches.
 * done_flag (device word, may be NULL): set to done_value (!= 0) once every
 *   output is stored and visible device-wide, as mvk_flag_signal would after
 *   the call, but without a launch of its own.
 * Errors: MVK_EINVAL, MVK_ERANGE (ell > 16 or B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_client_prepare(const mvk_key *key, const mvk_sparse *ex, const mvk_sparse *ey,
                              uint32_t *Mx, uint32_t *My, uint32_t *R, uint32_t *U,
                              uint32_t *done_flag, uint32_t done_value, void *stream);

/*
 * mvk_client_prepare for G <= MVK_MAX_GROUP keys that share their input (for
 * example q, k and v): keys of one shape m x n and one privacy code (the same
 * cx arrays), so that the noise vectors ex and the input mask Mx are shared;
 * My[g] = P_g e_b, R[g] = Gy_g e_q and U[g] = e_q^T Q_g for each key with its
 * own challenges ey[g] (the same count and t for every g).  My, R, U, ey: host
 * arrays of G pointers (device buffers as mvk_client_prepare).  One launch
 * when Nx and Ny are at most 16384 (else the longer syndromes first, in their
 * own launches); same outputs, bit for bit, as G calls of mvk_client_prepare.
 * Errors: as mvk_client_prepare, plus MVK_EINVAL (G out of range, keys of
 * different shapes or privacy codes, challenge sets of different sizes).
 */
mvk_status mvk_client_prepare_group(uint32_t G, const mvk_key *const *keys, const mvk_sparse *ex,
                                    const mvk_sparse *const *ey, uint32_t *Mx, uint32_t *const *My,
                                    uint32_t *const *R, uint32_t *const *U, uint32_t *done_flag, uint32_t done_value,
                                    void *stream);

/*
 * Client preparation of several inputs and the keys they feed in one call
 * (for example the four inputs and seven projections of a decoder layer):
 * every syndrome of block length at most 16384 and every row gather of the
 * call run in one launch, instead of one launch per input.
 *   G    : 1..MVK_MAX_PREP keys; keys, ex, ey, Mx, My, R, U: host arrays of G
 *          entries (ex, ey, done_flags may also be NULL as a whole)
 *   ex[g]: noise of key g's input (NULL or count 0: no masks for key g).
 *          Keys whose Mx[g] is the same buffer share that input: their ex[g]
 *          must then describe the same vectors (the same idx and val buffers,
 *          count and t) and their privacy codes must be the same arrays; the
 *          input mask is computed once.
 *   ey[g]: challenges of key g (NULL or count 0: none)
 *   Mx[g], My[g], R[g], U[g]: as mvk_client_prepare for key g
 *   done_flags[g] (device word or NULL): set to done_value once every output
 *          of the call is stored and visible device-wide
 * Same outputs, bit for bit, as G calls of mvk_client_prepare.
 * Errors: as mvk_client_prepare, plus MVK_EINVAL (G out of range, keys that
 * share an input buffer with different noise or privacy codes).
 */
#define MVK_MAX_PREP 8u
mvk_status mvk_client_prepare_multi(uint32_t G, const mvk_key *const *keys, const mvk_sparse *const *ex,
                                    const mvk_sparse *const *ey, uint32_t *const *Mx, uint32_t *const *My,
                                    uint32_t *const *R, uint32_t *const *U, uint32_t *const *done_flags,
                                    uint32_t done_value, void *stream);

/*
 * Encrypt with a prepared input mask: Xhat = X + Mx (B x n, element-wise mod p).
 * Same result as mvk_encode with the noise vectors Mx was prepared from.
 * X, Mx: device, read; Xhat: device, written (may alias X).
 * ready_flag (device word, may be NULL): first wait until
 *   *ready_flag == ready_value, then clear it, as mvk_flag_wait would before
 *   the call (same time-out rules: timeout_us, timed_out), but without a
 *   launch of its own.
 * Errors: MVK_EINVAL (a flag with value 0 or timeout 0).
 */
mvk_status mvk_encode_masked(const mvk_key *key, const uint32_t *X, uint32_t B, const uint32_t *Mx,
                             uint32_t *Xhat, uint32_t *ready_flag, uint32_t ready_value,
                             uint32_t timeout_us, uint32_t *timed_out, void *stream);

/*
 * Decrypt + Verify with prepared masks and challenge vectors (from
 * mvk_client_prepare): Y_b = Yhat_b - My_b, v_L = U_q . Xhat_b,
 * v_R = R_q . Yhat_b, accept[b] = 1 iff v_L == v_R for every q < ell.  Same
 * outputs, bit for bit, as mvk_decode_verify with the same noise and
 * challenges; no gathers (every input is read once, coalesced).
 *   My: B x m;  R: ell x m;  U: ell x n (device, read);  other arguments as
 *   mvk_decode_verify.
 * Errors: MVK_EINVAL, MVK_ERANGE (ell > 16 or B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_decode_verify_masked(const mvk_key *key, const uint32_t *Xhat, const uint32_t *Yhat,
                                    uint32_t B, const uint32_t *My, uint32_t ell, const uint32_t *R,
                                    const uint32_t *U, uint32_t *Y, uint32_t *vL, uint32_t *vR,
                                    uint32_t *accept, void *stream);

/*
 * One client turn between two server calls of independent queries (the
 * standard mode of Sec. 7, where the client's work for the next query runs
 * while the server is busy): mvk_decode_verify_masked of one response and
 * mvk_encode_masked of the next query in one launch when the decode/verify
 * is small (B (m + n) <= 32768, ell <= 4), else as the two calls.
 *   key, Xhat, Yhat, B, My, ell, R, U, Y, vL, vR, accept: as
 *       mvk_decode_verify_masked (the response of the current query)
 *   X_next, B_next, Mx_next, Xhat_next, ready_flag, ready_value, timeout_us,
 *       timed_out: as mvk_encode_masked with the same key (the next query;
 *       B_next may be 0 with no ready_flag: no next query)
 * Same outputs, bit for bit, as the two calls.
 * Errors: as the two calls.
 */
mvk_status mvk_decode_verify_encode_masked(const mvk_key *key, const uint32_t *Xhat, const uint32_t *Yhat,
                                           uint32_t B, const uint32_t *My, uint32_t ell, const uint32_t *R,
                                           const uint32_t *U, uint32_t *Y, uint32_t *vL, uint32_t *vR,
                                           uint32_t *accept, const uint32_t *X_next, uint32_t B_next,
                                           const uint32_t *Mx_next, uint32_t *Xhat_next, uint32_t *ready_flag,
                                           uint32_t ready_value, uint32_t timeout_us, uint32_t *timed_out,
                                           void *stream);

/*
 * mvk_decode_verify_masked for G <= MVK_MAX_GROUP matrices that share the
 * queries Xhat (for example q, k and v, evaluated by
 * mvk_server_eval_packed_group): problem g has its key keys[g] (all keys of
 * one shape m x n), response Yhat[g], prepared vectors My[g], R[g], U[g]
 * (from mvk_client_prepare with keys[g]) and outputs Y[g], vL[g], vR[g],
 * accept[g]; every array is a host array of G device pointers (vL, vR may be
 * NULL, or hold NULL entries).  Same outputs, bit for bit, as G calls of
 * mvk_decode_verify_masked; one launch where the problem is large enough for
 * the element-block kernel (B * (m + n) above 32768 words, ell <= 4), else
 * one per matrix.
 * Errors: MVK_EINVAL (null pointer, G out of range, keys of different
 * shapes), MVK_ERANGE (ell > 16 or B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_decode_verify_masked_group(uint32_t G, const mvk_key *const *keys, const uint32_t *Xhat, uint32_t B,
                                          const uint32_t *const *Yhat, const uint32_t *const *My, uint32_t ell,
                                          const uint32_t *const *R, const uint32_t *const *U, uint32_t *const *Y,
                                          uint32_t *const *vL, uint32_t *const *vR, uint32_t *const *accept,
                                          void *stream);

/*
 * Stream flags: order work on two streams whose launches are captured in two
 * separate HIP graphs (a graph cannot wait for another graph's work).
 * mvk_flag_signal: when the stream reaches it (all earlier work on the stream
 *   complete and visible device-wide), *flag = value (value != 0).
 * mvk_flag_wait: the stream waits until *flag == value, then sets *flag = 0
 *   (one wait consumes one signal), and only then runs later work.  The wait
 *   polls from one thread of one workgroup; after timeout_us microseconds it
 *   gives up, leaves *flag, sets *timed_out (device word, may be NULL) to
 *   nonzero and lets the stream continue: the caller must check *timed_out
 *   before trusting what follows.  flag, timed_out: device words.
 * HIP multiplexes streams onto a few hardware queues, and a waiting kernel
 * holds up everything queued behind it on its queue: submit the signalling
 * stream's work before the waits that depend on it (for two graphs, replay
 * the signalling graph first), so that a shared queue only serialises the
 * two streams instead of running the waits into their time-outs.
 * Errors: MVK_EINVAL (null flag, value 0 or timeout 0).
 */
mvk_status mvk_flag_signal(uint32_t *flag, uint32_t value, void *stream);
mvk_status mvk_flag_wait(uint32_t *flag, uint32_t value, uint32_t timeout_us, uint32_t *timed_out,
                         void *stream);

/*
 * Batch verification (Protocol Batch-vMVMD, Sec. 5.4): B claims
 * M_b x_b = y_b with M_b in F^{m x n}, all keyed with the same verification
 * code G (k = m, N = r*m): Q_b = G^T M_b from each claim's mvk_keygen.  The
 * challenge projections u_b = Q_b^T e are computed by the server and checked
 * with a second RAA code G' (k = B*n, N' = r'*B*n).
 *
 * Preprocess, auxiliary part:
 *   Q     : host array of B device pointers, Q[b] is Q_b (N x n)
 *   c2    : the secondary code, c2->k == B*n
 *   QtT   : device, N x Bn, written: row i = (Q_1[i, :], ..., Q_B[i, :])
 *           (what the server keeps, as the transpose of the stacked Qt)
 *   Qaux  : device, N x N', written: Qaux = QtT G' (the client's state)
 * Uses a workspace of about N*N' words.  Errors: MVK_EINVAL, MVK_ERANGE (also N
 * above 65535 * 64), MVK_ENOMEM.
 */
mvk_status mvk_batch_preprocess(uint32_t B, const uint32_t *const *Q, uint32_t N, uint32_t n,
                                const mvk_code *c2, uint32_t *QtT, uint32_t *Qaux, void *stream);

/*
 * Batch verification, server step: for every primary challenge e_q (shared by
 * all claims), Ut[q] = Qt e_q = sum_{j in supp(e_q)} e_j QtT[j, :]  (B*n),
 * whose entries [b*n, b*n + n) are u_b = Q_b^T e_q.
 *   QtT: device, N x Bn (from mvk_batch_preprocess);  e: ell (1..16)
 *   challenges of t positions < N;  Ut: device, ell x Bn, written.
 * Errors: MVK_EINVAL, MVK_ERANGE (ell > 16).
 */
mvk_status mvk_batch_project(const uint32_t *QtT, uint32_t N, uint32_t n, uint32_t B,
                             const mvk_sparse *e, uint32_t *Ut, void *stream);

/*
 * Batch verification, client checks, with the secondary challenges e2
 * (ell2 = 1..16 challenges of t' positions < N') drawn after Ut is fixed:
 *   original   vL[q][b] = (u_b of Ut[q]) . x_b  ==  vR[q][b] = (G e_q) . y_b
 *   secondary  sL[q][j] = e_q^T Qaux e2_j      ==  sR[q][j] = (G' e2_j) . Ut[q]
 * accept[b] = 1 iff every secondary pair of the batch and every original pair
 * of claim b agree (a failed secondary check rejects the whole batch).
 *   cy: primary code (k = m);  c2: secondary code (k = B*n);  Qaux: N x N';
 *   X: B x n, Y: B x m (device);  vL, vR: ell x B;  sL, sR: ell x ell2
 *   (device, may be NULL);  accept: device, B words.
 * Errors: MVK_EINVAL, MVK_ERANGE (ell or ell2 > 16, B > 65535), MVK_ENOMEM.
 */
mvk_status mvk_batch_verify(const mvk_code *cy, const mvk_code *c2, const uint32_t *Qaux, uint32_t m,
                            uint32_t n, uint32_t B, const uint32_t *X, const uint32_t *Y,
                            const mvk_sparse *e, const uint32_t *Ut, const mvk_sparse *e2, uint32_t *vL,
                            uint32_t *vR, uint32_t *sL, uint32_t *sR, uint32_t *accept, void *stream);

/*
 * RAA encoding w -> G^T w (App. B, "Linear-time encoding") for `count`
 * vectors.  w: device, count x k field array; out: device, count x N.
 * Uses a workspace of about N*count words (plus 2/256 of that).
 * Errors: MVK_EINVAL, MVK_ERANGE (N*count*4 above 2^62 bytes, count above
 * 65535 * 64), MVK_ENOMEM.
 */
mvk_status mvk_raa_encode(const mvk_code *code, const uint32_t *w, uint32_t count, uint32_t *out,
                          void *stream);

/*
 * RAA syndrome v -> G v (App. B, transposition principle) for `count` dense
 * vectors.  v: device, count x N field array; out: device, count x k.
 * Errors: MVK_EINVAL, MVK_ERANGE (count > 65535), MVK_ENOMEM.
 */
mvk_status mvk_raa_syndrome(const mvk_code *code, const uint32_t *v, uint32_t count,
                            uint32_t *out, void *stream);

/*
 * Streaming read of `bytes` bytes at `data` (device, 16-byte aligned, bytes a
 * multiple of 16), nothing computed but a checksum: the HBM read floor for a
 * buffer of that size, which server_eval's stream of W is measured against.
 * sink: device, MVK_STREAM_READ_BLOCKS uint32 words; word w receives the XOR
 * of the 32-bit words read by workgroup w (zero for workgroups the launch
 * does not have), so the XOR of all sink words is the XOR of the whole buffer.
 * Errors: MVK_EINVAL (null or misaligned pointer, bytes not a multiple of 16).
 */
#define MVK_STREAM_READ_BLOCKS 4096u
mvk_status mvk_stream_read(const void *data, size_t bytes, uint32_t *sink, void *stream);

/*
 * Frees the workspace buffers that growths have retired (see the conventions
 * above), after waiting for the device.  Call it only when no HIP graph
 * captured before those growths will be replayed again.
 */
mvk_status mvk_workspace_release(void);

/*
 * A stream of the current device whose kernels run only on the compute units
 * [first_cu, first_cu + count), numbered as the device's compute-unit mask
 * numbers them (a CU mask on the stream's hardware queue; default priority).
 * For schedules with two independent streams, such as the client's
 * preparation beside the online calls of the pipelined mode (Sec. 7): two
 * disjoint ranges keep the streams' workgroups off each other's compute
 * units, so a kernel waiting on a flag never holds units the other stream's
 * producer needs.  Release with mvk_stream_destroy, which waits for the
 * stream, destroys it, and retires the library's workspace of that stream
 * (freed by mvk_workspace_release, like the buffers a workspace growth
 * retires).
 * Errors: MVK_EINVAL (stream NULL, count 0, or a range past the device's
 * compute units), MVK_EHIP.
 */
mvk_status mvk_stream_create_cu_range(uint32_t first_cu, uint32_t count, void **stream);
mvk_status mvk_stream_destroy(void *stream);

/* ---------------------------------------------------------------------------
 * Seeded calls: the library draws the method's randomness.
 *
 * Protocol pvMVMD (Sec. 6.1) samples the two RAA codes in Preprocess (App. B:
 * uniform permutations pi1, pi2 of [0, N) and diagonals v1, v2 with entries
 * uniform in F_p^*), fresh noise e_x <- E_{tx}^{Nx} for every query column in
 * Encrypt, and the challenges e <- E_{ty}^{Ny} in Verify once the responses
 * are fixed (E_t^N: exactly t nonzero entries, Sec. 3; Lemma 5.1 draws the
 * support uniformly and the values uniformly in F_p^*).  The calls below draw
 * them from 64-bit seeds; the same seed reproduces the same draws.  The paper
 * does not fix a generator; the library follows this specification:
 *   - SplitMix64 (Steele, Lea and Flood, 2014): the state advances by
 *     0x9E3779B97F4A7C15 and each output is the state passed through the
 *     finaliser z ^= z>>30; z *= 0xBF58476D1CE4E5B9; z ^= z>>27;
 *     z *= 0x94D049BB133111EB; z ^= z>>31.
 *   - Stream c of (seed, tag) starts from finaliser(seed ^ tag ^ finaliser(c)).
 *   - An integer below b: outputs z >= 2^64 - (2^64 mod b) are rejected, the
 *     value is z mod b (after 64 rejections, the last z mod b).  A value in
 *     F_p^*: the top 31 bits of an output, rejected unless in [1, p-1] (after
 *     64 rejections, 1).
 *   - A code (k, r): stream 0; pi1, then pi2 by Fisher-Yates (from the
 *     identity, for i = N-1 down to 1 swap entries i and below(i+1)), then the
 *     N values of v1, then those of v2.
 *   - Sparse vector c of E_t^N: stream c; positions below(N), repeats skipped,
 *     until t are held, in draw order (after 2^24 draws the smallest free
 *     positions complete it); then its t values in F_p^*.
 * Tags (ASCII, big-endian) separate the purposes of one seed.
 */
#define MVK_TAG_CODE_X 0x6D766B2D636F6478ull    /* "mvk-codx": the privacy code Gx */
#define MVK_TAG_CODE_Y 0x6D766B2D636F6479ull    /* "mvk-cody": the verification code Gy */
#define MVK_TAG_NOISE 0x6D766B2D6E6F6973ull     /* "mvk-nois": e_x of Encrypt */
#define MVK_TAG_CHALLENGE 0x6D766B2D6368616Cull /* "mvk-chal": e of Verify */
/* As a seed: draw the seed itself from the operating system (getrandom). */
#define MVK_SEED_FRESH 0xFFFFFFFFFFFFFFFFull
/* Largest sparsity t the seeded calls accept. */
#define MVK_SEEDED_MAX_T 4096u

/* pp: the public parameters of Preprocess (both codes, P^T and Q), and st:
 * the secret state of Encrypt (the noise vectors).  Both are library-owned,
 * with their device memory; the *_free calls release them. */
typedef struct mvk_pp mvk_pp;
typedef struct mvk_st mvk_st;

/*
 * The sampling specification above on the host, for callers that keep the
 * draws themselves (and for tests).  mvk_sample_code: a code of dimension k
 * and block length N = r*k into pi1, pi2, v1, v2 (host, N words each).
 * mvk_sample_sparse: `count` draws from E_t^N into idx, val (host, count x t
 * words each; t <= N).  The values are in the build's field.
 * Errors: MVK_EINVAL (null pointer, k, r or N zero, t > N), MVK_ERANGE (N above
 * 2^31 - 1).
 */
mvk_status mvk_sample_code(uint32_t k, uint32_t r, uint64_t seed, uint64_t tag, uint32_t *pi1, uint32_t *pi2,
                           uint32_t *v1, uint32_t *v2);
mvk_status mvk_sample_sparse(uint32_t count, uint32_t N, uint32_t t, uint64_t seed, uint64_t tag, uint32_t *idx,
                             uint32_t *val);

/*
 * Preprocess with codes the library draws (Protocol pvMVMD, Preprocess; App. B):
 * Gx (k = n, rate 1/r_x) from (code_seed, MVK_TAG_CODE_X), Gy (k = m, rate
 * 1/r_y) from (code_seed, MVK_TAG_CODE_Y), then P^T = (W Gx)^T and Q = Gy^T W
 * as mvk_keygen.  W: device, m x n int8.  *out receives a new pp holding one
 * device allocation (the code arrays, P^T and Q); mvk_pp_key gives the
 * mvk_key view every other call takes.  Waits for `stream` (the code arrays
 * are copied from the host), so it cannot be captured in a graph.
 * Errors: MVK_EINVAL, MVK_ERANGE (n > MVK_MAX_N, a block length above
 * 2^31 - 1, a buffer above 2^62 bytes), MVK_ENOMEM, MVK_ERANDOM, MVK_EHIP.
 */
mvk_status mvk_keygen_seeded(uint32_t m, uint32_t n, uint32_t r_x, uint32_t r_y, uint64_t code_seed,
                             const int8_t *W, void *stream, mvk_pp **out);
/* The key of pp (valid until mvk_pp_free); NULL for a NULL pp. */
const mvk_key *mvk_pp_key(const mvk_pp *pp);
/* Frees pp and its device memory (hipFree; work that reads the key must be
 * complete).  NULL is ignored. */
void mvk_pp_free(mvk_pp *pp);

/*
 * Encrypt with noise the library draws (Protocol pvMVMD, Encrypt): column b
 * gets e_b = sparse vector b of E_{t_x}^{Nx} from (noise_seed, MVK_TAG_NOISE),
 * drawn on the device, and Xhat_b = X_b + Gx e_b (as mvk_encode).  Every call
 * must use a new seed (Sec. 4.2: reusing the noise of a column leaks the
 * difference of the two queries); MVK_SEED_FRESH takes one from the
 * operating system.  *st receives a new state holding the noise (device
 * memory), the secret st of Encrypt that decode needs; mvk_st_noise exposes it.
 *   X: device, B x n (plaintext);  Xhat: device, B x n, written.
 * Stream-ordered like mvk_encode (the draws are a kernel on `stream`).
 * Errors: MVK_EINVAL (t_x > Nx, null pointer), MVK_ERANGE (B > 65535,
 * t_x > MVK_SEEDED_MAX_T), MVK_ENOMEM, MVK_ERANDOM, MVK_EHIP.
 */
mvk_status mvk_encode_seeded(const mvk_key *key, const uint32_t *X, uint32_t B, uint32_t t_x, uint64_t noise_seed,
                             uint32_t *Xhat, mvk_st **st, void *stream);
/* The noise of st (B sparse vectors of t_x positions; device arrays). */
const mvk_sparse *mvk_st_noise(const mvk_st *st);
/* Frees st and its device memory (work that reads it must be complete). */
void mvk_st_free(mvk_st *st);

/*
 * Verify + Decrypt with challenges the library draws (Protocol pvMVMD, Verify
 * and Decrypt): ell challenges, challenge q = sparse vector q of E_{t_y}^{Ny}
 * from (chal_seed, MVK_TAG_CHALLENGE), drawn on the device when the call
 * runs, after the responses Yhat it is given; then everything as
 * mvk_decode_verify with the noise of st (B = the column count of st).
 * Outputs as mvk_decode_verify.  Errors: as mvk_decode_verify, plus
 * MVK_EINVAL (null st, t_y > Ny), MVK_ERANGE (t_y > MVK_SEEDED_MAX_T),
 * MVK_ERANDOM.
 */
mvk_status mvk_decode_verify_seeded(const mvk_key *key, const mvk_st *st, const uint32_t *Xhat,
                                    const uint32_t *Yhat, uint32_t t_y, uint32_t ell, uint64_t chal_seed,
                                    uint32_t *Y, uint32_t *vL, uint32_t *vR, uint32_t *accept, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MVK_H_ */
