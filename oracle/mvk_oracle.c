/*
 * CPU oracle for the pvMVMD hot path (Maverick, arxiv 2609.10264).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library.  The product (the HIP library under
 * paper_2609_10264_amd/) shares no code with it and never calls it.
 *
 * Plain, slow, obviously-correct C.  Every field operation is done with the
 * '%' operator on 64-bit unsigned integers; nothing is blocked, fused or
 * reordered beyond what the paper's definitions state.  Indices are 0-based.
 *
 * Field: F_p, p fixed when the file is compiled: 2^31 - 1 by default, or the
 * BabyBear prime 15 * 2^27 + 1 (the field of the paper's Sec. 7.1) with
 * -DORC_P=2013265921.  Any prime below 2^31 works: every product of two
 * field elements and every sum of two fits in 64 bits before its '%'.
 * Field arrays are uint32 in [0, p).
 * Signed int8 weights are embedded as w mod p (Sec. 7.2, "Model quantization":
 * signed integers are embedded into the field).
 *
 * RAA code (App. B): G = R * Pi1 * V1 * A * Pi2 * V2 * A, G in F^{k x N},
 * N = r*k, with
 *   R_{i,j}  = 1 iff position j lies in the i-th block of r positions,
 *   Pi_{i,j} = 1 iff pi(j) = i,
 *   V        = diag(v),
 *   A_{i,j}  = 1 iff i <= j (upper triangular).
 * Hence (0-based):  R^T w  : out[j] = w[j / r]           (repeat)
 *                   Pi^T w : out[j] = w[pi[j]]           (gather)
 *                   Pi v   : out[pi[j]] = v[j]           (scatter)
 *                   A^T w  : out[j] = sum_{i<=j} w[i]    (prefix sum)
 *                   A v    : out[i] = sum_{j>=i} v[j]    (suffix sum)
 *                   R v    : out[i] = sum_{q<r} v[i*r+q] (fold)
 *
 * Functions:
 *   orc_encT        G^T w  (App. B, "Linear-time encoding")
 *   orc_syn         G v    (App. B, transposition principle)
 *   orc_server_eval Y^ = W X^ mod p                (Protocol pvMVMD, server step)
 *   orc_keygen      P^T = (W Gx)^T, Q = Gy^T W     (Protocol pvMVMD, Preprocess)
 *   orc_encode      X^ = X + Gx e_x                (Protocol pvMVMD, Encrypt)
 *   orc_decode      Y = Y^ - P e_x                 (Protocol pvMVMD, Decrypt)
 *   orc_verify      sparse coded Freivalds check   (Protocol pvMVMD, Verify;
 *                                                   Protocol vMVMD, Verify)
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef ORC_P
#define ORC_P 2147483647ULL
#endif

/* Count of field operations (additions, subtractions, multiplications) since
 * the last orc_ops_reset: lets a test compare the RAA maps' cost with the
 * bounds App. B states (at most 4N for an encoding, 5N for a syndrome).
 * Only the counting build (-DORC_COUNT_OPS, single-threaded use) counts; in
 * the other builds the functions below are re-entrant and the library may be
 * called from several threads at once (each call on its own outputs). */
#ifdef ORC_COUNT_OPS
static uint64_t g_ops;
#define ORC_COUNT() (++g_ops)
#else
#define ORC_COUNT() ((void)0)
#endif
void orc_ops_reset(void) {
#ifdef ORC_COUNT_OPS
    g_ops = 0;
#endif
}
uint64_t orc_ops_count(void) {
#ifdef ORC_COUNT_OPS
    return g_ops;
#else
    return 0;
#endif
}
int orc_counts_ops(void) {
#ifdef ORC_COUNT_OPS
    return 1;
#else
    return 0;
#endif
}

static uint64_t fadd(uint64_t a, uint64_t b) { ORC_COUNT(); return (a + b) % ORC_P; }
static uint64_t fsub(uint64_t a, uint64_t b) { ORC_COUNT(); return (a + ORC_P - b) % ORC_P; }
static uint64_t fmul(uint64_t a, uint64_t b) { ORC_COUNT(); return (a * b) % ORC_P; }

/* Embedding of a signed integer into F_p. */
static uint64_t emb(int64_t w) {
    int64_t r = w % (int64_t)ORC_P;
    if (r < 0) r += (int64_t)ORC_P;
    return (uint64_t)r;
}

uint32_t orc_prime(void) { return (uint32_t)ORC_P; }

/*
 * Encoding w -> G^T w, F^k -> F^N (App. B).  G^T = A^T V2 Pi2^T A^T V1 Pi1^T R^T,
 * applied right to left: repeat, gather by pi1, scale by v1, prefix sum,
 * gather by pi2, scale by v2, prefix sum.
 */
void orc_encT(uint32_t k, uint32_t r, const uint32_t *pi1, const uint32_t *pi2,
              const uint32_t *v1, const uint32_t *v2, const uint32_t *w, uint32_t *out) {
    uint64_t N = (uint64_t)k * r;
    uint64_t *t0 = (uint64_t *)malloc(N * sizeof(uint64_t));
    uint64_t *t1 = (uint64_t *)malloc(N * sizeof(uint64_t));
    /* R^T: repeat */
    for (uint64_t j = 0; j < N; j++) t0[j] = w[j / r];
    /* Pi1^T: gather */
    for (uint64_t j = 0; j < N; j++) t1[j] = t0[pi1[j]];
    /* V1 */
    for (uint64_t j = 0; j < N; j++) t1[j] = fmul(v1[j], t1[j]);
    /* A^T: prefix sum */
    for (uint64_t j = 1; j < N; j++) t1[j] = fadd(t1[j - 1], t1[j]);
    /* Pi2^T: gather */
    for (uint64_t j = 0; j < N; j++) t0[j] = t1[pi2[j]];
    /* V2 */
    for (uint64_t j = 0; j < N; j++) t0[j] = fmul(v2[j], t0[j]);
    /* A^T: prefix sum */
    for (uint64_t j = 1; j < N; j++) t0[j] = fadd(t0[j - 1], t0[j]);
    for (uint64_t j = 0; j < N; j++) out[j] = (uint32_t)t0[j];
    free(t0);
    free(t1);
}

/*
 * Syndrome v -> G v, F^N -> F^k (App. B).  G = R Pi1 V1 A Pi2 V2 A, applied
 * right to left: suffix sum, scale by v2, scatter by pi2, suffix sum, scale
 * by v1, scatter by pi1, fold blocks of r.
 */
void orc_syn(uint32_t k, uint32_t r, const uint32_t *pi1, const uint32_t *pi2,
             const uint32_t *v1, const uint32_t *v2, const uint32_t *v, uint32_t *out) {
    uint64_t N = (uint64_t)k * r;
    uint64_t *s0 = (uint64_t *)malloc(N * sizeof(uint64_t));
    uint64_t *s1 = (uint64_t *)malloc(N * sizeof(uint64_t));
    for (uint64_t j = 0; j < N; j++) s0[j] = v[j] % ORC_P;
    /* A: suffix sum */
    for (uint64_t j = N - 1; j-- > 0;) s0[j] = fadd(s0[j], s0[j + 1]);
    /* V2 */
    for (uint64_t j = 0; j < N; j++) s0[j] = fmul(v2[j], s0[j]);
    /* Pi2: scatter */
    for (uint64_t j = 0; j < N; j++) s1[pi2[j]] = s0[j];
    /* A: suffix sum */
    for (uint64_t j = N - 1; j-- > 0;) s1[j] = fadd(s1[j], s1[j + 1]);
    /* V1 */
    for (uint64_t j = 0; j < N; j++) s1[j] = fmul(v1[j], s1[j]);
    /* Pi1: scatter */
    for (uint64_t j = 0; j < N; j++) s0[pi1[j]] = s1[j];
    /* R: fold */
    for (uint64_t i = 0; i < k; i++) {
        uint64_t acc = 0;
        for (uint64_t q = 0; q < r; q++) acc = fadd(acc, s0[i * r + q]);
        out[i] = (uint32_t)acc;
    }
    free(s0);
    free(s1);
}

/*
 * Server evaluation: Yhat[b][i] = sum_k emb(W[i][k]) * Xhat[b][k] mod p,
 * for rows i in [row0, row1).  W is m x n row-major int8; Xhat is B x n
 * (query b at Xhat + b*n); Yhat is B x m.  Protocol pvMVMD: the server
 * returns y^ = M x^ (one field matrix-vector product per query).
 */
void orc_server_eval_rows(const int8_t *W, uint32_t m, uint32_t n, const uint32_t *Xhat,
                          uint32_t B, uint32_t *Yhat, uint32_t row0, uint32_t row1) {
    for (uint32_t b = 0; b < B; b++) {
        const uint32_t *x = Xhat + (uint64_t)b * n;
        for (uint32_t i = row0; i < row1 && i < m; i++) {
            const int8_t *w = W + (uint64_t)i * n;
            uint64_t acc = 0;
            for (uint32_t k = 0; k < n; k++) acc = fadd(acc, fmul(emb(w[k]), x[k]));
            Yhat[(uint64_t)b * m + i] = (uint32_t)acc;
        }
    }
}

void orc_server_eval(const int8_t *W, uint32_t m, uint32_t n, const uint32_t *Xhat,
                     uint32_t B, uint32_t *Yhat) {
    orc_server_eval_rows(W, m, n, Xhat, B, Yhat, 0, m);
}

/*
 * Preprocess (Protocol pvMVMD): P = W Gx in F^{m x Nx}, Q = Gy^T W in F^{Ny x n}.
 * P^T = Gx^T W^T is m encodings of the rows of W; Q is n encodings of the
 * columns of W (Sec. 6.3, "Preprocessing time").
 * PT is stored Nx x m row-major (PT[j*m + i] = P[i][j]); Q is Ny x n row-major.
 *
 * orc_keygen_PT_rows: the columns i in [i0, i1) of PT (encodings of rows i of W).
 * orc_keygen_Q_cols:  the columns k in [k0, k1) of Q (encodings of columns k of W).
 * Ranges that do not overlap write disjoint entries, so they may run at once.
 */
void orc_keygen_PT_rows(const int8_t *W, uint32_t m, uint32_t n, uint32_t rx, const uint32_t *xpi1,
                        const uint32_t *xpi2, const uint32_t *xv1, const uint32_t *xv2, uint32_t *PT,
                        uint32_t i0, uint32_t i1) {
    uint64_t Nx = (uint64_t)rx * n;
    uint32_t *row = (uint32_t *)malloc((uint64_t)n * sizeof(uint32_t));
    uint32_t *enc = (uint32_t *)malloc(Nx * sizeof(uint32_t));
    for (uint32_t i = i0; i < i1 && i < m; i++) {
        for (uint32_t k = 0; k < n; k++) row[k] = (uint32_t)emb(W[(uint64_t)i * n + k]);
        orc_encT(n, rx, xpi1, xpi2, xv1, xv2, row, enc);
        for (uint64_t j = 0; j < Nx; j++) PT[j * m + i] = enc[j];
    }
    free(row);
    free(enc);
}

void orc_keygen_Q_cols(const int8_t *W, uint32_t m, uint32_t n, uint32_t ry, const uint32_t *ypi1,
                       const uint32_t *ypi2, const uint32_t *yv1, const uint32_t *yv2, uint32_t *Q,
                       uint32_t k0, uint32_t k1) {
    uint64_t Ny = (uint64_t)ry * m;
    uint32_t *col = (uint32_t *)malloc((uint64_t)m * sizeof(uint32_t));
    uint32_t *enc = (uint32_t *)malloc(Ny * sizeof(uint32_t));
    for (uint32_t k = k0; k < k1 && k < n; k++) {
        for (uint32_t i = 0; i < m; i++) col[i] = (uint32_t)emb(W[(uint64_t)i * n + k]);
        orc_encT(m, ry, ypi1, ypi2, yv1, yv2, col, enc);
        for (uint64_t j = 0; j < Ny; j++) Q[j * n + k] = enc[j];
    }
    free(col);
    free(enc);
}

/* Both outputs at once; either pointer may be NULL to skip it. */
void orc_keygen(const int8_t *W, uint32_t m, uint32_t n,
                uint32_t rx, const uint32_t *xpi1, const uint32_t *xpi2, const uint32_t *xv1, const uint32_t *xv2,
                uint32_t ry, const uint32_t *ypi1, const uint32_t *ypi2, const uint32_t *yv1, const uint32_t *yv2,
                uint32_t *PT, uint32_t *Q) {
    if (PT) orc_keygen_PT_rows(W, m, n, rx, xpi1, xpi2, xv1, xv2, PT, 0, m);
    if (Q) orc_keygen_Q_cols(W, m, n, ry, ypi1, ypi2, yv1, yv2, Q, 0, n);
}

/*
 * Encrypt (Protocol pvMVMD): e_x <- E_{tx}^{Nx} (given as tx (index, value)
 * pairs per column), x' = Gx e_x, x^ = x + x'.  X, Xhat are B x n.
 */
void orc_encode(uint32_t n, uint32_t rx, const uint32_t *pi1, const uint32_t *pi2,
                const uint32_t *v1, const uint32_t *v2, const uint32_t *X, uint32_t B,
                const uint32_t *ex_idx, const uint32_t *ex_val, uint32_t tx, uint32_t *Xhat) {
    uint64_t Nx = (uint64_t)rx * n;
    uint32_t *e = (uint32_t *)malloc(Nx * sizeof(uint32_t));
    uint32_t *xp = (uint32_t *)malloc((uint64_t)n * sizeof(uint32_t));
    for (uint32_t b = 0; b < B; b++) {
        memset(e, 0, Nx * sizeof(uint32_t));
        for (uint32_t s = 0; s < tx; s++) {
            uint64_t j = ex_idx[(uint64_t)b * tx + s];
            e[j] = (uint32_t)fadd(e[j], ex_val[(uint64_t)b * tx + s]);
        }
        orc_syn(n, rx, pi1, pi2, v1, v2, e, xp);
        for (uint32_t k = 0; k < n; k++)
            Xhat[(uint64_t)b * n + k] = (uint32_t)fadd(X[(uint64_t)b * n + k], xp[k]);
    }
    free(e);
    free(xp);
}

/*
 * Decrypt (Protocol pvMVMD): y = y^ - P e_x = y^ - sum_{j in supp(e_x)} e_j P[:, j]
 * (Table "Cost tally for the client online phase of pvMVMD").
 * PT is Nx x m (row j is column j of P).  Yhat, Y are B x m.
 */
void orc_decode(const uint32_t *PT, uint32_t m, const uint32_t *Yhat, uint32_t B,
                const uint32_t *ex_idx, const uint32_t *ex_val, uint32_t tx, uint32_t *Y) {
    for (uint32_t b = 0; b < B; b++) {
        for (uint32_t i = 0; i < m; i++) {
            uint64_t mask = 0;
            for (uint32_t s = 0; s < tx; s++) {
                uint64_t j = ex_idx[(uint64_t)b * tx + s];
                mask = fadd(mask, fmul(ex_val[(uint64_t)b * tx + s], PT[j * m + i]));
            }
            Y[(uint64_t)b * m + i] = (uint32_t)fsub(Yhat[(uint64_t)b * m + i], mask);
        }
    }
}

/*
 * Verify (Protocol pvMVMD, which runs the Verify of Protocol vMVMD on the
 * ciphertexts):
 *   z_b = Gy^T y^_b;  for each repetition q: e <- E_{ty}^{Ny};
 *   v_L = (e^T Q) x^_b,  v_R = e^T z_b;  reject iff v_L != v_R.
 * One challenge per repetition is shared by all B columns (Sec. 5.4: the same
 * sparse challenge may be shared across claims).  ey_idx/ey_val are ell x ty.
 * Outputs: vL, vR (ell x B, may be NULL), accept (B): 1 iff every repetition
 * matched for that column.
 */
void orc_verify(uint32_t m, uint32_t n, uint32_t ry, const uint32_t *pi1, const uint32_t *pi2,
                const uint32_t *v1, const uint32_t *v2, const uint32_t *Q,
                const uint32_t *Xhat, const uint32_t *Yhat, uint32_t B,
                const uint32_t *ey_idx, const uint32_t *ey_val, uint32_t ty, uint32_t ell,
                uint32_t *vL, uint32_t *vR, uint8_t *accept) {
    uint64_t Ny = (uint64_t)ry * m;
    uint32_t *z = (uint32_t *)malloc(Ny * (uint64_t)B * sizeof(uint32_t));
    uint64_t *u = (uint64_t *)malloc((uint64_t)n * sizeof(uint64_t));
    for (uint32_t b = 0; b < B; b++) {
        orc_encT(m, ry, pi1, pi2, v1, v2, Yhat + (uint64_t)b * m, z + (uint64_t)b * Ny);
        accept[b] = 1;
    }
    for (uint32_t q = 0; q < ell; q++) {
        const uint32_t *ei = ey_idx + (uint64_t)q * ty;
        const uint32_t *ev = ey_val + (uint64_t)q * ty;
        /* u = e^T Q = sum_{j in supp(e)} e_j Q[j, :] */
        for (uint32_t k = 0; k < n; k++) u[k] = 0;
        for (uint32_t s = 0; s < ty; s++)
            for (uint32_t k = 0; k < n; k++) u[k] = fadd(u[k], fmul(ev[s], Q[(uint64_t)ei[s] * n + k]));
        for (uint32_t b = 0; b < B; b++) {
            const uint32_t *x = Xhat + (uint64_t)b * n;
            uint64_t l = 0, rr = 0;
            for (uint32_t k = 0; k < n; k++) l = fadd(l, fmul(u[k], x[k]));
            for (uint32_t s = 0; s < ty; s++) rr = fadd(rr, fmul(ev[s], z[(uint64_t)b * Ny + ei[s]]));
            if (vL) vL[(uint64_t)q * B + b] = (uint32_t)l;
            if (vR) vR[(uint64_t)q * B + b] = (uint32_t)rr;
            if (l != rr) accept[b] = 0;
        }
    }
    free(z);
    free(u);
}

/*
 * Protocol Batch-vMVMD (Sec. 5.4), Preprocess, auxiliary matrix:
 *   Qt = [Q_1 | ... | Q_B]^T in F^{Bn x N},  Qaux = Qt^T G' in F^{N x N'}.
 * Row i of Qt^T is (Q_1[i, :], ..., Q_B[i, :]) (length Bn), so row i of Qaux
 * is that row times G', i.e. the encoding G'^T of it (App. B).
 * Qs: B x N x n (Q_b at Qs + b*N*n); the secondary code has k = B*n, block
 * length N' = r2*B*n.  Qaux: N x N'.
 */
void orc_batch_aux(uint32_t B, uint32_t N, uint32_t n, const uint32_t *Qs, uint32_t r2,
                   const uint32_t *pi1, const uint32_t *pi2, const uint32_t *v1, const uint32_t *v2,
                   uint32_t *Qaux) {
    uint64_t k2 = (uint64_t)B * n, N2 = k2 * r2;
    uint32_t *row = (uint32_t *)malloc(k2 * sizeof(uint32_t));
    for (uint64_t i = 0; i < N; i++) {
        for (uint64_t b = 0; b < B; b++)
            for (uint64_t c = 0; c < n; c++) row[b * n + c] = Qs[(b * N + i) * n + c];
        orc_encT((uint32_t)k2, r2, pi1, pi2, v1, v2, row, Qaux + i * N2);
    }
    free(row);
}

/*
 * Batch-vMVMD, Verify, server step: for every primary challenge e(q),
 * u~(q) = Qt e(q) in F^{Bn}; entry b*n + c is sum_{j in supp(e)} e_j Q_b[j, c].
 * e_idx, e_val: ell x t; out: ell x Bn.
 */
void orc_batch_project(uint32_t B, uint32_t N, uint32_t n, const uint32_t *Qs, const uint32_t *e_idx,
                       const uint32_t *e_val, uint32_t t, uint32_t ell, uint32_t *out) {
    (void)N;
    uint64_t Bn = (uint64_t)B * n;
    for (uint64_t q = 0; q < ell; q++) {
        for (uint64_t b = 0; b < B; b++) {
            for (uint64_t c = 0; c < n; c++) {
                uint64_t acc = 0;
                for (uint64_t s = 0; s < t; s++) {
                    uint64_t j = e_idx[q * t + s];
                    acc = fadd(acc, fmul(e_val[q * t + s], Qs[(b * N + j) * n + c]));
                }
                out[q * Bn + b * n + c] = (uint32_t)acc;
            }
        }
    }
}

/*
 * Batch-vMVMD, Verify, client checks:
 *   z_b = G^T y_b;  r(j) = G' e'(j);
 *   secondary, every (q, j):  sL = (e(q))^T Qaux e'(j),  sR = (r(j))^T u~(q);
 *   original, every (q, b):   vL = (u_b(q))^T x_b,       vR = (e(q))^T z_b,
 * where u_b(q) is entries [b*n, b*n + n) of u~(q).  The batch is accepted iff
 * every secondary pair agrees; claim b iff, in addition, every original pair
 * of b agrees (the caller combines them).
 * Primary code G: k = m, rate r (pi1, pi2, v1, v2); secondary code G': k = B*n,
 * rate r2 (qi1, qi2, w1, w2).  X: B x n, Y: B x m, Qaux: N x N' (N = r*m,
 * N' = r2*B*n), e: ell x t, ut: ell x Bn, e2: ell2 x t2.
 * Outputs vL, vR: ell x B; sL, sR: ell x ell2.
 */
void orc_batch_verify(uint32_t m, uint32_t n, uint32_t B, uint32_t r, const uint32_t *pi1, const uint32_t *pi2,
                      const uint32_t *v1, const uint32_t *v2, uint32_t r2, const uint32_t *qi1, const uint32_t *qi2,
                      const uint32_t *w1, const uint32_t *w2, const uint32_t *Qaux, const uint32_t *X,
                      const uint32_t *Y, const uint32_t *e_idx, const uint32_t *e_val, uint32_t t, uint32_t ell,
                      const uint32_t *ut, const uint32_t *e2_idx, const uint32_t *e2_val, uint32_t t2,
                      uint32_t ell2, uint32_t *vL, uint32_t *vR, uint32_t *sL, uint32_t *sR) {
    uint64_t N = (uint64_t)r * m, Bn = (uint64_t)B * n, N2 = Bn * r2;
    uint32_t *z = (uint32_t *)malloc(N * sizeof(uint32_t));
    uint32_t *e2 = (uint32_t *)malloc(N2 * sizeof(uint32_t));
    uint32_t *rj = (uint32_t *)malloc(Bn * sizeof(uint32_t));
    /* original checks */
    for (uint64_t b = 0; b < B; b++) {
        orc_encT(m, r, pi1, pi2, v1, v2, Y + b * m, z);
        for (uint64_t q = 0; q < ell; q++) {
            uint64_t l = 0, rr = 0;
            for (uint64_t c = 0; c < n; c++) l = fadd(l, fmul(ut[q * Bn + b * n + c], X[b * n + c]));
            for (uint64_t s = 0; s < t; s++) rr = fadd(rr, fmul(e_val[q * t + s], z[e_idx[q * t + s]]));
            vL[q * B + b] = (uint32_t)l;
            vR[q * B + b] = (uint32_t)rr;
        }
    }
    /* secondary checks */
    for (uint64_t j = 0; j < ell2; j++) {
        for (uint64_t c = 0; c < N2; c++) e2[c] = 0;
        for (uint64_t s = 0; s < t2; s++) e2[e2_idx[j * t2 + s]] = e2_val[j * t2 + s];
        orc_syn((uint32_t)Bn, r2, qi1, qi2, w1, w2, e2, rj);
        for (uint64_t q = 0; q < ell; q++) {
            uint64_t lhs = 0, rhs = 0;
            for (uint64_t a = 0; a < t; a++)
                for (uint64_t s = 0; s < t2; s++) {
                    uint64_t ent = Qaux[(uint64_t)e_idx[q * t + a] * N2 + e2_idx[j * t2 + s]];
                    lhs = fadd(lhs, fmul(fmul(e_val[q * t + a], ent), e2_val[j * t2 + s]));
                }
            for (uint64_t c = 0; c < Bn; c++) rhs = fadd(rhs, fmul(rj[c], ut[q * Bn + c]));
            sL[q * ell2 + j] = (uint32_t)lhs;
            sR[q * ell2 + j] = (uint32_t)rhs;
        }
    }
    free(z);
    free(e2);
    free(rj);
}

/*
 * Seeded sampling of the method's random draws: the codes of Preprocess
 * (App. B: two uniform permutations and two diagonals over F_p^*), the noise
 * e_x <- E_{tx}^{Nx} of Encrypt and the challenges e <- E_{ty}^{Ny} of Verify
 * (Sec. 3: exactly t nonzero entries; Lemma 5.1 draws the support uniformly
 * and the values uniformly in F_p^*).  The paper does not fix a generator;
 * this is a written specification, followed independently by the library:
 *
 *   mix(z)    = SplitMix64's output function (Steele, Lea and Flood, 2014):
 *               z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
 *               z *= 0x94D049BB133111EB; z ^= z >> 31
 *   stream    : a 64-bit state s; each draw is s += 0x9E3779B97F4A7C15, then mix(s)
 *   stream (seed, tag, c) starts at s = mix(seed ^ tag ^ mix(c))
 *   below(b)  : draw z until z < 2^64 - (2^64 mod b) (no rejection when
 *               2^64 mod b = 0); return z mod b.  At most 64 draws: if all
 *               are rejected, the last one's z mod b
 *   nonzero   : draw z until 1 <= (z >> 33) <= p - 1; return z >> 33.  At
 *               most 64 draws: if none is accepted, the value 1
 *   permutation of [0, N): the identity, then for i = N-1 down to 1:
 *               j = below(i + 1), swap entries i and j (Fisher-Yates)
 *   code (k, r) from (seed, tag): stream c = 0; pi1 = permutation, then
 *               pi2 = permutation, then N nonzero values v1, then N values v2
 *   sparse vector c of E_t^N from (seed, tag): stream c; positions
 *               j = below(N), skipping a j already taken, until t are taken
 *               (kept in draw order), at most 2^24 of them per vector (then
 *               the smallest positions not taken, in increasing order, fill
 *               the rest); then t nonzero values
 * The caps only make every loop finite: with t <= N the chance of reaching
 * any of them is below 2^-100 for every size this library accepts.
 */
static uint64_t sm_mix(uint64_t z) {
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ULL;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBULL;
    z ^= z >> 31;
    return z;
}

static uint64_t sm_draw(uint64_t *s) {
    *s += 0x9E3779B97F4A7C15ULL;
    return sm_mix(*s);
}

static uint64_t sm_start(uint64_t seed, uint64_t tag, uint64_t c) { return sm_mix(seed ^ tag ^ sm_mix(c)); }

static uint64_t sm_below(uint64_t *s, uint64_t b) {
    uint64_t rem = (0 - b) % b; /* 2^64 mod b */
    uint64_t z = 0;
    for (int d = 0; d < 64; d++) {
        z = sm_draw(s);
        if (rem == 0 || z < 0 - rem) return z % b;
    }
    return z % b;
}

static uint32_t sm_nonzero(uint64_t *s) {
    for (int d = 0; d < 64; d++) {
        uint64_t v = sm_draw(s) >> 33;
        if (v >= 1 && v <= ORC_P - 1) return (uint32_t)v;
    }
    return 1;
}

/* The raw stream from a given state (for the generator's published test values). */
void orc_sm64_draws(uint64_t state, uint32_t count, uint64_t *out) {
    for (uint32_t i = 0; i < count; i++) out[i] = sm_draw(&state);
}

static void sm_permutation(uint64_t *s, uint64_t N, uint32_t *a) {
    for (uint64_t j = 0; j < N; j++) a[j] = (uint32_t)j;
    for (uint64_t i = N - 1; i >= 1 && i < N; i--) {
        uint64_t j = sm_below(s, i + 1);
        uint32_t t = a[i];
        a[i] = a[j];
        a[j] = t;
    }
}

/* A random RAA code of dimension k and rate 1/r: arrays of N = k*r words. */
void orc_sample_code(uint32_t k, uint32_t r, uint64_t seed, uint64_t tag, uint32_t *pi1, uint32_t *pi2,
                     uint32_t *v1, uint32_t *v2) {
    uint64_t N = (uint64_t)k * r;
    uint64_t s = sm_start(seed, tag, 0);
    sm_permutation(&s, N, pi1);
    sm_permutation(&s, N, pi2);
    for (uint64_t j = 0; j < N; j++) v1[j] = sm_nonzero(&s);
    for (uint64_t j = 0; j < N; j++) v2[j] = sm_nonzero(&s);
}

/* `count` draws from E_t^N (t <= N): idx, val are count x t. */
void orc_sample_sparse(uint32_t count, uint32_t N, uint32_t t, uint64_t seed, uint64_t tag, uint32_t *idx,
                       uint32_t *val) {
    for (uint32_t c = 0; c < count; c++) {
        uint64_t s = sm_start(seed, tag, c);
        uint32_t *ic = idx + (uint64_t)c * t;
        uint32_t got = 0;
        for (uint64_t d = 0; got < t && d < (1ULL << 24); d++) {
            uint32_t j = (uint32_t)sm_below(&s, N);
            int taken = 0;
            for (uint32_t q = 0; q < got; q++)
                if (ic[q] == j) taken = 1;
            if (!taken) ic[got++] = j;
        }
        for (uint32_t j = 0; got < t && j < N; j++) {
            int taken = 0;
            for (uint32_t q = 0; q < got; q++)
                if (ic[q] == j) taken = 1;
            if (!taken) ic[got++] = j;
        }
        for (uint32_t q = 0; q < t; q++) val[(uint64_t)c * t + q] = sm_nonzero(&s);
    }
}
