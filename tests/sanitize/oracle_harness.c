/* Drives every oracle function on small and edge-case inputs so that a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer sees every
 * loop bound, index and arithmetic step (CPU only; the test that builds and
 * runs it is tests/test_sanitizers.py).  Exit status 0 and no sanitizer
 * report means no out-of-bounds access, overflow of signed arithmetic or
 * other undefined behaviour was met. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/mvk_oracle.c"

static uint32_t *arr(size_t n) { return (uint32_t *)calloc(n ? n : 1, sizeof(uint32_t)); }

static void run(uint32_t m, uint32_t n, uint32_t B, uint32_t r, uint32_t tx, uint32_t ty, uint32_t ell,
                uint64_t seed) {
    uint64_t Nx = (uint64_t)r * n, Ny = (uint64_t)r * m;
    int8_t *W = (int8_t *)malloc((size_t)m * n);
    for (uint64_t i = 0; i < (uint64_t)m * n; i++) W[i] = (int8_t)((i * 37 + seed) % 256 - 128);
    uint32_t *xp1 = arr(Nx), *xp2 = arr(Nx), *xv1 = arr(Nx), *xv2 = arr(Nx);
    uint32_t *yp1 = arr(Ny), *yp2 = arr(Ny), *yv1 = arr(Ny), *yv2 = arr(Ny);
    orc_sample_code(n, r, seed, 1, xp1, xp2, xv1, xv2);
    orc_sample_code(m, r, seed, 2, yp1, yp2, yv1, yv2);
    uint32_t *X = arr((size_t)B * n), *Xh = arr((size_t)B * n), *Yh = arr((size_t)B * m), *Y = arr((size_t)B * m);
    for (uint64_t i = 0; i < (uint64_t)B * n; i++) X[i] = (uint32_t)((i * 2654435761u + seed) % ORC_P);
    uint32_t *exi = arr((size_t)B * tx), *exv = arr((size_t)B * tx), *eyi = arr((size_t)ell * ty),
             *eyv = arr((size_t)ell * ty);
    orc_sample_sparse(B, (uint32_t)Nx, tx, seed, 3, exi, exv);
    orc_sample_sparse(ell, (uint32_t)Ny, ty, seed, 4, eyi, eyv);
    uint32_t *PT = arr(Nx * m), *Q = arr(Ny * n);
    orc_keygen(W, m, n, r, xp1, xp2, xv1, xv2, r, yp1, yp2, yv1, yv2, PT, Q);
    orc_keygen_PT_rows(W, m, n, r, xp1, xp2, xv1, xv2, PT, m / 2, m + 3);
    orc_keygen_Q_cols(W, m, n, r, yp1, yp2, yv1, yv2, Q, 0, n);
    orc_encode(n, r, xp1, xp2, xv1, xv2, X, B, exi, exv, tx, Xh);
    orc_server_eval(W, m, n, Xh, B, Yh);
    orc_server_eval_rows(W, m, n, Xh, B, Yh, m, m + 5);
    uint32_t *vL = arr((size_t)ell * B), *vR = arr((size_t)ell * B);
    uint8_t *acc = (uint8_t *)calloc(B ? B : 1, 1);
    orc_verify(m, n, r, yp1, yp2, yv1, yv2, Q, Xh, Yh, B, eyi, eyv, ty, ell, vL, vR, acc);
    for (uint32_t b = 0; b < B; b++)
        if (!acc[b]) {
            fprintf(stderr, "honest response rejected (m=%u n=%u)\n", m, n);
            exit(2);
        }
    orc_decode(PT, m, Yh, B, exi, exv, tx, Y);
    /* decode(server(encode(x))) = W x */
    uint32_t *Yp = arr((size_t)B * m);
    orc_server_eval(W, m, n, X, B, Yp);
    if (memcmp(Y, Yp, (size_t)B * m * sizeof(uint32_t)) != 0) {
        fprintf(stderr, "completeness failed (m=%u n=%u)\n", m, n);
        exit(3);
    }
    /* batch verification over two claims of the same matrix */
    uint32_t Bb = 2, r2 = 2, t2 = ty < 2 * n ? ty : 1;
    uint64_t k2 = (uint64_t)Bb * n, N2 = k2 * r2;
    uint32_t *qp1 = arr(N2), *qp2 = arr(N2), *w1 = arr(N2), *w2 = arr(N2);
    orc_sample_code((uint32_t)k2, r2, seed, 5, qp1, qp2, w1, w2);
    uint32_t *Qs = arr(2 * Ny * n), *Qaux = arr(Ny * N2), *ut = arr((size_t)ell * k2);
    memcpy(Qs, Q, Ny * n * sizeof(uint32_t));
    memcpy(Qs + Ny * n, Q, Ny * n * sizeof(uint32_t));
    orc_batch_aux(Bb, (uint32_t)Ny, n, Qs, r2, qp1, qp2, w1, w2, Qaux);
    orc_batch_project(Bb, (uint32_t)Ny, n, Qs, eyi, eyv, ty, ell, ut);
    uint32_t *e2i = arr((size_t)ell * t2), *e2v = arr((size_t)ell * t2);
    orc_sample_sparse(ell, (uint32_t)N2, t2, seed, 6, e2i, e2v);
    uint32_t *bvL = arr((size_t)ell * Bb), *bvR = arr((size_t)ell * Bb), *sL = arr((size_t)ell * ell),
             *sR = arr((size_t)ell * ell);
    uint32_t *X2 = arr(k2), *Y2 = arr((size_t)Bb * m);
    memcpy(X2, X, (size_t)n * sizeof(uint32_t));
    memcpy(X2 + n, X, (size_t)n * sizeof(uint32_t));
    orc_server_eval(W, m, n, X2, Bb, Y2);
    orc_batch_verify(m, n, Bb, r, yp1, yp2, yv1, yv2, r2, qp1, qp2, w1, w2, Qaux, X2, Y2, eyi, eyv, ty, ell, ut, e2i,
                     e2v, t2, ell, bvL, bvR, sL, sR);
    for (uint32_t i = 0; i < ell * Bb; i++)
        if (bvL[i] != bvR[i]) exit(4);
    for (uint32_t i = 0; i < ell * ell; i++)
        if (sL[i] != sR[i]) exit(5);
    uint64_t draws[4];
    orc_sm64_draws(seed, 4, draws);
    free(W); free(xp1); free(xp2); free(xv1); free(xv2); free(yp1); free(yp2); free(yv1); free(yv2);
    free(X); free(Xh); free(Yh); free(Y); free(Yp); free(exi); free(exv); free(eyi); free(eyv); free(PT); free(Q);
    free(vL); free(vR); free(acc); free(qp1); free(qp2); free(w1); free(w2); free(Qs); free(Qaux); free(ut);
    free(e2i); free(e2v); free(bvL); free(bvR); free(sL); free(sR); free(X2); free(Y2);
}

int main(void) {
    run(1, 1, 1, 1, 1, 1, 1, 1);          /* the smallest problem: N = 1 */
    run(3, 5, 2, 2, 3, 2, 2, 2);          /* ragged, t close to N */
    run(17, 9, 3, 3, 27, 31, 2, 3);       /* t_x = Nx: full support */
    run(40, 33, 4, 3, 6, 31, 3, 4);
    run(64, 64, 1, 8, 160, 31, 2, 5);     /* the paper's rate and noise weight */
    orc_ops_reset();
    printf("ok %llu\n", (unsigned long long)orc_ops_count());
    return 0;
}
