// Calls the C ABI's host-side argument and size checks (every path below
// returns before any device work) so that a build with UndefinedBehavior-
// Sanitizer on the host code sees the size arithmetic of the checks (CPU
// only; built and run by tests/test_sanitizers.py).
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include "mvk.h"

static int fails = 0;
static void expect(mvk_status got, mvk_status want, const char* what) {
    if (got != want) {
        fprintf(stderr, "%s: got %d, expected %d\n", what, (int)got, (int)want);
        ++fails;
    }
}

int main() {
    void* fake = (void*)0x1000;
    const uint32_t* u = (const uint32_t*)fake;
    uint32_t* w = (uint32_t*)fake;
    const int8_t* W = (const int8_t*)fake;
    expect(mvk_server_eval(W, 4, MVK_MAX_N + 1, u, 1, w, nullptr), MVK_ERANGE, "server_eval n");
    expect(mvk_server_eval_packed_static(W, 28672, 131071, u, 64, w, nullptr), MVK_ERANGE, "static scratch");
    expect(mvk_server_eval_packed_static(W, 0xFFFFFFFFu, 131071, u, 0xFFFFFFFFu, w, nullptr), MVK_ERANGE,
           "static scratch, huge");
    mvk_code cx = {1, 0x7FFFFFFFu, u, u, u, u};
    mvk_code cy = {0x7FFFFFFFu, 1, u, u, u, u};
    mvk_key key = {0x7FFFFFFFu, 1, cx, cy, w, w};
    expect(mvk_keygen(&key, W, nullptr), MVK_ERANGE, "keygen sizes");
    mvk_code big = {1u << 30, 1, u, u, u, u};
    expect(mvk_raa_encode(&big, u, 0xFFFFFFFFu, w, nullptr), MVK_ERANGE, "raa_encode sizes");
    mvk_code small = {8, 2, u, u, u, u};
    expect(mvk_raa_syndrome(&small, u, 65536, w, nullptr), MVK_ERANGE, "raa_syndrome count");
    const uint32_t* qs[1] = {u};
    expect(mvk_batch_preprocess(1, qs, 0xFFFFFFFFu, 1u << 30, &big, w, w, nullptr), MVK_ERANGE, "batch sizes");
    mvk_pp* pp = nullptr;
    expect(mvk_keygen_seeded(1u << 30, 8, 3, 3, 1, W, nullptr, &pp), MVK_ERANGE, "keygen_seeded Ny");
    expect(mvk_keygen_seeded(0xFFFFFFFFu, 0xFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 1, W, nullptr, &pp), MVK_ERANGE,
           "keygen_seeded huge");
    mvk_key k8 = {8, 8, small, small, w, w};
    mvk_st* st = nullptr;
    expect(mvk_encode_seeded(&k8, u, 65536, 4, 1, w, &st, nullptr), MVK_ERANGE, "encode_seeded B");
    expect(mvk_encode_seeded(&k8, u, 2, 0xFFFFFFFFu, 1, w, &st, nullptr), MVK_ERANGE, "encode_seeded t");
    uint32_t a[8], b[8];
    expect(mvk_sample_sparse(1, 4, 5, 0, 0, a, b), MVK_EINVAL, "sample_sparse t > N");
    expect(mvk_sample_code(0xFFFFu, 0xFFFFu, 0, 0, a, a, a, a), MVK_ERANGE, "sample_code N");
    expect(mvk_sample_sparse(2, 8, 3, 0xFFFFFFFFFFFFFFFFull, MVK_TAG_NOISE, a, b), MVK_OK, "sample_sparse");
    // Preparation calls whose syndrome and counter sizes are computed on the
    // host before the workspace is requested (with no device, the request then
    // fails): long challenge blocks (Ny = 18000 > 16384) with 16 challenges,
    // keys sharing an input, and the multi-input form.  Only where no device
    // exists: the arrays are not device memory.
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev == 0) {
        (void)hipGetLastError();
        mvk_code cxs = {200, 1, u, u, u, u}, cyl = {6000, 3, u, u, u, u};
        mvk_key kl = {6000, 200, cxs, cyl, w, w};
        mvk_sparse ex = {u, u, 5, 1}, ey = {u, u, 31, 16};
        expect(mvk_client_prepare(&kl, &ex, &ey, w, w, w, w, nullptr, 0, nullptr), MVK_EHIP, "prepare sizes");
        const mvk_key* ks[2] = {&kl, &kl};
        const mvk_sparse* eys[2] = {&ey, &ey};
        uint32_t* outs[2] = {w, w};
        expect(mvk_client_prepare_group(2, ks, &ex, eys, w, outs, outs, outs, nullptr, 0, nullptr), MVK_EHIP,
               "prepare_group sizes");
        const mvk_sparse* exs[2] = {&ex, nullptr};
        expect(mvk_client_prepare_multi(2, ks, exs, eys, outs, outs, outs, outs, nullptr, 0, nullptr), MVK_EHIP,
               "prepare_multi sizes");
    }
    if (pp || st) ++fails;
    printf(fails ? "FAILED %d\n" : "ok\n", fails);
    return fails ? 1 : 0;
}
