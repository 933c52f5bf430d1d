// C ABI of the pvMVMD hot-path library (declared in include/mvk.h).
//
// This layer validates sizes, owns the per-(device, stream) workspace and
// enqueues the kernels; all arithmetic happens in the kernels.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <sys/random.h>

#include <algorithm>
#include <cstdlib>
#include <initializer_list>
#include <map>
#include <mutex>
#include <utility>
#include <vector>

#include "mvk.h"
#include "field.h"
#include "mvk_internal.h"

namespace mvk {
namespace {

struct Workspace {
    void* ptr = nullptr;
    size_t size = 0;  // bytes of the whole buffer
    size_t ctrl = 0;  // bytes of the control region at its start
};

std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, Workspace>* g_ws = nullptr;
// Buffers replaced by a growth: graphs captured before the growth still hold
// their addresses, so they live until mvk_workspace_release.
std::vector<void*>* g_ws_retired = nullptr;

// True if `s` is capturing a graph (no allocation may happen then).
bool capturing(hipStream_t s) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return cs != hipStreamCaptureStatusNone;
}

// The first kCtrlBase bytes of every workspace hold control words; a call may
// ask for a larger control region.  The control region is zeroed when the
// workspace is allocated, and kernels that use it leave it zero.
constexpr size_t kCtrlBase = 256;

// Returns a device buffer of at least `bytes` private to (current device, s),
// placed after the control region of at least `ctrl_bytes` (>= kCtrlBase;
// *ctrl, may be null).  A growth retires the old buffer (earlier calls and
// captured graphs may still use it) and allocates one at least 1.5 times as
// large; pointers from earlier requests then refer to the retired buffer, so a
// call takes everything it needs from one workspace() request.  Under graph
// capture a growth is refused (MVK_ECAPTURE).
mvk_status workspace(hipStream_t s, size_t bytes, void** out, uint32_t** ctrl = nullptr, size_t ctrl_bytes = 0) {
    ctrl_bytes = ctrl_bytes < kCtrlBase ? kCtrlBase : (ctrl_bytes + 255) & ~(size_t)255;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return MVK_EHIP;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    if (!g_ws) g_ws = new std::map<std::pair<int, hipStream_t>, Workspace>();
    if (!g_ws_retired) g_ws_retired = new std::vector<void*>();
    Workspace& w = (*g_ws)[std::make_pair(dev, s)];
    const size_t need_ctrl = ctrl_bytes > w.ctrl ? ctrl_bytes : w.ctrl;
    if (w.size < need_ctrl + bytes || w.ctrl < need_ctrl) {
        if (capturing(s)) return MVK_ECAPTURE;
        size_t sz = need_ctrl + bytes;
        if (sz < w.size + w.size / 2) sz = w.size + w.size / 2;
        sz = sz < ((size_t)1 << 20) ? ((size_t)1 << 20) : sz;
        sz = (sz + 4095) & ~(size_t)4095;
        void* fresh = nullptr;
        if (hipMalloc(&fresh, sz) != hipSuccess) {
            (void)hipGetLastError();
            return MVK_ENOMEM;
        }
        // zero the new control region in stream order (the retired buffer may
        // still be in use by work queued earlier on `s`)
        if (launch_fill_u32((uint32_t*)fresh, need_ctrl / 4, 0u, s) != hipSuccess) {
            (void)hipFree(fresh);
            return MVK_EHIP;
        }
        if (w.ptr) g_ws_retired->push_back(w.ptr);
        w.ptr = fresh;
        w.size = sz;
        w.ctrl = need_ctrl;
    }
    *out = (char*)w.ptr + w.ctrl;
    if (ctrl) *ctrl = (uint32_t*)w.ptr;
    return MVK_OK;
}

inline mvk_status hip_status(hipError_t e) { return e == hipSuccess ? MVK_OK : MVK_EHIP; }

// MVK_VALIDATE=1 in the environment: the pvMVMD calls check that their field
// inputs are canonical before enqueuing anything else.
bool validate_mode() {
    const char* v = getenv("MVK_VALIDATE");
    return v && v[0] == '1' && v[1] == '\0';
}

// MVK_ERANGE if a[0, count) holds a word >= p, counted into the device word w.
// Waits for the stream (the validation mode is synchronous).
mvk_status check_canonical_at(const uint32_t* a, size_t count, uint32_t* w, hipStream_t s) {
    uint32_t bad = 0;
    if (launch_fill_u32(w, 1, 0u, s) != hipSuccess) return MVK_EHIP;
    if (launch_count_noncanonical(a, count, w, s) != hipSuccess) return MVK_EHIP;
    if (hipMemcpyAsync(&bad, w, sizeof(uint32_t), hipMemcpyDeviceToHost, s) != hipSuccess) return MVK_EHIP;
    if (hipStreamSynchronize(s) != hipSuccess) return MVK_EHIP;
    return bad ? MVK_ERANGE : MVK_OK;
}

// check_canonical_at with one device word per device, for this check.
mvk_status check_canonical(const uint32_t* a, size_t count, hipStream_t s) {
    if (!a || count == 0) return MVK_OK;
    static std::mutex mu;
    static std::map<int, uint32_t*> words;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return MVK_EHIP;
    std::lock_guard<std::mutex> lk(mu);
    uint32_t*& w = words[dev];
    if (!w && hipMalloc(&w, sizeof(uint32_t)) != hipSuccess) {
        (void)hipGetLastError();
        w = nullptr;
        return MVK_ENOMEM;
    }
    return check_canonical_at(a, count, w, s);
}

// check_canonical over several arrays; nulls are skipped.
mvk_status check_all(hipStream_t s, std::initializer_list<std::pair<const uint32_t*, size_t>> arrays) {
    for (const auto& a : arrays) {
        const mvk_status st = check_canonical(a.first, a.second, s);
        if (st) return st;
    }
    return MVK_OK;
}

inline size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

// True if a*b elements of `elem` bytes exceed 2^62 bytes: no such buffer can
// exist, and the size arithmetic below would wrap; the call returns MVK_ERANGE.
inline bool too_big(uint64_t a, uint64_t b, uint64_t elem) {
    return a != 0 && b > ((1ull << 62) / elem) / a;
}

// Row and query counts of the server product: below 2^31 each (the launch
// grids divide them with 32-bit rounding up), and W and Yhat below 2^62 bytes.
inline bool server_dims_too_big(uint32_t m, uint32_t n, uint32_t B) {
    return m > 0x7fffffffu || B > 0x7fffffffu || too_big(m, B, 4) || too_big(m, n, 1);
}

// Vectors per call of the syndrome kernels: the count is a grid dimension of
// the segmented form.
constexpr uint32_t kMaxSynCount = 65535u;

mvk_status check_code(const mvk_code* c, uint32_t k) {
    if (!c || !c->pi1 || !c->pi2 || !c->v1 || !c->v2) return MVK_EINVAL;
    if (c->k != k || c->r == 0 || k == 0) return MVK_EINVAL;
    if ((uint64_t)c->k * c->r > 0x7fffffffull) return MVK_ERANGE;
    return MVK_OK;
}

mvk_status check_key(const mvk_key* key) {
    if (!key || key->m == 0 || key->n == 0) return MVK_EINVAL;
    if (key->n > MVK_MAX_N) return MVK_ERANGE;
    mvk_status st = check_code(&key->cx, key->n);
    if (st) return st;
    return check_code(&key->cy, key->m);
}

// Challenges of Verify: 1 <= ell <= kMaxEll repetitions of t_y positions < Ny.
mvk_status check_challenges(const mvk_key* key, const mvk_sparse* ey) {
    if (!ey || ey->count == 0 || ey->t == 0 || !ey->idx || !ey->val) return MVK_EINVAL;
    if (ey->count > kMaxEll) return MVK_ERANGE;
    if ((uint64_t)ey->t > (uint64_t)key->cy.r * key->m) return MVK_EINVAL;
    return MVK_OK;
}

mvk_status check_decode_verify(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                               const mvk_sparse* ex, const mvk_sparse* ey, const uint32_t* Y,
                               const uint32_t* accept) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (B == 0) return MVK_OK;
    if (!key->PT || !key->Q || !Xhat || !Yhat || !Y || !accept || !ex) return MVK_EINVAL;
    if (ex->count != B || (ex->t && (!ex->idx || !ex->val))) return MVK_EINVAL;
    if ((uint64_t)ex->t > (uint64_t)key->cx.r * key->n) return MVK_EINVAL;
    st = check_challenges(key, ey);
    if (st) return st;
    if (B > 65535u) return MVK_ERANGE;
    return MVK_OK;
}

hipError_t launch_dv(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                     const mvk_sparse* ex, const mvk_sparse* ey, const uint32_t* R, uint32_t* Y, uint32_t* vL,
                     uint32_t* vR, uint32_t* accept, uint32_t* ctrl, hipStream_t s) {
    const uint32_t m = key->m, n = key->n;
    const uint32_t Nx = key->cx.r * n, Ny = key->cy.r * m;
    return launch_decode_verify(key->PT, key->Q, m, n, Nx, Ny, Xhat, Yhat, B, ex->idx, ex->val, ex->t, ey->idx,
                                ey->val, ey->t, ey->count, R, Y, ctrl, vL, vR, accept, s);
}

}  // namespace
}  // namespace mvk

using namespace mvk;

namespace {
mvk_status server_eval_impl(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B,
                            uint32_t* Yhat, int32_t path, bool packed, void* stream) {
    if (path != MVK_PATH_AUTO && path != MVK_PATH_VALU && path != MVK_PATH_MFMA) return MVK_EINVAL;
    if (packed && path == MVK_PATH_VALU) return MVK_EINVAL;
    if (m == 0 || B == 0) return MVK_OK;
    if (!Yhat) return MVK_EINVAL;
    if (server_dims_too_big(m, n, B)) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    if (n == 0) return hip_status(launch_fill_u32(Yhat, (size_t)m * B, 0u, s));
    if (!W || !Xhat) return MVK_EINVAL;
    if (n > MVK_MAX_N) return MVK_ERANGE;
    if (packed && (uintptr_t)W % 16 != 0) return MVK_EINVAL;
    if (validate_mode()) {
        const mvk_status st = check_canonical(Xhat, (size_t)B * n, s);
        if (st) return st;
    }
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    const ServerEvalPlan pl = server_eval_plan(m, n, B, path, packed);
    if (pl.ws_bytes || pl.ctrl_words) {
        const mvk_status st = workspace(s, pl.ws_bytes, &ws, &ctrl, kCtrlBase + 4 * pl.ctrl_words);
        if (st) return st;
    }
    // the row-block counters follow the first kCtrlBase bytes of the control region
    uint32_t* counters = ctrl ? (uint32_t*)((char*)ctrl + kCtrlBase) : nullptr;
    return hip_status(launch_server_eval(W, m, n, Xhat, B, Yhat, path, packed, ws, counters, s));
}
}  // namespace

extern "C" {

const char* mvk_status_str(mvk_status s) {
    switch (s) {
        case MVK_OK: return "ok";
        case MVK_EINVAL: return "invalid argument";
        case MVK_ERANGE: return "size or value out of range";
        case MVK_ENOMEM: return "out of device memory";
        case MVK_EHIP: return "HIP runtime error";
        case MVK_ERANDOM: return "the operating system's random source failed";
        case MVK_ECAPTURE: return "the workspace would have to grow during graph capture";
        default: return "unknown status";
    }
}

int32_t mvk_abi_version(void) { return MVK_ABI_VERSION; }

uint32_t mvk_field_modulus(void) { return mvk::kP; }

mvk_status mvk_server_eval(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B,
                           uint32_t* Yhat, void* stream) {
    return mvk_server_eval_path(W, m, n, Xhat, B, Yhat, MVK_PATH_AUTO, stream);
}

mvk_status mvk_server_eval_path(const int8_t* W, uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B,
                                uint32_t* Yhat, int32_t path, void* stream) {
    return server_eval_impl(W, m, n, Xhat, B, Yhat, path, false, stream);
}

size_t mvk_packed_weight_bytes(uint32_t m, uint32_t n) { return (m && n) ? packed_w_bytes(m, n) : 0; }

mvk_status mvk_pack_weights(const int8_t* W, uint32_t m, uint32_t n, int8_t* Wp, void* stream) {
    if (m == 0 || n == 0) return MVK_OK;
    if (!W || !Wp) return MVK_EINVAL;
    if (server_dims_too_big(m, n, 1)) return MVK_ERANGE;
    if ((uintptr_t)Wp % 16 != 0) return MVK_EINVAL;
    return hip_status(launch_pack_w(W, m, n, Wp, (hipStream_t)stream));
}

mvk_status mvk_server_eval_packed(const int8_t* Wp, uint32_t m, uint32_t n, const uint32_t* Xhat, uint32_t B,
                                  uint32_t* Yhat, void* stream) {
    return server_eval_impl(Wp, m, n, Xhat, B, Yhat, MVK_PATH_AUTO, true, stream);
}

mvk_status mvk_server_eval_packed_group(const int8_t* Wp, uint32_t G, uint32_t m, uint32_t n, const uint32_t* Xhat,
                                        uint32_t B, uint32_t* const* Yhat, void* stream) {
    if (G == 0 || G > MVK_MAX_GROUP || !Yhat) return MVK_EINVAL;
    if (G > 1 && m % 16 != 0) return MVK_EINVAL;
    for (uint32_t g = 0; g < G; ++g)
        if (!Yhat[g]) return MVK_EINVAL;
    if (m == 0 || B == 0) return MVK_OK;
    if (server_dims_too_big(G * (uint64_t)m > 0xffffffffull ? 0xffffffffu : G * m, n, B)) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    if (n == 0) {
        for (uint32_t g = 0; g < G; ++g)
            if (launch_fill_u32(Yhat[g], (size_t)m * B, 0u, s) != hipSuccess) return MVK_EHIP;
        return MVK_OK;
    }
    if (!Wp || !Xhat || (uintptr_t)Wp % 16 != 0) return MVK_EINVAL;
    if (n > MVK_MAX_N) return MVK_ERANGE;
    if (validate_mode()) {
        const mvk_status st = check_canonical(Xhat, (size_t)B * n, s);
        if (st) return st;
    }
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    const ServerEvalPlan pl = server_eval_plan(G * m, n, B, MVK_PATH_AUTO, true);
    if (pl.ws_bytes || pl.ctrl_words) {
        const mvk_status st = workspace(s, pl.ws_bytes, &ws, &ctrl, kCtrlBase + 4 * pl.ctrl_words);
        if (st) return st;
    }
    uint32_t* counters = ctrl ? (uint32_t*)((char*)ctrl + kCtrlBase) : nullptr;
    return hip_status(
        launch_server_eval_group(Wp, G, m, n, Xhat, B, Yhat, MVK_PATH_AUTO, true, ws, counters, s));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free server product: the scratch of the batched kernels (digit
// matrix, split-k partial sums and accumulators, row-block counters) lives in
// one statically sized device array instead of the per-stream workspace.
// ---------------------------------------------------------------------------
namespace {
constexpr size_t kScratchCtrlBytes = 64u << 10;  // word 0: validation count; control words from byte 256
constexpr size_t kScratchDataBytes = (size_t)MVK_STATIC_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kScratchCtrlBytes + kScratchDataBytes];

constexpr int kScratchMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kScratchMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up once
// per device (with that device current) and kept.
mvk_status scratch_address(uint8_t** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return MVK_EHIP;
    if (dev < 0 || dev >= kScratchMaxDevices) return MVK_ERANGE;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return MVK_EHIP;
        }
        g_scratch_ptr[dev] = (uint8_t*)p;
    }
    *out = g_scratch_ptr[dev];
    return MVK_OK;
}
}  // namespace

extern "C" {

mvk_status mvk_server_eval_packed_static(const int8_t* Wp, uint32_t m, uint32_t n, const uint32_t* Xhat,
                                         uint32_t B, uint32_t* Yhat, void* stream) {
    if (m == 0 || B == 0) return MVK_OK;
    if (!Yhat) return MVK_EINVAL;
    if (server_dims_too_big(m, n, B)) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    if (n == 0) return hip_status(launch_fill_u32(Yhat, (size_t)m * B, 0u, s));
    if (!Wp || !Xhat || (uintptr_t)Wp % 16 != 0) return MVK_EINVAL;
    if (n > MVK_MAX_N) return MVK_ERANGE;
    const ServerEvalPlan pl = server_eval_plan(m, n, B, MVK_PATH_AUTO, true);
    // the array holds the control words (from byte 256: counters and split-k
    // accumulators), then the data; at least the first 64 KiB are control
    const size_t ctrl_bytes = std::max(kScratchCtrlBytes, align_up(256 + 4 * pl.ctrl_words));
    if (pl.ws_bytes > kScratchCtrlBytes + kScratchDataBytes - ctrl_bytes) return MVK_ERANGE;
    const bool validate = validate_mode();
    if (!pl.ws_bytes && !pl.ctrl_words && !validate)
        return hip_status(launch_server_eval(Wp, m, n, Xhat, B, Yhat, MVK_PATH_AUTO, true, nullptr, nullptr, s));
    uint8_t* base = nullptr;
    mvk_status st = scratch_address(&base);
    if (st) return st;
    if (validate && (st = check_canonical_at(Xhat, (size_t)B * n, (uint32_t*)base, s))) return st;
    uint32_t* counters = (uint32_t*)(base + 256);
    // the counters start at zero for every call (a kernel, so that the call can be captured)
    if (pl.ctrl_words && launch_fill_u32(counters, pl.ctrl_words, 0u, s) != hipSuccess) return MVK_EHIP;
    return hip_status(launch_server_eval(Wp, m, n, Xhat, B, Yhat, MVK_PATH_AUTO, true, base + ctrl_bytes, counters,
                                         s));
}

mvk_status mvk_keygen(const mvk_key* key, const int8_t* W, void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (!W || !key->PT || !key->Q) return MVK_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t m = key->m, n = key->n;
    const size_t Nx = (size_t)key->cx.r * n, Ny = (size_t)key->cy.r * m;
    if (too_big(m, n, 1) || too_big(Nx, m, 4) || too_big(Ny, n, 4)) return MVK_ERANGE;
    if (m > kMaxEncVectors || n > kMaxEncVectors) return MVK_ERANGE;
    const size_t wt_bytes = align_up((size_t)m * n);
    const size_t t3_bytes = align_up((Nx * m > Ny * n ? Nx * m : Ny * n) * sizeof(uint32_t));
    const size_t seg_words = std::max(encT_seg_words(Nx, m), encT_seg_words(Ny, n));
    void* ws = nullptr;
    st = workspace(s, wt_bytes + t3_bytes + seg_words * sizeof(uint32_t), &ws);
    if (st) return st;
    int8_t* WT = (int8_t*)ws;
    uint32_t* t3 = (uint32_t*)((char*)ws + wt_bytes);
    uint32_t* seg = (uint32_t*)((char*)ws + wt_bytes + t3_bytes);
    // P^T = Gx^T W^T: vector i is row i of W = column i of W^T (n positions).
    hipError_t e = launch_transpose_i8(W, m, n, WT, s);
    if (e == hipSuccess) e = launch_encT_i8(key->cx, WT, (size_t)m, 1, m, t3, seg, key->PT, (size_t)m, 1, s);
    // Q = Gy^T W: vector k is column k of W (m positions).
    if (e == hipSuccess) e = launch_encT_i8(key->cy, W, (size_t)n, 1, n, t3, seg, key->Q, (size_t)n, 1, s);
    return hip_status(e);
}

mvk_status mvk_encode(const mvk_key* key, const uint32_t* X, uint32_t B, const mvk_sparse* ex, uint32_t* Xhat,
                      void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (B == 0) return MVK_OK;
    if (!X || !Xhat || !ex || ex->count != B || (ex->t && (!ex->idx || !ex->val))) return MVK_EINVAL;
    if (B > kMaxSynCount) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    const size_t Nx = (size_t)key->cx.r * key->n;
    if (ex->t > Nx) return MVK_EINVAL;
    if (validate_mode() && (st = check_all(s, {{X, (size_t)B * key->n}, {ex->val, (size_t)B * ex->t}}))) return st;
    void* ws = nullptr;
    st = workspace(s, syn_scratch_bytes(B, Nx), &ws);
    if (st) return st;
    return hip_status(launch_syn_sparse(key->cx, ex->idx, ex->val, ex->t, B, X, (uint32_t*)ws, Xhat, s));
}

mvk_status mvk_verify_prepare(const mvk_key* key, const mvk_sparse* ey, uint32_t* R, void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (!R) return MVK_EINVAL;
    st = check_challenges(key, ey);
    if (st) return st;
    hipStream_t s = (hipStream_t)stream;
    const size_t Ny = (size_t)key->cy.r * key->m;
    void* ws = nullptr;
    st = workspace(s, syn_scratch_bytes(ey->count, Ny), &ws);
    if (st) return st;
    return hip_status(launch_syn_sparse(key->cy, ey->idx, ey->val, ey->t, ey->count, nullptr, (uint32_t*)ws, R, s));
}

mvk_status mvk_decode_verify_prepared(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                      const mvk_sparse* ex, const mvk_sparse* ey, const uint32_t* R, uint32_t* Y,
                                      uint32_t* vL, uint32_t* vR, uint32_t* accept, void* stream) {
    mvk_status st = check_decode_verify(key, Xhat, Yhat, B, ex, ey, Y, accept);
    if (st || B == 0) return st;
    if (!R) return MVK_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    if (validate_mode() && (st = check_all(s, {{Xhat, (size_t)B * key->n}, {Yhat, (size_t)B * key->m},
                                               {R, (size_t)ey->count * key->m}})))
        return st;
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    st = workspace(s, 0, &ws, &ctrl, dv_ctrl_bytes(key->m, key->n, B, ey->count));
    if (st) return st;
    return hip_status(launch_dv(key, Xhat, Yhat, B, ex, ey, R, Y, vL, vR, accept, ctrl, s));
}

}  // extern "C"

namespace {
// Challenges that decode_verify_run draws itself (the seeded Verify).
struct ChallengeDraw {
    uint64_t seed;
};

// decode_verify after the argument checks; Y may be null (no decryption
// output) and ex may have t = 0 (no gathers of Pᵀ).  With `draw`, the ell
// challenges of t positions that `ey` describes (its idx/val are ignored) are
// first drawn into the workspace from draw->seed (sample.h).
mvk_status decode_verify_run(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                             const mvk_sparse* ey_in, uint32_t* Y, uint32_t* vL, uint32_t* vR, uint32_t* accept,
                             hipStream_t s, const mvk_sparse* ex, const ChallengeDraw* draw = nullptr) {
    const uint32_t m = key->m, ell = ey_in->count;
    const size_t Ny = (size_t)key->cy.r * m;
    const size_t e_bytes = draw ? align_up((size_t)2 * ell * ey_in->t * 4) : 0;
    const size_t r_bytes = align_up((size_t)ell * m * 4);
    const size_t syn_bytes = align_up(syn_scratch_bytes(ell, Ny));
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    const mvk_status st =
        workspace(s, e_bytes + r_bytes + syn_bytes, &ws, &ctrl, dv_ctrl_bytes(m, key->n, B, ell));
    if (st) return st;
    mvk_sparse drawn = *ey_in;
    if (draw) {
        uint32_t* idx = (uint32_t*)ws;
        uint32_t* val = idx + (size_t)ell * ey_in->t;
        if (launch_sample_sparse(draw->seed, MVK_TAG_CHALLENGE, ell, (uint32_t)Ny, ey_in->t, idx, val, s) !=
            hipSuccess)
            return MVK_EHIP;
        drawn.idx = idx;
        drawn.val = val;
    }
    const mvk_sparse* ey = &drawn;
    uint32_t* rv = (uint32_t*)((char*)ws + e_bytes);
    uint32_t* syn_scratch = (uint32_t*)((char*)ws + e_bytes + r_bytes);
    if (Ny <= kSynScratchAbove &&
        dv_syn_fits(m, key->n, (uint32_t)Ny, B, ell, dv_decode_cols(m, B, key->PT, Yhat, Y, rv))) {
        // one launch: the syndromes overlap the Decrypt and Verify gathers
        const mvk_code& cy = key->cy;
        return hip_status(launch_decode_verify_syn(
            key->PT, key->Q, m, key->n, key->cx.r * key->n, (uint32_t)Ny, Xhat, Yhat, B, ex->idx, ex->val, ex->t,
            ey->idx, ey->val, ey->t, ell, cy.r, cy.pi1, cy.pi2, cy.v1, cy.v2, rv, Y, ctrl, vL, vR, accept, s));
    }
    // r_q = Gy e_q for every repetition (shared by all columns)
    hipError_t e = launch_syn_sparse(key->cy, ey->idx, ey->val, ey->t, ell, nullptr, syn_scratch, rv, s);
    if (e == hipSuccess) e = launch_dv(key, Xhat, Yhat, B, ex, ey, rv, Y, vL, vR, accept, ctrl, s);
    return hip_status(e);
}
}  // namespace

extern "C" {

mvk_status mvk_decode_verify(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                             const mvk_sparse* ex, const mvk_sparse* ey, uint32_t* Y, uint32_t* vL, uint32_t* vR,
                             uint32_t* accept, void* stream) {
    mvk_status st = check_decode_verify(key, Xhat, Yhat, B, ex, ey, Y, accept);
    if (st || B == 0) return st;
    if (validate_mode() && (st = check_all((hipStream_t)stream, {{Xhat, (size_t)B * key->n},
                                                                  {Yhat, (size_t)B * key->m}})))
        return st;
    return decode_verify_run(key, Xhat, Yhat, B, ey, Y, vL, vR, accept, (hipStream_t)stream, ex);
}

mvk_status mvk_verify(const mvk_key* key, const uint32_t* X, const uint32_t* Y, uint32_t B, const mvk_sparse* ey,
                      uint32_t* vL, uint32_t* vR, uint32_t* accept, void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (B == 0) return MVK_OK;
    if (!key->Q || !X || !Y || !accept) return MVK_EINVAL;
    st = check_challenges(key, ey);
    if (st) return st;
    if (B > 65535u) return MVK_ERANGE;
    if (validate_mode() && (st = check_all((hipStream_t)stream, {{X, (size_t)B * key->n}, {Y, (size_t)B * key->m}})))
        return st;
    const mvk_sparse none = {nullptr, nullptr, 0u, B};  // no noise: nothing to decrypt
    return decode_verify_run(key, X, Y, B, ey, nullptr, vL, vR, accept, (hipStream_t)stream, &none);
}

// Control word of the workgroup counters of client_prepare and encode_masked.
constexpr int kPrepCounterWord = 4;

mvk_status mvk_client_prepare(const mvk_key* key, const mvk_sparse* ex, const mvk_sparse* ey, uint32_t* Mx,
                              uint32_t* My, uint32_t* R, uint32_t* U, uint32_t* done_flag, uint32_t done_value,
                              void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (done_flag && done_value == 0) return MVK_EINVAL;
    const uint32_t nx = ex ? ex->count : 0u;
    if (nx) {
        if (!Mx || !My || !key->PT || (ex->t && (!ex->idx || !ex->val))) return MVK_EINVAL;
        if ((uint64_t)ex->t > (uint64_t)key->cx.r * key->n) return MVK_EINVAL;
        if (nx > 65535u) return MVK_ERANGE;
    }
    const uint32_t ny = ey ? ey->count : 0u;
    if (ny) {
        st = check_challenges(key, ey);
        if (st) return st;
        if (!R || !U || !key->Q) return MVK_EINVAL;
    }
    hipStream_t s = (hipStream_t)stream;
    if (nx == 0 && ny == 0) return done_flag ? hip_status(launch_flag_signal(done_flag, done_value, s)) : MVK_OK;
    const size_t scratch = prep_scratch_bytes(&key, 1, nx, ny);
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    st = workspace(s, scratch, &ws, &ctrl, 4 * (kPrepCounterWord + prep_ctrl_words(*key, nx, ny)));
    if (st) return st;
    return hip_status(launch_client_prepare(*key, nx ? ex->idx : nullptr, nx ? ex->val : nullptr, nx ? ex->t : 0u,
                                            nx, ny ? ey->idx : nullptr, ny ? ey->val : nullptr, ny ? ey->t : 0u, ny,
                                            Mx, My, R, U, (uint32_t*)ws, scratch, &ctrl[kPrepCounterWord], done_flag,
                                            done_value, s));
}

mvk_status mvk_client_prepare_group(uint32_t G, const mvk_key* const* keys, const mvk_sparse* ex,
                                    const mvk_sparse* const* ey, uint32_t* Mx, uint32_t* const* My,
                                    uint32_t* const* R, uint32_t* const* U, uint32_t* done_flag, uint32_t done_value,
                                    void* stream) {
    if (G == 0 || G > MVK_MAX_GROUP || !keys) return MVK_EINVAL;
    for (uint32_t g = 0; g < G; ++g) {
        const mvk_status st = check_key(keys[g]);
        if (st) return st;
        const mvk_key &k = *keys[g], &k0 = *keys[0];
        // one shape and one privacy code: the noise and its mask are shared
        if (k.m != k0.m || k.n != k0.n || k.cx.r != k0.cx.r || k.cx.pi1 != k0.cx.pi1 || k.cx.pi2 != k0.cx.pi2 ||
            k.cx.v1 != k0.cx.v1 || k.cx.v2 != k0.cx.v2 || k.cy.r != k0.cy.r)
            return MVK_EINVAL;
    }
    if (done_flag && done_value == 0) return MVK_EINVAL;
    const mvk_key& key = *keys[0];
    const uint32_t nx = ex ? ex->count : 0u;
    if (nx) {
        if (!Mx || !My || (ex->t && (!ex->idx || !ex->val))) return MVK_EINVAL;
        if ((uint64_t)ex->t > (uint64_t)key.cx.r * key.n) return MVK_EINVAL;
        if (nx > 65535u) return MVK_ERANGE;
        for (uint32_t g = 0; g < G; ++g)
            if (!My[g] || !keys[g]->PT) return MVK_EINVAL;
    }
    uint32_t ny = 0, ty = 0;
    const uint32_t* eyi[MVK_MAX_GROUP] = {};
    const uint32_t* eyv[MVK_MAX_GROUP] = {};
    if (ey) {
        for (uint32_t g = 0; g < G; ++g) {
            if (!ey[g]) return MVK_EINVAL;
            if (ey[g]->count != ey[0]->count || ey[g]->t != ey[0]->t) return MVK_EINVAL;
        }
        ny = ey[0]->count;
        ty = ey[0]->t;
    }
    if (ny) {
        if (!R || !U) return MVK_EINVAL;
        for (uint32_t g = 0; g < G; ++g) {
            const mvk_status st = check_challenges(keys[g], ey[g]);
            if (st) return st;
            if (!R[g] || !U[g] || !keys[g]->Q) return MVK_EINVAL;
            eyi[g] = ey[g]->idx;
            eyv[g] = ey[g]->val;
        }
    }
    hipStream_t s = (hipStream_t)stream;
    if (nx == 0 && ny == 0) return done_flag ? hip_status(launch_flag_signal(done_flag, done_value, s)) : MVK_OK;
    const size_t scratch = prep_scratch_bytes(keys, G, nx, ny);
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    mvk_status st = workspace(s, scratch, &ws, &ctrl, 4 * (kPrepCounterWord + prep_ctrl_words(keys, G, nx, ny)));
    if (st) return st;
    return hip_status(launch_client_prepare_group(G, keys, nx ? ex->idx : nullptr, nx ? ex->val : nullptr,
                                                  nx ? ex->t : 0u, nx, eyi, eyv, ty, ny, Mx, My, R, U,
                                                  (uint32_t*)ws, scratch, &ctrl[kPrepCounterWord], done_flag,
                                                  done_value, s));
}

mvk_status mvk_client_prepare_multi(uint32_t G, const mvk_key* const* keys, const mvk_sparse* const* ex,
                                    const mvk_sparse* const* ey, uint32_t* const* Mx, uint32_t* const* My,
                                    uint32_t* const* R, uint32_t* const* U, uint32_t* const* done_flags,
                                    uint32_t done_value, void* stream) {
    if (G == 0 || G > MVK_MAX_PREP || !keys) return MVK_EINVAL;
    PrepInputDesc ins[kMaxPrep];
    PrepProbDesc probs[kMaxPrep];
    uint32_t* flags[kMaxPrep];
    uint32_t NI = 0, nflags = 0;
    bool work = false;
    for (uint32_t g = 0; g < G; ++g) {
        mvk_status st = check_key(keys[g]);
        if (st) return st;
        const mvk_key& k = *keys[g];
        uint32_t in = kPrepNoInput;
        const mvk_sparse* e = ex ? ex[g] : nullptr;
        if (e && e->count) {
            if (!Mx || !Mx[g] || !My || !My[g] || !k.PT || (e->t && (!e->idx || !e->val))) return MVK_EINVAL;
            if ((uint64_t)e->t > (uint64_t)k.cx.r * k.n) return MVK_EINVAL;
            if (e->count > 65535u) return MVK_ERANGE;
            for (uint32_t j = 0; j < NI; ++j) {
                if (ins[j].Mx != Mx[g]) continue;
                // a shared input: the same noise vectors over the same privacy code
                const mvk_code& c = *ins[j].cx;
                if (ins[j].idx != e->idx || ins[j].val != e->val || ins[j].t != e->t || ins[j].count != e->count ||
                    c.k != k.cx.k || c.r != k.cx.r || c.pi1 != k.cx.pi1 || c.pi2 != k.cx.pi2 || c.v1 != k.cx.v1 ||
                    c.v2 != k.cx.v2)
                    return MVK_EINVAL;
                in = j;
            }
            if (in == kPrepNoInput) {
                ins[NI] = PrepInputDesc{&k.cx, e->idx, e->val, e->t, e->count, Mx[g]};
                in = NI++;
            }
            work = true;
        }
        const mvk_sparse* q = ey ? ey[g] : nullptr;
        const uint32_t ny = q ? q->count : 0u;
        if (ny) {
            st = check_challenges(&k, q);
            if (st) return st;
            if (!R || !R[g] || !U || !U[g] || !k.Q) return MVK_EINVAL;
            work = true;
        }
        probs[g] = PrepProbDesc{&k, in, ny ? q->idx : nullptr, ny ? q->val : nullptr, ny ? q->t : 0u, ny,
                                in != kPrepNoInput ? My[g] : nullptr, ny ? R[g] : nullptr, ny ? U[g] : nullptr};
        if (done_flags && done_flags[g]) {
            bool seen = false;
            for (uint32_t f = 0; f < nflags; ++f) seen = seen || flags[f] == done_flags[g];
            if (!seen) flags[nflags++] = done_flags[g];
        }
    }
    if (nflags && done_value == 0) return MVK_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    if (!work) {
        for (uint32_t f = 0; f < nflags; ++f)
            if (launch_flag_signal(flags[f], done_value, s) != hipSuccess) return MVK_EHIP;
        return MVK_OK;
    }
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    const size_t scratch = prep_scratch_bytes(ins, NI, probs, G);
    const mvk_status st = workspace(s, scratch, &ws, &ctrl, 4 * (kPrepCounterWord + prep_ctrl_words(ins, NI, probs, G)));
    if (st) return st;
    return hip_status(launch_client_prepare_multi(ins, NI, probs, G, (uint32_t*)ws, scratch, &ctrl[kPrepCounterWord],
                                                  nflags ? flags : nullptr, nflags, done_value, s));
}

mvk_status mvk_encode_masked(const mvk_key* key, const uint32_t* X, uint32_t B, const uint32_t* Mx, uint32_t* Xhat,
                             uint32_t* ready_flag, uint32_t ready_value, uint32_t timeout_us, uint32_t* timed_out,
                             void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (ready_flag && (ready_value == 0 || timeout_us == 0)) return MVK_EINVAL;
    if (B == 0 && !ready_flag) return MVK_OK;
    if (B && (!X || !Mx || !Xhat)) return MVK_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    // (Mx may still be in preparation on another stream when a flag orders it)
    if (validate_mode() && (st = check_all(s, {{X, (size_t)B * key->n}, {ready_flag ? nullptr : Mx, (size_t)B * key->n}})))
        return st;
    uint32_t* ctrl = nullptr;
    if (ready_flag) {
        void* ws = nullptr;
        st = workspace(s, 0, &ws, &ctrl);
        if (st) return st;
    }
    return hip_status(launch_add_masks(X, Mx, (size_t)B * key->n, Xhat, ready_flag, ready_value, timeout_us,
                                       timed_out, ctrl ? &ctrl[kPrepCounterWord] : nullptr, s));
}

mvk_status mvk_decode_verify_masked(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat, uint32_t B,
                                    const uint32_t* My, uint32_t ell, const uint32_t* R, const uint32_t* U,
                                    uint32_t* Y, uint32_t* vL, uint32_t* vR, uint32_t* accept, void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (B == 0) return MVK_OK;
    if (!Xhat || !Yhat || !My || !R || !U || !Y || !accept || ell == 0) return MVK_EINVAL;
    if (ell > kMaxEll || B > 65535u) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    if (validate_mode() && (st = check_all(s, {{Xhat, (size_t)B * key->n}, {Yhat, (size_t)B * key->m},
                                               {My, (size_t)B * key->m}, {R, (size_t)ell * key->m},
                                               {U, (size_t)ell * key->n}})))
        return st;
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    st = workspace(s, 0, &ws, &ctrl, dv_ctrl_bytes(key->m, key->n, B, ell));
    if (st) return st;
    return hip_status(launch_decode_verify_masked(key->m, key->n, Xhat, Yhat, B, My, ell, R, U, Y, ctrl, vL, vR,
                                                  accept, s));
}

mvk_status mvk_decode_verify_encode_masked(const mvk_key* key, const uint32_t* Xhat, const uint32_t* Yhat,
                                           uint32_t B, const uint32_t* My, uint32_t ell, const uint32_t* R,
                                           const uint32_t* U, uint32_t* Y, uint32_t* vL, uint32_t* vR,
                                           uint32_t* accept, const uint32_t* X_next, uint32_t B_next,
                                           const uint32_t* Mx_next, uint32_t* Xhat_next, uint32_t* ready_flag,
                                           uint32_t ready_value, uint32_t timeout_us, uint32_t* timed_out,
                                           void* stream) {
    mvk_status st = check_key(key);
    if (st) return st;
    if (ready_flag && (ready_value == 0 || timeout_us == 0)) return MVK_EINVAL;
    if (B_next && (!X_next || !Mx_next || !Xhat_next)) return MVK_EINVAL;
    if (B == 0)
        return mvk_encode_masked(key, X_next, B_next, Mx_next, Xhat_next, ready_flag, ready_value, timeout_us,
                                 timed_out, stream);
    if (B_next == 0 && !ready_flag)
        return mvk_decode_verify_masked(key, Xhat, Yhat, B, My, ell, R, U, Y, vL, vR, accept, stream);
    if (!Xhat || !Yhat || !My || !R || !U || !Y || !accept || ell == 0) return MVK_EINVAL;
    if (ell > kMaxEll || B > 65535u) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    if (validate_mode() &&
        (st = check_all(s, {{Xhat, (size_t)B * key->n}, {Yhat, (size_t)B * key->m}, {My, (size_t)B * key->m},
                            {R, (size_t)ell * key->m}, {U, (size_t)ell * key->n}, {X_next, (size_t)B_next * key->n},
                            {ready_flag ? nullptr : Mx_next, (size_t)B_next * key->n}})))
        return st;
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    // the decode/verify's control words from word 0, the masked encode's
    // counter at word kPrepCounterWord (a word those layouts leave unused)
    st = workspace(s, 0, &ws, &ctrl,
                   std::max(dv_ctrl_bytes(key->m, key->n, B, ell), (size_t)4 * (kPrepCounterWord + 1)));
    if (st) return st;
    return hip_status(launch_client_turn(key->m, key->n, Xhat, Yhat, B, My, ell, R, U, Y, ctrl, vL, vR, accept,
                                         X_next, Mx_next, (size_t)B_next * key->n, Xhat_next, ready_flag,
                                         ready_value, timeout_us, timed_out, &ctrl[kPrepCounterWord], s));
}

mvk_status mvk_decode_verify_masked_group(uint32_t G, const mvk_key* const* keys, const uint32_t* Xhat, uint32_t B,
                                          const uint32_t* const* Yhat, const uint32_t* const* My, uint32_t ell,
                                          const uint32_t* const* R, const uint32_t* const* U, uint32_t* const* Y,
                                          uint32_t* const* vL, uint32_t* const* vR, uint32_t* const* accept,
                                          void* stream) {
    if (G == 0 || G > MVK_MAX_GROUP || !keys || !Yhat || !My || !R || !U || !Y || !accept) return MVK_EINVAL;
    for (uint32_t g = 0; g < G; ++g) {
        const mvk_status st = check_key(keys[g]);
        if (st) return st;
        if (keys[g]->m != keys[0]->m || keys[g]->n != keys[0]->n) return MVK_EINVAL;
    }
    if (B == 0) return MVK_OK;
    if (!Xhat || ell == 0) return MVK_EINVAL;
    for (uint32_t g = 0; g < G; ++g)
        if (!Yhat[g] || !My[g] || !R[g] || !U[g] || !Y[g] || !accept[g]) return MVK_EINVAL;
    if (ell > kMaxEll || B > 65535u) return MVK_ERANGE;
    const uint32_t m = keys[0]->m, n = keys[0]->n;
    hipStream_t s = (hipStream_t)stream;
    if (validate_mode()) {
        mvk_status st = check_canonical(Xhat, (size_t)B * n, s);
        for (uint32_t g = 0; g < G && !st; ++g)
            st = check_all(s, {{Yhat[g], (size_t)B * m}, {My[g], (size_t)B * m}, {R[g], (size_t)ell * m},
                               {U[g], (size_t)ell * n}});
        if (st) return st;
    }
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    const mvk_status st = workspace(s, 0, &ws, &ctrl, 4 * G * dv_group_ctrl_stride(m, n, B, ell));
    if (st) return st;
    return hip_status(launch_decode_verify_masked_group(G, m, n, Xhat, B, Yhat, My, ell, R, U, Y, vL, vR, accept,
                                                        ctrl, s));
}

mvk_status mvk_flag_signal(uint32_t* flag, uint32_t value, void* stream) {
    if (!flag || value == 0) return MVK_EINVAL;
    return hip_status(launch_flag_signal(flag, value, (hipStream_t)stream));
}

mvk_status mvk_flag_wait(uint32_t* flag, uint32_t value, uint32_t timeout_us, uint32_t* timed_out, void* stream) {
    if (!flag || value == 0 || timeout_us == 0) return MVK_EINVAL;
    return hip_status(launch_flag_wait(flag, value, timeout_us, timed_out, (hipStream_t)stream));
}

mvk_status mvk_batch_preprocess(uint32_t B, const uint32_t* const* Q, uint32_t N, uint32_t n, const mvk_code* c2,
                                uint32_t* QtT, uint32_t* Qaux, void* stream) {
    if (B == 0 || N == 0 || n == 0 || !Q || !c2 || !QtT || !Qaux) return MVK_EINVAL;
    const uint64_t Bn = (uint64_t)B * n;
    if (Bn > 0x7fffffffull) return MVK_ERANGE;
    mvk_status st = check_code(c2, (uint32_t)Bn);
    if (st) return st;
    for (uint32_t b = 0; b < B; ++b)
        if (!Q[b]) return MVK_EINVAL;
    const uint64_t N2 = Bn * c2->r;
    if (too_big(N, N2, sizeof(uint32_t))) return MVK_ERANGE;
    if (N > kMaxEncVectors) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    const size_t t3_bytes = align_up((size_t)N * N2 * sizeof(uint32_t));  // column scratch of the batched encoder
    st = workspace(s, t3_bytes + encT_seg_words(N2, N) * sizeof(uint32_t), &ws);
    if (st) return st;
    for (uint32_t b = 0; b < B; ++b) {
        const hipError_t e = hipMemcpy2DAsync(QtT + (size_t)b * n, Bn * sizeof(uint32_t), Q[b], (size_t)n * 4,
                                              (size_t)n * 4, N, hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return MVK_EHIP;
    }
    return hip_status(launch_encT_u32(*c2, QtT, 1, Bn, N, (uint32_t*)ws, (uint32_t*)((char*)ws + t3_bytes), Qaux, 1,
                                      N2, s));
}

mvk_status mvk_batch_project(const uint32_t* QtT, uint32_t N, uint32_t n, uint32_t B, const mvk_sparse* e,
                             uint32_t* Ut, void* stream) {
    if (!QtT || !Ut || !e || N == 0 || n == 0 || B == 0) return MVK_EINVAL;
    if ((uint64_t)B * n > 0x7fffffffull) return MVK_ERANGE;
    if (e->count == 0 || e->t == 0 || !e->idx || !e->val || e->t > N) return MVK_EINVAL;
    if (e->count > kMaxEll) return MVK_ERANGE;
    return hip_status(launch_gather_rows(QtT, B * n, N, e->idx, e->val, e->t, e->count, Ut, (hipStream_t)stream));
}

mvk_status mvk_batch_verify(const mvk_code* cy, const mvk_code* c2, const uint32_t* Qaux, uint32_t m, uint32_t n,
                            uint32_t B, const uint32_t* X, const uint32_t* Y, const mvk_sparse* e, const uint32_t* Ut,
                            const mvk_sparse* e2, uint32_t* vL, uint32_t* vR, uint32_t* sL, uint32_t* sR,
                            uint32_t* accept, void* stream) {
    if (m == 0 || n == 0 || B == 0) return m && n ? MVK_OK : MVK_EINVAL;
    const uint64_t Bn = (uint64_t)B * n;
    if (Bn > 0x7fffffffull || B > 65535u) return MVK_ERANGE;
    mvk_status st = check_code(cy, m);
    if (st) return st;
    st = check_code(c2, (uint32_t)Bn);
    if (st) return st;
    if (!Qaux || !X || !Y || !Ut || !accept || !e || !e2) return MVK_EINVAL;
    const uint64_t N = (uint64_t)cy->r * m, N2 = Bn * c2->r;
    for (const mvk_sparse* v : {e, e2}) {
        if (v->count == 0 || v->t == 0 || !v->idx || !v->val) return MVK_EINVAL;
        if (v->count > kMaxEll) return MVK_ERANGE;
    }
    if (e->t > N || e2->t > N2 || N2 > 0x7fffffffull) return MVK_EINVAL;
    const uint32_t ell = e->count, ell2 = e2->count;
    hipStream_t s = (hipStream_t)stream;
    const size_t r_bytes = align_up((size_t)ell * m * 4), rs_bytes = align_up((size_t)ell2 * Bn * 4);
    size_t syn_bytes = 0;
    syn_bytes = syn_scratch_bytes(ell, N);
    if (syn_scratch_bytes(ell2, N2) > syn_bytes) syn_bytes = syn_scratch_bytes(ell2, N2);
    void* ws = nullptr;
    uint32_t* ctrl = nullptr;
    st = workspace(s, r_bytes + rs_bytes + syn_bytes, &ws, &ctrl, batch_ctrl_bytes(m, n, B, ell, ell2));
    if (st) return st;
    uint32_t* R = (uint32_t*)ws;
    uint32_t* Rs = (uint32_t*)((char*)ws + r_bytes);
    uint32_t* scratch = (uint32_t*)((char*)ws + r_bytes + rs_bytes);
    // primary syndromes R_q = G e_q and secondary syndromes r_j = G' e'_j
    hipError_t err = launch_syn_sparse(*cy, e->idx, e->val, e->t, ell, nullptr, scratch, R, s);
    if (err == hipSuccess) err = launch_syn_sparse(*c2, e2->idx, e2->val, e2->t, ell2, nullptr, scratch, Rs, s);
    if (err == hipSuccess)
        err = launch_batch_check(m, n, B, X, Y, Ut, R, Rs, Qaux, (uint32_t)N, (uint32_t)N2, e->idx, e->val, e->t, ell,
                                 e2->idx, e2->val, e2->t, ell2, ctrl, vL, vR, sL, sR, accept, s);
    return hip_status(err);
}

mvk_status mvk_raa_encode(const mvk_code* code, const uint32_t* w, uint32_t count, uint32_t* out, void* stream) {
    if (!code) return MVK_EINVAL;
    mvk_status st = check_code(code, code->k);
    if (st) return st;
    if (count == 0) return MVK_OK;
    if (!w || !out) return MVK_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    const size_t N = (size_t)code->k * code->r;
    if (too_big(N, count, sizeof(uint32_t))) return MVK_ERANGE;
    if (count > kMaxEncVectors) return MVK_ERANGE;
    void* ws = nullptr;
    const size_t t3_bytes = align_up(N * count * sizeof(uint32_t));
    st = workspace(s, t3_bytes + encT_seg_words(N, count) * sizeof(uint32_t), &ws);
    if (st) return st;
    return hip_status(
        launch_encT_u32(*code, w, 1, code->k, count, (uint32_t*)ws, (uint32_t*)((char*)ws + t3_bytes), out, 1, N, s));
}

mvk_status mvk_raa_syndrome(const mvk_code* code, const uint32_t* v, uint32_t count, uint32_t* out, void* stream) {
    if (!code) return MVK_EINVAL;
    mvk_status st = check_code(code, code->k);
    if (st) return st;
    if (count == 0) return MVK_OK;
    if (!v || !out) return MVK_EINVAL;
    if (count > kMaxSynCount) return MVK_ERANGE;
    hipStream_t s = (hipStream_t)stream;
    const size_t N = (size_t)code->k * code->r;
    void* ws = nullptr;
    st = workspace(s, syn_scratch_bytes(count, N), &ws);
    if (st) return st;
    return hip_status(launch_syn_dense(*code, v, count, (uint32_t*)ws, out, s));
}

mvk_status mvk_stream_read(const void* data, size_t bytes, uint32_t* sink, void* stream) {
    if (bytes == 0) return MVK_OK;
    if (!data || !sink || ((uintptr_t)data & 15) || (bytes & 15)) return MVK_EINVAL;
    return hip_status(launch_stream_read(data, bytes, sink, MVK_STREAM_READ_BLOCKS, (hipStream_t)stream));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Seeded calls (the library draws the method's randomness, sample.h)
// ---------------------------------------------------------------------------
struct mvk_pp {
    mvk_key key;
    void* mem;  // one device allocation: both codes' arrays, PT, Q
};

struct mvk_st {
    mvk_sparse ex;
    void* mem;  // device: idx then val (count x t words each)
};

namespace {
// A seed from the operating system for MVK_SEED_FRESH; other seeds pass through.
mvk_status resolve_seed(uint64_t* seed) {
    if (*seed != MVK_SEED_FRESH) return MVK_OK;
    uint64_t v = 0;
    size_t got = 0;
    while (got < sizeof(v)) {
        const ssize_t r = getrandom((char*)&v + got, sizeof(v) - got, 0);
        if (r <= 0) return MVK_ERANDOM;
        got += (size_t)r;
    }
    *seed = v;
    return MVK_OK;
}
}  // namespace

extern "C" {

mvk_status mvk_workspace_release(void) {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    if (!g_ws_retired || g_ws_retired->empty()) return MVK_OK;
    if (hipDeviceSynchronize() != hipSuccess) return MVK_EHIP;
    for (void* p : *g_ws_retired) (void)hipFree(p);
    g_ws_retired->clear();
    return MVK_OK;
}

mvk_status mvk_stream_create_cu_range(uint32_t first_cu, uint32_t count, void** stream) {
    if (!stream || count == 0) return MVK_EINVAL;
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
        return MVK_EHIP;
    if ((uint64_t)first_cu + count > (uint64_t)ncu) return MVK_EINVAL;
    std::vector<uint32_t> mask(((size_t)ncu + 31) / 32, 0u);
    for (uint32_t c = first_cu; c < first_cu + count; ++c) mask[c / 32] |= 1u << (c % 32);
    hipStream_t s = nullptr;
    if (hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data()) != hipSuccess) {
        (void)hipGetLastError();
        return MVK_EHIP;
    }
    *stream = s;
    return MVK_OK;
}

mvk_status mvk_stream_destroy(void* stream) {
    if (!stream) return MVK_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    if (hipStreamSynchronize(s) != hipSuccess) return MVK_EHIP;
    {
        // the stream's workspaces join the retired buffers (graphs captured on
        // the stream may still hold their addresses): freed by
        // mvk_workspace_release, and a later stream that gets the same handle
        // starts with a fresh workspace
        std::lock_guard<std::mutex> lk(g_ws_mu);
        if (g_ws) {
            for (auto it = g_ws->begin(); it != g_ws->end();) {
                if (it->first.second == s) {
                    if (!g_ws_retired) g_ws_retired = new std::vector<void*>();
                    if (it->second.ptr) g_ws_retired->push_back(it->second.ptr);
                    it = g_ws->erase(it);
                } else {
                    ++it;
                }
            }
        }
    }
    return hip_status(hipStreamDestroy(s));
}

mvk_status mvk_sample_code(uint32_t k, uint32_t r, uint64_t seed, uint64_t tag, uint32_t* pi1, uint32_t* pi2,
                           uint32_t* v1, uint32_t* v2) {
    if (!pi1 || !pi2 || !v1 || !v2 || k == 0 || r == 0) return MVK_EINVAL;
    if ((uint64_t)k * r > 0x7fffffffull) return MVK_ERANGE;
    sample_code_host(k, r, seed, tag, pi1, pi2, v1, v2);
    return MVK_OK;
}

mvk_status mvk_sample_sparse(uint32_t count, uint32_t N, uint32_t t, uint64_t seed, uint64_t tag, uint32_t* idx,
                             uint32_t* val) {
    if (count == 0 || t == 0) return MVK_OK;
    if (!idx || !val || N == 0 || t > N) return MVK_EINVAL;
    sample_sparse_host(count, N, t, seed, tag, idx, val);
    return MVK_OK;
}

mvk_status mvk_keygen_seeded(uint32_t m, uint32_t n, uint32_t r_x, uint32_t r_y, uint64_t code_seed,
                             const int8_t* W, void* stream, mvk_pp** out) {
    if (!out) return MVK_EINVAL;
    *out = nullptr;
    if (!W || m == 0 || n == 0 || r_x == 0 || r_y == 0) return MVK_EINVAL;
    if (n > MVK_MAX_N) return MVK_ERANGE;
    const uint64_t Nx = (uint64_t)r_x * n, Ny = (uint64_t)r_y * m;
    if (Nx > 0x7fffffffull || Ny > 0x7fffffffull) return MVK_ERANGE;
    if (too_big(Nx, m, 4) || too_big(Ny, n, 4)) return MVK_ERANGE;
    mvk_status st = resolve_seed(&code_seed);
    if (st) return st;
    // host draws of both codes: pi1, pi2, v1, v2 of Gx, then of Gy
    std::vector<uint32_t> hx(4 * Nx), hy(4 * Ny);
    sample_code_host(n, r_x, code_seed, MVK_TAG_CODE_X, &hx[0], &hx[Nx], &hx[2 * Nx], &hx[3 * Nx]);
    sample_code_host(m, r_y, code_seed, MVK_TAG_CODE_Y, &hy[0], &hy[Ny], &hy[2 * Ny], &hy[3 * Ny]);
    const size_t cx_bytes = align_up(4 * Nx * 4), cy_bytes = align_up(4 * Ny * 4);
    const size_t pt_bytes = align_up(Nx * m * 4), q_bytes = align_up(Ny * n * 4);
    void* mem = nullptr;
    if (hipMalloc(&mem, cx_bytes + cy_bytes + pt_bytes + q_bytes) != hipSuccess) {
        (void)hipGetLastError();
        return MVK_ENOMEM;
    }
    hipStream_t s = (hipStream_t)stream;
    uint32_t* dx = (uint32_t*)mem;
    uint32_t* dy = (uint32_t*)((char*)mem + cx_bytes);
    mvk_pp* pp = new mvk_pp;
    pp->mem = mem;
    pp->key.m = m;
    pp->key.n = n;
    pp->key.cx = mvk_code{n, r_x, dx, dx + Nx, dx + 2 * Nx, dx + 3 * Nx};
    pp->key.cy = mvk_code{m, r_y, dy, dy + Ny, dy + 2 * Ny, dy + 3 * Ny};
    pp->key.PT = (uint32_t*)((char*)mem + cx_bytes + cy_bytes);
    pp->key.Q = (uint32_t*)((char*)mem + cx_bytes + cy_bytes + pt_bytes);
    // the host arrays must outlive the copies: wait for them
    hipError_t e = hipMemcpyAsync(dx, hx.data(), 4 * Nx * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(dy, hy.data(), 4 * Ny * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    st = e == hipSuccess ? mvk_keygen(&pp->key, W, stream) : MVK_EHIP;
    if (st) {
        (void)hipStreamSynchronize(s);
        (void)hipFree(mem);
        delete pp;
        return st;
    }
    *out = pp;
    return MVK_OK;
}

const mvk_key* mvk_pp_key(const mvk_pp* pp) { return pp ? &pp->key : nullptr; }

void mvk_pp_free(mvk_pp* pp) {
    if (!pp) return;
    (void)hipFree(pp->mem);
    delete pp;
}

mvk_status mvk_encode_seeded(const mvk_key* key, const uint32_t* X, uint32_t B, uint32_t t_x, uint64_t noise_seed,
                             uint32_t* Xhat, mvk_st** st_out, void* stream) {
    if (!st_out) return MVK_EINVAL;
    *st_out = nullptr;
    mvk_status st = check_key(key);
    if (st) return st;
    if (B == 0 || !X || !Xhat) return MVK_EINVAL;
    if (B > kMaxSynCount || t_x > MVK_SEEDED_MAX_T) return MVK_ERANGE;
    const uint64_t Nx = (uint64_t)key->cx.r * key->n;
    if (t_x > Nx) return MVK_EINVAL;
    st = resolve_seed(&noise_seed);
    if (st) return st;
    hipStream_t s = (hipStream_t)stream;
    void* mem = nullptr;
    const size_t words = (size_t)B * t_x;
    if (words && hipMalloc(&mem, 2 * words * 4) != hipSuccess) {
        (void)hipGetLastError();
        return MVK_ENOMEM;
    }
    mvk_st* state = new mvk_st;
    state->mem = mem;
    uint32_t* idx = (uint32_t*)mem;
    state->ex = mvk_sparse{idx, words ? idx + words : nullptr, t_x, B};
    st = hip_status(launch_sample_sparse(noise_seed, MVK_TAG_NOISE, B, (uint32_t)Nx, t_x, idx,
                                         idx ? idx + words : nullptr, s));
    if (!st) st = mvk_encode(key, X, B, &state->ex, Xhat, stream);
    if (st) {
        (void)hipStreamSynchronize(s);
        (void)hipFree(mem);
        delete state;
        return st;
    }
    *st_out = state;
    return MVK_OK;
}

const mvk_sparse* mvk_st_noise(const mvk_st* st) { return st ? &st->ex : nullptr; }

void mvk_st_free(mvk_st* st) {
    if (!st) return;
    if (st->mem) (void)hipFree(st->mem);
    delete st;
}

mvk_status mvk_decode_verify_seeded(const mvk_key* key, const mvk_st* st, const uint32_t* Xhat,
                                    const uint32_t* Yhat, uint32_t t_y, uint32_t ell, uint64_t chal_seed,
                                    uint32_t* Y, uint32_t* vL, uint32_t* vR, uint32_t* accept, void* stream) {
    if (!st) return MVK_EINVAL;
    mvk_status s0 = check_key(key);
    if (s0) return s0;
    if (ell == 0 || t_y == 0) return MVK_EINVAL;
    if (ell > kMaxEll || t_y > MVK_SEEDED_MAX_T) return MVK_ERANGE;
    if ((uint64_t)t_y > (uint64_t)key->cy.r * key->m) return MVK_EINVAL;
    const uint32_t B = st->ex.count;
    // the challenge arrays are drawn inside the call: a stand-in for the checks
    static const uint32_t placeholder = 0;
    const mvk_sparse ey = {&placeholder, &placeholder, t_y, ell};
    s0 = check_decode_verify(key, Xhat, Yhat, B, &st->ex, &ey, Y, accept);
    if (s0 || B == 0) return s0;
    hipStream_t s = (hipStream_t)stream;
    if (validate_mode() && (s0 = check_all(s, {{Xhat, (size_t)B * key->n}, {Yhat, (size_t)B * key->m}})))
        return s0;
    s0 = resolve_seed(&chal_seed);
    if (s0) return s0;
    const ChallengeDraw draw{chal_seed};
    return decode_verify_run(key, Xhat, Yhat, B, &ey, Y, vL, vR, accept, s, &st->ex, &draw);
}

}  // extern "C"
