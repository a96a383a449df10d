// C ABI of the HSA library (declarations and contract in include/hsa.h): argument
// validation, default scales, workspace sizes and dispatch to the kernel launchers.
// Nothing is enqueued unless every check passes.
#include <math.h>

#include <atomic>
#include <mutex>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "common.h"
#include "hsa.h"

namespace {

thread_local char g_err[512] = "";

// Kernel-family overrides per op (hsa_attn_set_path), indexed by hsa_op_t.
std::atomic<int> g_path[8];

hsa_attn_status_t fail(hsa_attn_status_t s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return s;
}

hsa_attn_status_t ok() {
    g_err[0] = '\0';
    return HSA_ATTN_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

#define CHECK_PTR(ptr, name)                                                              \
    do {                                                                                  \
        if ((ptr) == nullptr)                                                             \
            return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "%s is NULL", name);              \
        if (!aligned16(ptr))                                                              \
            return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);\
    } while (0)

// Shape checks shared by every op; fills the kernel-side description.
// wide_rows: the call is a selection over inputs of its own, whose rows may be longer than
// an attention head (h = 1, bf16, 256 / 512 / 1024 columns)
hsa_attn_status_t make_dims(const hsa_attn_params_t* p, hsa::Dims* dm, bool wide_rows = false) {
    if (p == nullptr) return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "params is NULL");
    if (p->batch < 0 || p->seqlen < 0)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "batch and seqlen must be >= 0");
    if (p->n_qheads < 1 || p->n_kvheads < 1 || p->n_qheads % p->n_kvheads != 0)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT,
                    "n_qheads (%d) must be a positive multiple of n_kvheads (%d)", p->n_qheads,
                    p->n_kvheads);
    if (p->dtype != HSA_DTYPE_F32 && p->dtype != HSA_DTYPE_BF16)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "unknown dtype %d", (int)p->dtype);
    if (p->topk < 1) return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "topk must be >= 1");
    if (p->chunk < 1) return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "chunk must be >= 1");
    if (p->head_dim < 1) return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "head_dim must be >= 1");
    if ((p->flags & ~(HSA_FLAG_STICK_BREAKING | HSA_FLAG_SOFTMAX_OFF_BY_ONE)) != 0)
        return fail(HSA_ATTN_ERR_UNSUPPORTED,
                    "flags 0x%x: only HSA_FLAG_STICK_BREAKING and HSA_FLAG_SOFTMAX_OFF_BY_ONE "
                    "are supported", p->flags);
    const int h = p->n_qheads / p->n_kvheads;
    if (h > 16) return fail(HSA_ATTN_ERR_UNSUPPORTED, "at most 16 query heads per KV head");
    const bool wide = wide_rows && h == 1 && p->dtype == HSA_DTYPE_BF16 &&
                      (p->head_dim == 256 || p->head_dim == 512 || p->head_dim == 1024);
    if (p->head_dim != 64 && p->head_dim != 128 && !wide)
        return fail(HSA_ATTN_ERR_UNSUPPORTED,
                    "head_dim %d not in {64, 128} (a selection over its own inputs also takes "
                    "256, 512 or 1024 with n_qheads == n_kvheads, bf16)",
                    p->head_dim);
    if (p->chunk != 16 && p->chunk != 32 && p->chunk != 64 && p->chunk != 128)
        return fail(HSA_ATTN_ERR_UNSUPPORTED, "chunk %d not in {16, 32, 64, 128}", p->chunk);
    if (p->topk > 32) return fail(HSA_ATTN_ERR_UNSUPPORTED, "topk %d > 32", p->topk);
    if (p->dtype == HSA_DTYPE_F32 && p->chunk * p->head_dim > 8192)
        return fail(HSA_ATTN_ERR_UNSUPPORTED, "float32 needs chunk * head_dim <= 8192");
    if ((long long)p->batch * p->n_kvheads > 65535)
        return fail(HSA_ATTN_ERR_UNSUPPORTED, "batch * n_kvheads > 65535");
    dm->B = p->batch;
    dm->L = p->seqlen;
    dm->H = p->n_qheads;
    dm->G = p->n_kvheads;
    dm->h = h;
    dm->d = p->head_dim;
    dm->S = p->chunk;
    dm->k = p->topk;
    dm->C = p->seqlen / p->chunk;
    dm->Call = (p->seqlen + p->chunk - 1) / p->chunk;
    dm->beta = p->sm_scale > 0.f ? p->sm_scale : (float)(1.0 / sqrt((double)p->head_dim));
    dm->alpha = p->sel_scale > 0.f ? p->sel_scale : (float)(1.0 / sqrt((double)h * p->head_dim));
    dm->stick = (p->flags & HSA_FLAG_STICK_BREAKING) ? 1 : 0;
    dm->off1 = (p->flags & HSA_FLAG_SOFTMAX_OFF_BY_ONE) ? 1 : 0;
    dm->dwo = nullptr;
    dm->dwacc = 0;
    return HSA_ATTN_OK;
}

hsa_attn_status_t launched(hipError_t e, const char* what) {
    if (e != hipSuccess)
        return fail(HSA_ATTN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

size_t op_workspace(const hsa::Dims& dm, bool in_bf16, int op) {
    switch (op) {
        case HSA_OP_FORWARD: return hsa::forward_workspace(dm, in_bf16);
        case HSA_OP_BACKWARD: return hsa::backward_workspace(dm);
        case HSA_OP_DECODE: return hsa::decode_workspace(dm);
        case HSA_OP_SELECT_BACKWARD: return hsa::select_backward_workspace(dm);
        case HSA_OP_DECODE_HOST: return hsa::decode_host_workspace(dm, in_bf16);
        default: return 0;
    }
}

hsa_attn_status_t check_ws(const hsa::Dims& dm, bool in_bf16, int op, const void* ws,
                           size_t ws_bytes) {
    const size_t need = op_workspace(dm, in_bf16, op);
    if (need == 0) return HSA_ATTN_OK;
    if (ws_bytes < need)
        return fail(HSA_ATTN_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, %zu needed",
                    ws_bytes, need);
    CHECK_PTR(ws, "ws");
    return HSA_ATTN_OK;
}

// A cache in host memory: pinned memory the device can address, from its first to its last
// byte; *dev receives the device-side address of p.
hsa_attn_status_t host_cache(const void* p, size_t bytes, const char* name, const void** dev) {
    if (p == nullptr) return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (!aligned16(p))
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
    for (const char* x : {(const char*)p, (const char*)p + bytes - 1}) {
        hipPointerAttribute_t a;
        if (hipPointerGetAttributes(&a, x) != hipSuccess || a.type != hipMemoryTypeHost) {
            (void)hipGetLastError();
            return fail(HSA_ATTN_ERR_INVALID_ARGUMENT,
                        "%s is not pinned host memory over its %zu bytes (allocate it with "
                        "hipHostMalloc)", name, bytes);
        }
    }
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, const_cast<void*>(p), 0) != hipSuccess || d == nullptr) {
        (void)hipGetLastError();
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "%s has no device mapping", name);
    }
    *dev = d;
    return HSA_ATTN_OK;
}

}  // namespace

extern "C" {

hsa_attn_status_t hsa_landmarks(const hsa_attn_params_t* p, const void* K, void* Kbar,
                                hsa_dtype_t kbar_dtype, int32_t chunk_begin, int32_t chunk_end,
                                void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (kbar_dtype != HSA_DTYPE_F32 && kbar_dtype != HSA_DTYPE_BF16)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "unknown kbar_dtype %d", (int)kbar_dtype);
    if (chunk_begin < 0 || chunk_end < chunk_begin || chunk_end > dm.C)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "chunk range [%d, %d) outside [0, %d]",
                    chunk_begin, chunk_end, dm.C);
    if (dm.B == 0 || chunk_end == chunk_begin) return ok();
    CHECK_PTR(K, "K");
    CHECK_PTR(Kbar, "Kbar");
    return launched(hsa::launch_landmarks(dm, p->dtype == HSA_DTYPE_BF16, K, Kbar,
                                          kbar_dtype == HSA_DTYPE_BF16, chunk_begin, chunk_end,
                                          (hipStream_t)stream),
                    "hsa_landmarks");
}

hsa_attn_status_t hsa_select_topk(const hsa_attn_params_t* p, const void* Q, const float* Kbar,
                                  int32_t* idx, float* w, void* ws, size_t ws_bytes,
                                  void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm, true);
    if (s != HSA_ATTN_OK) return s;
    (void)ws;
    (void)ws_bytes;
    if (dm.B == 0 || dm.L == 0) return ok();
    CHECK_PTR(Q, "Q");
    if (dm.C > 0) CHECK_PTR(Kbar, "Kbar");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    return launched(hsa::launch_select(dm, p->dtype == HSA_DTYPE_BF16, Q, Kbar, idx, w,
                                       (hipStream_t)stream),
                    "hsa_select_topk");
}

hsa_attn_status_t hsa_forward(const hsa_attn_params_t* p, const void* Q, const void* K,
                              const void* V, const int32_t* idx, const float* w, void* O,
                              void* ws, size_t ws_bytes, void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (dm.B == 0 || dm.L == 0) return ok();
    s = check_ws(dm, p->dtype == HSA_DTYPE_BF16, HSA_OP_FORWARD, ws, ws_bytes);
    if (s != HSA_ATTN_OK) return s;
    CHECK_PTR(Q, "Q");
    CHECK_PTR(K, "K");
    CHECK_PTR(V, "V");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    CHECK_PTR(O, "O");
    return launched(hsa::launch_forward(dm, p->dtype == HSA_DTYPE_BF16, Q, K, V, idx, w, O, ws,
                                        (hipStream_t)stream),
                    "hsa_forward");
}

hsa_attn_status_t hsa_backward(const hsa_attn_params_t* p, const void* Q, const void* K,
                               const void* V, const float* Kbar, const int32_t* idx,
                               const float* w, const void* dO, void* dQ, void* dK, void* dV,
                               void* ws, size_t ws_bytes, void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (dm.B == 0 || dm.L == 0) return ok();
    s = check_ws(dm, p->dtype == HSA_DTYPE_BF16, HSA_OP_BACKWARD, ws, ws_bytes);
    if (s != HSA_ATTN_OK) return s;
    CHECK_PTR(Q, "Q");
    CHECK_PTR(K, "K");
    CHECK_PTR(V, "V");
    if (dm.C > 0) CHECK_PTR(Kbar, "Kbar");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    CHECK_PTR(dO, "dO");
    CHECK_PTR(dQ, "dQ");
    CHECK_PTR(dK, "dK");
    CHECK_PTR(dV, "dV");
    return launched(hsa::launch_backward(dm, p->dtype == HSA_DTYPE_BF16, Q, K, V, Kbar, idx, w,
                                         dO, dQ, dK, dV, ws, (hipStream_t)stream),
                    "hsa_backward");
}

hsa_attn_status_t hsa_backward_attn(const hsa_attn_params_t* p, const void* Q, const void* K,
                                    const void* V, const int32_t* idx, const float* w,
                                    const void* dO, void* dQ, void* dK, void* dV, float* dw,
                                    int32_t accumulate_dw, void* ws, size_t ws_bytes,
                                    void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (dm.B == 0 || dm.L == 0) return ok();
    s = check_ws(dm, p->dtype == HSA_DTYPE_BF16, HSA_OP_BACKWARD, ws, ws_bytes);
    if (s != HSA_ATTN_OK) return s;
    CHECK_PTR(Q, "Q");
    CHECK_PTR(K, "K");
    CHECK_PTR(V, "V");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    CHECK_PTR(dO, "dO");
    CHECK_PTR(dQ, "dQ");
    CHECK_PTR(dK, "dK");
    CHECK_PTR(dV, "dV");
    CHECK_PTR(dw, "dw");
    dm.dwo = dw;
    dm.dwacc = accumulate_dw != 0 ? 1 : 0;
    return launched(hsa::launch_backward(dm, p->dtype == HSA_DTYPE_BF16, Q, K, V, nullptr, idx,
                                         w, dO, dQ, dK, dV, ws, (hipStream_t)stream),
                    "hsa_backward_attn");
}

hsa_attn_status_t hsa_select_backward(const hsa_attn_params_t* p, const void* Q,
                                      const float* Kbar, const int32_t* idx, const float* w,
                                      const float* dw, void* dQ, float* dKbar, void* ws,
                                      size_t ws_bytes, void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm, true);
    if (s != HSA_ATTN_OK) return s;
    if (!hsa::select_backward_supported(dm))
        return fail(HSA_ATTN_ERR_UNSUPPORTED, "head_dim %d", dm.d);
    if (dm.B == 0 || dm.L == 0) return ok();
    s = check_ws(dm, p->dtype == HSA_DTYPE_BF16, HSA_OP_SELECT_BACKWARD, ws, ws_bytes);
    if (s != HSA_ATTN_OK) return s;
    CHECK_PTR(Q, "Q");
    if (dm.C > 0) {
        CHECK_PTR(Kbar, "Kbar");
        CHECK_PTR(dKbar, "dKbar");
    }
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    CHECK_PTR(dw, "dw");
    CHECK_PTR(dQ, "dQ");
    return launched(hsa::launch_select_backward(dm, p->dtype == HSA_DTYPE_BF16, Q, Kbar, idx, w,
                                                dw, dQ, dKbar, ws, (hipStream_t)stream),
                    "hsa_select_backward");
}

hsa_attn_status_t hsa_decode(const hsa_attn_params_t* p, const void* q, const void* Kcache,
                             const void* Vcache, const void* Kbar_cache, hsa_dtype_t kbar_dtype,
                             const int32_t* cache_len, void* o, int32_t* idx, float* w, void* ws,
                             size_t ws_bytes, void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (kbar_dtype != HSA_DTYPE_F32 && kbar_dtype != HSA_DTYPE_BF16)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "unknown kbar_dtype %d", (int)kbar_dtype);
    if (dm.G > 16) return fail(HSA_ATTN_ERR_UNSUPPORTED, "decode supports at most 16 KV heads");
    if (dm.B == 0) return ok();
    s = check_ws(dm, p->dtype == HSA_DTYPE_BF16, HSA_OP_DECODE, ws, ws_bytes);
    if (s != HSA_ATTN_OK) return s;
    CHECK_PTR(q, "q");
    CHECK_PTR(o, "o");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    if (dm.C > 0) {
        CHECK_PTR(Kcache, "Kcache");
        CHECK_PTR(Vcache, "Vcache");
        CHECK_PTR(Kbar_cache, "Kbar_cache");
    }
    if (cache_len != nullptr && ((uintptr_t)cache_len & 3u))
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "cache_len is not 4-byte aligned");
    return launched(hsa::launch_decode(dm, p->dtype == HSA_DTYPE_BF16, q, Kcache, Vcache,
                                       Kbar_cache, kbar_dtype == HSA_DTYPE_BF16, cache_len, o,
                                       idx, w, ws, (hipStream_t)stream),
                    "hsa_decode");
}

}  // extern "C"

namespace {

// Scratch memory of hsa_decode_noalloc: one array per GPU, held until the process ends.  In
// host code `scratch` is only a stand-in for the symbol; the device address of each GPU's
// copy comes from hipGetSymbolAddress and is kept per device.
constexpr size_t kNoAllocScratchBytes = (size_t)HSA_DECODE_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The calling thread's current device's copy of `scratch` (resolved once per device, with
// that device current); nullptr with the detail in g_err on failure.
void* device_scratch() {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        fail(HSA_ATTN_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
        return nullptr;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        fail(HSA_ATTN_ERR_UNSUPPORTED, "device %d beyond the %d supported", dev, kMaxDevices);
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || ptr == nullptr) {
            fail(HSA_ATTN_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
            return nullptr;
        }
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

hsa_attn_status_t hsa_decode_noalloc(const hsa_attn_params_t* p, const void* q,
                                     const void* Kcache, const void* Vcache,
                                     const void* Kbar_cache, hsa_dtype_t kbar_dtype,
                                     const int32_t* cache_len, void* o, int32_t* idx, float* w,
                                     void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (kbar_dtype != HSA_DTYPE_F32 && kbar_dtype != HSA_DTYPE_BF16)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "unknown kbar_dtype %d", (int)kbar_dtype);
    if (dm.G > 16) return fail(HSA_ATTN_ERR_UNSUPPORTED, "decode supports at most 16 KV heads");
    if (dm.B == 0) return ok();
    const size_t need = hsa::decode_workspace(dm);
    if (need > kNoAllocScratchBytes)
        return fail(HSA_ATTN_ERR_UNSUPPORTED,
                    "hsa_decode_noalloc: these shapes need %zu bytes of scratch, more than its "
                    "%zu (use hsa_decode with a workspace)", need, kNoAllocScratchBytes);
    CHECK_PTR(q, "q");
    CHECK_PTR(o, "o");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    if (dm.C > 0) {
        CHECK_PTR(Kcache, "Kcache");
        CHECK_PTR(Vcache, "Vcache");
        CHECK_PTR(Kbar_cache, "Kbar_cache");
    }
    if (cache_len != nullptr && ((uintptr_t)cache_len & 3u))
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "cache_len is not 4-byte aligned");
    void* ws = device_scratch();
    if (ws == nullptr) return HSA_ATTN_ERR_HIP;
    return launched(hsa::launch_decode(dm, p->dtype == HSA_DTYPE_BF16, q, Kcache, Vcache,
                                       Kbar_cache, kbar_dtype == HSA_DTYPE_BF16, cache_len, o,
                                       idx, w, ws, (hipStream_t)stream),
                    "hsa_decode_noalloc");
}

hsa_attn_status_t hsa_decode_host(const hsa_attn_params_t* p, const void* q,
                                  const void* Kcache_host, const void* Vcache_host,
                                  const void* Kbar_cache, hsa_dtype_t kbar_dtype,
                                  const int32_t* cache_len, void* o, int32_t* idx, float* w,
                                  void* ws, size_t ws_bytes, void* stream) {
    hsa::Dims dm;
    hsa_attn_status_t s = make_dims(p, &dm);
    if (s != HSA_ATTN_OK) return s;
    if (kbar_dtype != HSA_DTYPE_F32 && kbar_dtype != HSA_DTYPE_BF16)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "unknown kbar_dtype %d", (int)kbar_dtype);
    if (dm.G > 16) return fail(HSA_ATTN_ERR_UNSUPPORTED, "decode supports at most 16 KV heads");
    if (dm.B == 0) return ok();
    const bool bf = p->dtype == HSA_DTYPE_BF16;
    s = check_ws(dm, bf, HSA_OP_DECODE_HOST, ws, ws_bytes);
    if (s != HSA_ATTN_OK) return s;
    CHECK_PTR(q, "q");
    CHECK_PTR(o, "o");
    CHECK_PTR(idx, "idx");
    CHECK_PTR(w, "w");
    const void* kd = nullptr;
    const void* vd = nullptr;
    if (dm.C > 0) {
        const size_t bytes = (size_t)dm.B * dm.L * dm.G * dm.d * (bf ? 2 : 4);
        s = host_cache(Kcache_host, bytes, "Kcache_host", &kd);
        if (s != HSA_ATTN_OK) return s;
        s = host_cache(Vcache_host, bytes, "Vcache_host", &vd);
        if (s != HSA_ATTN_OK) return s;
        CHECK_PTR(Kbar_cache, "Kbar_cache");
    }
    if (cache_len != nullptr && ((uintptr_t)cache_len & 3u))
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "cache_len is not 4-byte aligned");
    return launched(hsa::launch_decode_host(dm, bf, q, kd, vd, Kbar_cache,
                                            kbar_dtype == HSA_DTYPE_BF16, cache_len, o, idx, w,
                                            ws, (hipStream_t)stream),
                    "hsa_decode_host");
}

size_t hsa_attn_workspace_size(const hsa_attn_params_t* p, int op) {
    hsa::Dims dm;
    if (make_dims(p, &dm, op == HSA_OP_SELECT || op == HSA_OP_SELECT_BACKWARD) != HSA_ATTN_OK)
        return 0;
    return op_workspace(dm, p->dtype == HSA_DTYPE_BF16, op);
}

const char* hsa_attn_status_string(hsa_attn_status_t s) {
    switch (s) {
        case HSA_ATTN_OK: return "success";
        case HSA_ATTN_ERR_INVALID_ARGUMENT: return "invalid argument";
        case HSA_ATTN_ERR_UNSUPPORTED: return "unsupported configuration";
        case HSA_ATTN_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
        case HSA_ATTN_ERR_HIP: return "HIP error";
    }
    return "unknown status";
}

const char* hsa_attn_last_error(void) { return g_err; }

}  // extern "C"

namespace hsa {
int path_override(int op) {
    return (op >= 0 && op < 8) ? g_path[op].load(std::memory_order_relaxed) : HSA_PATH_AUTO;
}
}  // namespace hsa

extern "C" hsa_attn_status_t hsa_attn_set_path(int op, int path) {
    auto valid_for = [](int o, int pth) {
        switch (pth) {
            case HSA_PATH_AUTO:
            case HSA_PATH_GENERIC: return true;
            case HSA_PATH_TWO_PASS:
            case HSA_PATH_FUSED: return o == HSA_OP_BACKWARD;
            case HSA_PATH_CHUNK_MAJOR:
            case HSA_PATH_TILE_MAJOR: return o == HSA_OP_FORWARD;
            default: return false;
        }
    };
    const int ops[4] = {HSA_OP_SELECT, HSA_OP_FORWARD, HSA_OP_BACKWARD, HSA_OP_DECODE};
    if (op == -1) {
        if (path != HSA_PATH_AUTO && path != HSA_PATH_GENERIC)
            return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "path %d does not apply to every op", path);
        for (int o : ops) g_path[o].store(path, std::memory_order_relaxed);
        return ok();
    }
    if (op != HSA_OP_SELECT && op != HSA_OP_FORWARD && op != HSA_OP_BACKWARD &&
        op != HSA_OP_DECODE)
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "op %d has no kernel families", op);
    if (!valid_for(op, path))
        return fail(HSA_ATTN_ERR_INVALID_ARGUMENT, "path %d does not apply to op %d", path, op);
    g_path[op].store(path, std::memory_order_relaxed);
    return ok();
}

extern "C" int hsa_attn_get_path(int op) {
    if (op != HSA_OP_SELECT && op != HSA_OP_FORWARD && op != HSA_OP_BACKWARD &&
        op != HSA_OP_DECODE)
        return -1;
    return g_path[op].load(std::memory_order_relaxed);
}
