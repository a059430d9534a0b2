// C ABI front end: argument validation (before any HIP call), device check and
// dispatch to the kernel launchers.  See include/apex4.h for the contract.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>

#include "apex4.h"
#include "apex4_internal.h"

namespace {

constexpr int kMaxDevices = 64;
// 0 = unknown, 1 = gfx950, -1 = other architecture.
std::atomic<int> g_arch_ok[kMaxDevices];

constexpr int64_t kMaxChannelK = 65536;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return APEX4_ERR_DEVICE;
    if (dev < kMaxDevices) {
        const int known = g_arch_ok[dev].load(std::memory_order_relaxed);
        if (known == 1) return APEX4_OK;
        if (known == -1) return APEX4_ERR_DEVICE;
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return APEX4_ERR_DEVICE;
    const bool ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    if (dev < kMaxDevices) g_arch_ok[dev].store(ok ? 1 : -1, std::memory_order_relaxed);
    return ok ? APEX4_OK : APEX4_ERR_DEVICE;
}

// Shape rules shared by the GEMM entry points.
int check_gemm_shape(int64_t M, int64_t N, int64_t K) {
    if (M < 0 || N < 1 || K < 32 || (K % 32) != 0) return APEX4_ERR_SHAPE;
    if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    // the kernels address a packed operand row by row with 32-bit byte offsets
    if (M * (K / 2) > 0xFFFFFFFFll || N * (K / 2) > 0xFFFFFFFFll) return APEX4_ERR_SHAPE;
    return APEX4_OK;
}

int check_gemm_group(int64_t K, int64_t G) {
    if (G <= 0) return APEX4_ERR_GROUP;
    // one group per row: the kernels hold 256 P of the whole row in one int32,
    // exact while 2^14 K < 2^31 with room for the split sums
    if (G == K) return K <= kMaxChannelK ? APEX4_OK : APEX4_ERR_GROUP;
    if (G != 32 && G != 64 && G != 128 && G != 256 && G != 512 && G != 1024) return APEX4_ERR_GROUP;
    if (K % G != 0) return APEX4_ERR_SHAPE;
    return APEX4_OK;
}

// Buffers sized by M (or by a row window) may be NULL when that size is zero.
bool present(const void* p, int64_t rows) { return p != nullptr || rows == 0; }

int check_quant_args(const void* x, int64_t M, int64_t K, int64_t G, const void* A_q, const void* s_a) {
    if (!present(x, M) || !present(A_q, M) || !present(s_a, M)) return APEX4_ERR_NULL;
    if (M < 0 || K < 32 || (K % 32) != 0 || M > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    if (G <= 0 || (G % 32) != 0 || G > K) return APEX4_ERR_GROUP;
    if (K % G != 0) return APEX4_ERR_SHAPE;
    if (!aligned16(x) || !aligned16(A_q) || !aligned16(s_a)) return APEX4_ERR_ALIGN;
    return APEX4_OK;
}

int check_gemm_args(const void* A_q, const void* s_a, const void* W_q, const void* s_w, int64_t M,
                    int64_t N, int64_t K, int64_t G, const void* Y) {
    if (!present(A_q, M) || !present(s_a, M) || !W_q || !s_w || !present(Y, M)) return APEX4_ERR_NULL;
    int rc = check_gemm_shape(M, N, K);
    if (rc) return rc;
    rc = check_gemm_group(K, G);
    if (rc) return rc;
    if (!aligned16(A_q) || !aligned16(s_a) || !aligned16(W_q) || !aligned16(s_w) || !aligned16(Y))
        return APEX4_ERR_ALIGN;
    return APEX4_OK;
}

}  // namespace

extern "C" {

const char* apex4_status_string(int status) {
    switch (status) {
        case APEX4_OK: return "APEX4_OK";
        case APEX4_ERR_NULL: return "APEX4_ERR_NULL: a required pointer is NULL";
        case APEX4_ERR_SHAPE: return "APEX4_ERR_SHAPE: M, N, K or the row window is out of range";
        case APEX4_ERR_GROUP: return "APEX4_ERR_GROUP: unsupported group size";
        case APEX4_ERR_ALIGN: return "APEX4_ERR_ALIGN: a pointer is not 16-byte aligned";
        case APEX4_ERR_LAUNCH: return "APEX4_ERR_LAUNCH: kernel launch failed";
        case APEX4_ERR_DEVICE: return "APEX4_ERR_DEVICE: no gfx950 device is current";
        case APEX4_ERR_WORKSPACE:
            return "APEX4_ERR_WORKSPACE: workspace NULL or too small (apex4_w4a4_gemm_noalloc: the split needs more "
                   "than its static scratch)";
        default: return "APEX4: unknown status";
    }
}

int apex4_version(void) { return 200; }

int apex4_quantize_act(const void* x, int64_t M, int64_t K, int64_t G, uint8_t* A_q, void* s_a,
                       void* stream) {
    int rc = check_quant_args(x, M, K, G, A_q, s_a);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    hipError_t e = apex4::launch_quantize(static_cast<const uint16_t*>(x), M, K, G, A_q,
                                          static_cast<uint16_t*>(s_a), static_cast<hipStream_t>(stream));
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int apex4_w4a4_gemm(const uint8_t* A_q, const void* s_a, const uint8_t* W_q, const void* s_w, int64_t M,
                    int64_t N, int64_t K, int64_t G, void* Y, void* stream) {
    int rc = check_gemm_args(A_q, s_a, W_q, s_w, M, N, K, G, Y);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    hipError_t e = apex4::launch_gemm(A_q, static_cast<const uint16_t*>(s_a), W_q,
                                      static_cast<const uint16_t*>(s_w), M, N, K, G, static_cast<uint16_t*>(Y),
                                      static_cast<hipStream_t>(stream));
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int apex4_w4a4_gemm_workspace_size(int64_t M, int64_t N, int64_t K, int64_t G, int64_t* bytes) {
    if (!bytes) return APEX4_ERR_NULL;
    int rc = check_gemm_shape(M, N, K);
    if (rc) return rc;
    rc = check_gemm_group(K, G);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    *bytes = apex4::splitk_workspace_bytes(M, N, K, G);
    return APEX4_OK;
}

namespace {

// The dispatch of apex4_w4a4_gemm (workspace == NULL) or apex4_w4a4_gemm_ws,
// with an optional dump of exact group sums and the general-tile switch.
int gemm_dispatch(const uint8_t* A_q, const void* s_a, const uint8_t* W_q, const void* s_w, int64_t M, int64_t N,
                  int64_t K, int64_t G, void* Y, void* workspace, int64_t workspace_bytes, apex4::Dump dump,
                  bool general, bool wt, void* stream) {
    const auto sa = static_cast<const uint16_t*>(s_a);
    const auto sw = static_cast<const uint16_t*>(s_w);
    const auto y = static_cast<uint16_t*>(Y);
    const auto st = static_cast<hipStream_t>(stream);
    const int64_t need = workspace ? apex4::splitk_workspace_bytes(M, N, K, G) : 0;
    hipError_t e;
    if (need == 0) {
        e = apex4::launch_gemm(A_q, sa, W_q, sw, M, N, K, G, y, st, dump, general, wt);
    } else {
        if (workspace_bytes < need) return APEX4_ERR_WORKSPACE;
        e = apex4::launch_gemm_splitk(A_q, sa, W_q, sw, M, N, K, G, y, static_cast<float*>(workspace), st, dump,
                                      general, wt);
    }
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

// Tiled weights (apex4_tile_weights): one group per 128-wide stage or more, and
// 32-bit offsets into the tiled buffer.
int check_tiled(int64_t N, int64_t K, int64_t G) {
    if (G < 128) return APEX4_ERR_GROUP;
    if (apex4::tiled_weight_bytes(N, K) > 0xFFFFFFFFll) return APEX4_ERR_SHAPE;
    return APEX4_OK;
}

int check_window(int64_t M, int64_t m0, int64_t mr, const void* P) {
    if (!present(P, mr)) return APEX4_ERR_NULL;
    if (m0 < 0 || mr < 0 || m0 > M || mr > M - m0) return APEX4_ERR_SHAPE;
    if (!aligned16(P)) return APEX4_ERR_ALIGN;
    return APEX4_OK;
}

}  // namespace

int apex4_w4a4_gemm_ws(const uint8_t* A_q, const void* s_a, const uint8_t* W_q, const void* s_w, int64_t M,
                       int64_t N, int64_t K, int64_t G, void* Y, void* workspace, int64_t workspace_bytes,
                       void* stream) {
    int rc = check_gemm_args(A_q, s_a, W_q, s_w, M, N, K, G, Y);
    if (rc) return rc;
    if (workspace && !aligned16(workspace)) return APEX4_ERR_ALIGN;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    if (!workspace && apex4::splitk_workspace_bytes(M, N, K, G) > 0) return APEX4_ERR_WORKSPACE;
    return gemm_dispatch(A_q, s_a, W_q, s_w, M, N, K, G, Y, workspace, workspace_bytes, apex4::Dump(), false, false,
                         stream);
}

int apex4_w4a4_gemm_groupsums(const uint8_t* A_q, const uint8_t* W_q, int64_t M, int64_t N, int64_t K,
                              int64_t G, int64_t m0, int64_t mr, int32_t* P, void* stream) {
    if (!present(A_q, M) || !W_q || !present(P, mr)) return APEX4_ERR_NULL;
    int rc = check_gemm_shape(M, N, K);
    if (rc) return rc;
    rc = check_gemm_group(K, G);
    if (rc) return rc;
    rc = check_window(M, m0, mr, P);
    if (rc) return rc;
    if (!aligned16(A_q) || !aligned16(W_q)) return APEX4_ERR_ALIGN;
    rc = check_device();
    if (rc) return rc;
    if (mr == 0) return APEX4_OK;
    // the full M x N problem through apex4_w4a4_gemm's kernel choice, without
    // scales (no Y): only the window's sums are written
    const apex4::Dump dump{P, static_cast<int>(m0), static_cast<int>(mr)};
    return gemm_dispatch(A_q, nullptr, W_q, nullptr, M, N, K, G, nullptr, nullptr, 0, dump, false, false, stream);
}

}  // extern "C"

// Split-K partial planes (or stream-K counters and parts) of
// apex4_w4a4_gemm_noalloc.  Each device holds its own
// copy for the life of the process; host code reaches it only through the
// address hipGetSymbolAddress returns for the current device (the name itself
// is a host-side stand-in, not a device address).
static __device__ __align__(256) uint8_t scratch[APEX4_NOALLOC_SCRATCH_BYTES];

namespace {

void* g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// This device's `scratch`, looked up once per device with that device current.
int scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return APEX4_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return APEX4_ERR_LAUNCH;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return APEX4_OK;
}

}  // namespace

extern "C" {

int apex4_w4a4_gemm_noalloc(const uint8_t* A_q, const void* s_a, const uint8_t* W_q, const void* s_w, int64_t M,
                            int64_t N, int64_t K, int64_t G, void* Y, void* stream) {
    int rc = check_gemm_args(A_q, s_a, W_q, s_w, M, N, K, G, Y);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const int64_t need = apex4::splitk_workspace_bytes(M, N, K, G);
    if (need > APEX4_NOALLOC_SCRATCH_BYTES) return APEX4_ERR_WORKSPACE;
    void* ws = nullptr;
    if (need > 0) {
        rc = scratch_address(&ws);
        if (rc) return rc;
    }
    // every partial plane element is written before the reduce reads it, and
    // the stream-K counters are cleared by a fill kernel in the launch itself
    return gemm_dispatch(A_q, s_a, W_q, s_w, M, N, K, G, Y, ws, need, apex4::Dump(), false, false, stream);
}

int apex4_w4a4_gemm_debug(const uint8_t* A_q, const void* s_a, const uint8_t* W_q, const void* s_w, int64_t M,
                          int64_t N, int64_t K, int64_t G, void* Y, void* workspace, int64_t workspace_bytes,
                          int64_t m0, int64_t mr, int32_t* P, int flags, void* stream) {
    if (!present(P, mr)) return APEX4_ERR_NULL;
    int rc = check_gemm_args(A_q, s_a, W_q, s_w, M, N, K, G, Y);
    if (rc) return rc;
    if (workspace && !aligned16(workspace)) return APEX4_ERR_ALIGN;
    if (flags & ~(APEX4_DEBUG_GENERAL_TILES | APEX4_DEBUG_W_TILED)) return APEX4_ERR_SHAPE;
    const bool wt = (flags & APEX4_DEBUG_W_TILED) != 0;
    if (wt && (rc = check_tiled(N, K, G))) return rc;
    rc = check_window(M, m0, mr, P);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const apex4::Dump dump{mr > 0 ? P : nullptr, static_cast<int>(m0), static_cast<int>(mr)};
    return gemm_dispatch(A_q, s_a, W_q, s_w, M, N, K, G, Y, workspace, workspace_bytes, dump,
                         (flags & APEX4_DEBUG_GENERAL_TILES) != 0, wt, stream);
}

int apex4_tiled_weights_size(int64_t N, int64_t K, int64_t* bytes) {
    if (!bytes) return APEX4_ERR_NULL;
    if (N < 1 || K < 32 || (K % 32) != 0 || N > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    *bytes = apex4::tiled_weight_bytes(N, K);
    return APEX4_OK;
}

int apex4_tile_weights(const uint8_t* W_q, int64_t N, int64_t K, uint8_t* W_t, void* stream) {
    if (!W_q || !W_t) return APEX4_ERR_NULL;
    if (N < 1 || K < 32 || (K % 32) != 0 || N > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    if (N * (K / 2) > 0xFFFFFFFFll || apex4::tiled_weight_bytes(N, K) > 0xFFFFFFFFll) return APEX4_ERR_SHAPE;
    if (!aligned16(W_q) || !aligned16(W_t)) return APEX4_ERR_ALIGN;
    const int rc = check_device();
    if (rc) return rc;
    const hipError_t e = apex4::launch_tile_weights(W_q, N, K, W_t, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int apex4_w4a4_gemm_tiled(const uint8_t* A_q, const void* s_a, const uint8_t* W_t, const void* s_w, int64_t M,
                          int64_t N, int64_t K, int64_t G, void* Y, void* workspace, int64_t workspace_bytes,
                          void* stream) {
    int rc = check_gemm_args(A_q, s_a, W_t, s_w, M, N, K, G, Y);
    if (rc) return rc;
    if ((rc = check_tiled(N, K, G))) return rc;
    if (workspace && !aligned16(workspace)) return APEX4_ERR_ALIGN;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    return gemm_dispatch(A_q, s_a, W_t, s_w, M, N, K, G, Y, workspace, workspace_bytes, apex4::Dump(), false, true,
                         stream);
}

namespace {

int linear_dispatch(const void* x, const uint8_t* W_q, const void* s_w, int64_t M, int64_t N, int64_t K, int64_t G,
                    void* Y, uint8_t* A_q_work, void* s_a_work, apex4::Dump dump, bool wt, void* stream) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    const auto xh = static_cast<const uint16_t*>(x);
    const auto sw = static_cast<const uint16_t*>(s_w);
    const auto sa = static_cast<uint16_t*>(s_a_work);
    const auto y = static_cast<uint16_t*>(Y);
    if (apex4::fused_linear_fits(M, N, K, G, wt)) {
        const hipError_t e = apex4::launch_linear_fused(xh, W_q, sw, M, N, K, G, y, A_q_work, sa, st, dump, wt);
        return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
    }
    hipError_t e = apex4::launch_quantize(xh, M, K, G, A_q_work, sa, st);
    if (e != hipSuccess) return APEX4_ERR_LAUNCH;
    e = apex4::launch_gemm(A_q_work, sa, W_q, sw, M, N, K, G, y, st, dump, false, wt);
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int check_linear_args(const void* x, const uint8_t* W_q, const void* s_w, int64_t M, int64_t N, int64_t K, int64_t G,
                      const void* Y, const uint8_t* A_q_work, const void* s_a_work) {
    if (!present(x, M) || !W_q || !s_w || !present(Y, M) || !present(A_q_work, M) || !present(s_a_work, M))
        return APEX4_ERR_NULL;
    const int rc = check_gemm_args(A_q_work, s_a_work, W_q, s_w, M, N, K, G, Y);
    if (rc) return rc;
    return check_quant_args(x, M, K, G, A_q_work, s_a_work);
}

}  // namespace

int apex4_w4a4_linear(const void* x, const uint8_t* W_q, const void* s_w, int64_t M, int64_t N, int64_t K,
                      int64_t G, void* Y, uint8_t* A_q_work, void* s_a_work, void* stream) {
    int rc = check_linear_args(x, W_q, s_w, M, N, K, G, Y, A_q_work, s_a_work);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    return linear_dispatch(x, W_q, s_w, M, N, K, G, Y, A_q_work, s_a_work, apex4::Dump(), false, stream);
}

int apex4_w4a4_linear_tiled(const void* x, const uint8_t* W_t, const void* s_w, int64_t M, int64_t N, int64_t K,
                            int64_t G, void* Y, uint8_t* A_q_work, void* s_a_work, void* stream) {
    int rc = check_linear_args(x, W_t, s_w, M, N, K, G, Y, A_q_work, s_a_work);
    if (rc) return rc;
    if ((rc = check_tiled(N, K, G))) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    return linear_dispatch(x, W_t, s_w, M, N, K, G, Y, A_q_work, s_a_work, apex4::Dump(), true, stream);
}

int apex4_w4a4_linear_ws(const void* x, const uint8_t* W, const void* s_w, int64_t M, int64_t N, int64_t K,
                         int64_t G, void* Y, uint8_t* A_q_work, void* s_a_work, void* workspace,
                         int64_t workspace_bytes, int flags, void* stream) {
    int rc = check_linear_args(x, W, s_w, M, N, K, G, Y, A_q_work, s_a_work);
    if (rc) return rc;
    if (flags & ~APEX4_DEBUG_W_TILED) return APEX4_ERR_SHAPE;
    const bool wt = flags != 0;
    if (wt && (rc = check_tiled(N, K, G))) return rc;
    if (workspace && !aligned16(workspace)) return APEX4_ERR_ALIGN;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    // the workspace is checked before the quantizer runs, so that a refused
    // call writes nothing (the fused one-row kernel takes none)
    if (!apex4::fused_linear_fits(M, N, K, G, wt)) {
        const int64_t need = apex4::splitk_workspace_bytes(M, N, K, G);
        if (need > 0 && (!workspace || workspace_bytes < need)) return APEX4_ERR_WORKSPACE;
        hipStream_t st = static_cast<hipStream_t>(stream);
        const hipError_t e = apex4::launch_quantize(static_cast<const uint16_t*>(x), M, K, G, A_q_work,
                                                    static_cast<uint16_t*>(s_a_work), st);
        if (e != hipSuccess) return APEX4_ERR_LAUNCH;
        return gemm_dispatch(A_q_work, s_a_work, W, s_w, M, N, K, G, Y, need > 0 ? workspace : nullptr,
                             workspace_bytes, apex4::Dump(), false, wt, stream);
    }
    return linear_dispatch(x, W, s_w, M, N, K, G, Y, A_q_work, s_a_work, apex4::Dump(), wt, stream);
}

int apex4_w4a4_linear_debug(const void* x, const uint8_t* W_q, const void* s_w, int64_t M, int64_t N, int64_t K,
                            int64_t G, void* Y, uint8_t* A_q_work, void* s_a_work, int64_t m0, int64_t mr, int32_t* P,
                            int flags, void* stream) {
    if (!present(P, mr)) return APEX4_ERR_NULL;
    int rc = check_linear_args(x, W_q, s_w, M, N, K, G, Y, A_q_work, s_a_work);
    if (rc) return rc;
    if (flags & ~APEX4_DEBUG_W_TILED) return APEX4_ERR_SHAPE;
    const bool wt = flags != 0;
    if (wt && (rc = check_tiled(N, K, G))) return rc;
    rc = check_window(M, m0, mr, P);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const apex4::Dump dump{mr > 0 ? P : nullptr, static_cast<int>(m0), static_cast<int>(mr)};
    return linear_dispatch(x, W_q, s_w, M, N, K, G, Y, A_q_work, s_a_work, dump, wt, stream);
}

int apex4_w4a4_gemm_plan(int entry, int64_t M, int64_t N, int64_t K, int64_t G, int flags, int* kernel,
                         int* splits) {
    if (!kernel || !splits) return APEX4_ERR_NULL;
    int rc = check_gemm_shape(M, N, K);
    if (rc) return rc;
    rc = check_gemm_group(K, G);
    if (rc) return rc;
    if (entry < APEX4_ENTRY_GEMM || entry > APEX4_ENTRY_LINEAR_WS) return APEX4_ERR_SHAPE;
    if (flags & ~(APEX4_DEBUG_GENERAL_TILES | APEX4_DEBUG_W_TILED)) return APEX4_ERR_SHAPE;
    const bool linear = entry == APEX4_ENTRY_LINEAR || entry == APEX4_ENTRY_LINEAR_WS;
    if (linear && (flags & APEX4_DEBUG_GENERAL_TILES)) return APEX4_ERR_SHAPE;
    const bool wt = (flags & APEX4_DEBUG_W_TILED) != 0;
    if (wt && (rc = check_tiled(N, K, G))) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) {
        *kernel = 0;
        *splits = 0;
        return APEX4_OK;
    }
    if (linear && apex4::fused_linear_fits(M, N, K, G, wt)) {
        *kernel = apex4::kKernelFused;
        *splits = 1;
        return APEX4_OK;
    }
    const apex4::GemmPlan plan =
        apex4::plan_gemm(M, N, K, G, entry == APEX4_ENTRY_GEMM_WS || entry == APEX4_ENTRY_LINEAR_WS,
                         (flags & APEX4_DEBUG_GENERAL_TILES) != 0, wt);
    *kernel = plan.kernel;
    *splits = plan.splits;
    return APEX4_OK;
}

int apex4_pack_fp6(const uint8_t* q4, int64_t rows, int64_t K, uint8_t* q6, void* stream) {
    if (!present(q4, rows) || !present(q6, rows)) return APEX4_ERR_NULL;
    if (rows < 0 || K < 128 || (K % 128) != 0 || rows > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    if (!aligned16(q4) || !aligned16(q6)) return APEX4_ERR_ALIGN;
    const int rc = check_device();
    if (rc) return rc;
    if (rows == 0) return APEX4_OK;
    const hipError_t e = apex4::launch_pack_fp6(q4, rows, K, q6, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int apex4_w4a4_gemm_fp6(const uint8_t* A_6, const void* s_a, const uint8_t* W_6, const void* s_w, int64_t M,
                        int64_t N, int64_t K, int64_t G, void* Y, void* stream) {
    if (!present(A_6, M) || !present(s_a, M) || !W_6 || !s_w || !present(Y, M)) return APEX4_ERR_NULL;
    if (M < 0 || N < 1 || K < 128 || (K % 128) != 0) return APEX4_ERR_SHAPE;
    if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    // 32-bit byte offsets into each FP6 operand
    if (M * (3 * K / 4) > 0xFFFFFFFFll || N * (3 * K / 4) > 0xFFFFFFFFll) return APEX4_ERR_SHAPE;
    if (G != 128) return APEX4_ERR_GROUP;
    if (!aligned16(A_6) || !aligned16(s_a) || !aligned16(W_6) || !aligned16(s_w) || !aligned16(Y))
        return APEX4_ERR_ALIGN;
    const int rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const hipError_t e = apex4::launch_gemm_fp6(A_6, static_cast<const uint16_t*>(s_a), W_6,
                                                static_cast<const uint16_t*>(s_w), M, N, K,
                                                static_cast<uint16_t*>(Y), static_cast<hipStream_t>(stream));
    return e == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

namespace {
bool mx_group(int64_t G) { return G == 32 || G == 64 || G == 128 || G == 256 || G == 512 || G == 1024; }
}  // namespace

int apex4_quantize_mx(const void* x, int64_t M, int64_t K, int64_t G, uint8_t* Q6, uint8_t* e, void* stream) {
    if (!present(x, M) || !present(Q6, M) || !present(e, M)) return APEX4_ERR_NULL;
    if (M < 0 || K < 128 || (K % 128) != 0 || M > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    if (!mx_group(G) || G > K) return APEX4_ERR_GROUP;
    if (K % G != 0) return APEX4_ERR_SHAPE;
    if (!aligned16(x) || !aligned16(Q6) || !aligned16(e)) return APEX4_ERR_ALIGN;
    const int rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const hipError_t err = apex4::launch_quant_mx(static_cast<const uint16_t*>(x), M, K, G, Q6, e,
                                                  static_cast<hipStream_t>(stream));
    return err == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int check_mx_gemm_args(const void* A_6, const void* e_a, const void* W_6, const void* e_w, int64_t M, int64_t N,
                       int64_t K, int64_t G, const void* Y) {
    if (!present(A_6, M) || !present(e_a, M) || !W_6 || !e_w || !present(Y, M)) return APEX4_ERR_NULL;
    if (M < 0 || N < 1 || K < 128 || (K % 128) != 0) return APEX4_ERR_SHAPE;
    if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || K > 0x7FFFFFFF) return APEX4_ERR_SHAPE;
    if (M * (3 * K / 4) > 0xFFFFFFFFll || N * (3 * K / 4) > 0xFFFFFFFFll) return APEX4_ERR_SHAPE;
    if (!mx_group(G) || G > K) return APEX4_ERR_GROUP;
    if (K % G != 0) return APEX4_ERR_SHAPE;
    if (!aligned16(A_6) || !aligned16(e_a) || !aligned16(W_6) || !aligned16(e_w) || !aligned16(Y))
        return APEX4_ERR_ALIGN;
    return APEX4_OK;
}

int apex4_w4a4_gemm_mx(const uint8_t* A_6, const uint8_t* e_a, const uint8_t* W_6, const uint8_t* e_w, int64_t M,
                       int64_t N, int64_t K, int64_t G, void* Y, void* stream) {
    int rc = check_mx_gemm_args(A_6, e_a, W_6, e_w, M, N, K, G, Y);
    if (rc) return rc;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const hipError_t err = apex4::launch_gemm_mx(A_6, e_a, W_6, e_w, M, N, K, G, static_cast<uint16_t*>(Y),
                                                 static_cast<hipStream_t>(stream));
    return err == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

int apex4_w4a4_gemm_mx_workspace_size(int64_t M, int64_t N, int64_t K, int64_t G, int64_t* bytes) {
    if (!bytes) return APEX4_ERR_NULL;
    if (M < 0 || N < 1 || K < 128 || (K % 128) != 0 || M > 0x7FFFFFFF || N > 0x7FFFFFFF || K > 0x7FFFFFFF)
        return APEX4_ERR_SHAPE;
    if (!mx_group(G) || G > K) return APEX4_ERR_GROUP;
    if (K % G != 0) return APEX4_ERR_SHAPE;
    const int rc = check_device();
    if (rc) return rc;
    *bytes = apex4::mx_splitk_workspace_bytes(M, N, K, G);
    return APEX4_OK;
}

int apex4_w4a4_gemm_mx_ws(const uint8_t* A_6, const uint8_t* e_a, const uint8_t* W_6, const uint8_t* e_w, int64_t M,
                          int64_t N, int64_t K, int64_t G, void* Y, void* workspace, int64_t workspace_bytes,
                          void* stream) {
    int rc = check_mx_gemm_args(A_6, e_a, W_6, e_w, M, N, K, G, Y);
    if (rc) return rc;
    if (workspace && !aligned16(workspace)) return APEX4_ERR_ALIGN;
    rc = check_device();
    if (rc) return rc;
    if (M == 0) return APEX4_OK;
    const int64_t need = apex4::mx_splitk_workspace_bytes(M, N, K, G);
    if (need > 0 && (!workspace || workspace_bytes < need)) return APEX4_ERR_WORKSPACE;
    const hipError_t err =
        need == 0 ? apex4::launch_gemm_mx(A_6, e_a, W_6, e_w, M, N, K, G, static_cast<uint16_t*>(Y),
                                          static_cast<hipStream_t>(stream))
                  : apex4::launch_gemm_mx_splitk(A_6, e_a, W_6, e_w, M, N, K, G, static_cast<uint16_t*>(Y),
                                                 static_cast<float*>(workspace), static_cast<hipStream_t>(stream));
    return err == hipSuccess ? APEX4_OK : APEX4_ERR_LAUNCH;
}

}  // extern "C"
