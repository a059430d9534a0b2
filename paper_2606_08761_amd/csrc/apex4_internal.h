// Internal launcher interface between the C ABI front end (api.hip) and the
// kernel translation units.  Arguments are already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace apex4 {

// Allows `bytes` of dynamic LDS for kernel k on the current device, once per
// device: `done` (one per kernel, static at the call site) holds a bit per
// device id below 64; a larger id sets the attribute on every call.
inline hipError_t allow_dynamic_lds(const void* k, int bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = (dev >= 0 && dev < 64) ? (uint64_t{1} << dev) : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
    return e;
}

// Debug dump of the exact integer group sums P[m, n, g] (Eq. group_decomposition)
// from the kernel that computes Y: rows [m0, m0 + mr) of the GEMM into
// P[mr][N][K/G] (int32).  P == nullptr: no dump.  Kernels that add partial sums
// of a group (K split over waves, 32-code dot products) add them with integer
// atomics into a zeroed P; the others store each group sum once.
struct Dump {
    int32_t* P = nullptr;
    int m0 = 0;
    int mr = 0;
};

// K stages of 128 codes covering K (the last one partial when K % 128 != 0).
__host__ __device__ inline int64_t kstages(int64_t K) { return (K + 127) / 128; }

// Tiled weight layout (wt): [ceil(N/32)][kstages(K)][2][64][16 B], zero padded.
// Piece (t, s, j, l) holds bytes [64 s + 32 (l / 32) + 16 j, + 16) of the packed
// row 32 t + l % 32: the 32 bytes lane l of a 32-column MFMA fragment consumes
// in stage s are contiguous, and a wave's fragment is one 2 KB block.
inline int64_t tiled_weight_bytes(int64_t N, int64_t K) { return ((N + 31) / 32) * kstages(K) * 2048; }
hipError_t launch_tile_weights(const uint8_t* Wq, int64_t N, int64_t K, uint8_t* Wt, hipStream_t stream);

// Activation/weight quantizer (SymQuant, b = 4).
hipError_t launch_quantize(const uint16_t* x, int64_t M, int64_t K, int64_t G,
                           uint8_t* q, uint16_t* s, hipStream_t stream);

// Kernel choice of the W4A4 GEMM entry points (values of the public
// APEX4_KERNEL_* constants).
enum GemmKernel : int {
    kKernelGemv = 1,      // one row, v_dot8 on the packed codes
    kKernelFused = 2,     // one row, quantize in the prologue (linear only)
    kKernelDecode = 3,    // up to 32 rows, weights streamed once
    kKernelTile64 = 4,    // 64 x 128 tiles, 4 waves (K may split inside the workgroup)
    kKernelTile128 = 5,   // 128 x 256 tiles, 8 waves
    kKernelPingPong = 6,  // G = 128 on 128 x 256 tiles, ping-pong schedule
    kKernelDecodeSplit = 7,  // the few-row kernel in stream-K form (workspace path)
};
struct GemmPlan {
    GemmKernel kernel;
    int splits;  // S > 1: split over K across workgroups (workspace path; tile kernels)
};
// split: the workspace path may split K; force_tile: no one-row, few-row or
// ping-pong kernel (tests compare the general tile kernel against them).
GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int64_t G, bool split, bool force_tile, bool wt = false);

// W4A4 GEMM: the one-row, few-row or tile kernel by shape (force_tile: always
// the tile kernel, for tests).  With a dump, the same kernel also writes the
// window's group sums; sa == sw == nullptr then skips the scales and Y.
hipError_t launch_gemm(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                       const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G,
                       uint16_t* Y, hipStream_t stream, Dump dump = Dump(), bool force_tile = false,
                       bool wt = false);

// int32 fill of n elements (dump buffers that receive atomic partial sums).
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t stream);

// GEMM split over K across workgroups for shapes whose tiles leave CUs idle:
// S partial planes part[S][M][N] (fp32, or int32 for G = K; caller workspace
// of splitk_workspace_bytes bytes), summed in split order and rounded once.
// splitk_factor() == 1 (workspace 0) where no split applies; launch_gemm_splitk
// then runs launch_gemm.  force_tile: G = 128 on the general tile kernel.
int splitk_factor(int64_t M, int64_t N, int64_t K, int64_t G);
int64_t splitk_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_gemm_splitk(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw,
                              int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, float* part,
                              hipStream_t stream, Dump dump = Dump(), bool force_tile = false, bool wt = false);

// Y = binary16(sum of the S fp32 planes part[S][M N]) in plane order.
hipError_t launch_splitk_reduce(const float* part, int S, int64_t MN, uint16_t* Y, hipStream_t stream);

// Compute units of the current device (cached after the first call).
int device_cu_count();

// W4A4 GEMM for few rows: weights streamed once, K split over the waves of a
// workgroup.  decode_fits() says whether the shape is one it handles.
bool decode_fits(int64_t M, int64_t N, int64_t K, int64_t G);
// workspace (decode_split_workspace_bytes(M, N, K, G) bytes, or nullptr): when
// the round-robin tiles leave CUs idle, the stream-K form of the kernel evens
// the (tile, stage) units out over the CUs and adds the parts of cut tiles
// through the workspace in a fixed order (decode_split_workspace_bytes is 0
// where it does not apply).
int64_t decode_split_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_gemm_decode(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                              const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G,
                              uint16_t* Y, hipStream_t stream, Dump dump = Dump(), bool wt = false,
                              void* workspace = nullptr);

// W4A4 GEMM for one row on the vector ALUs (v_dot8_i32_i4 on the packed
// codes): weight rows streamed from HBM in 1 KB runs; two rows too on tiled
// weights (wt).  gemv_fits() says whether the shape is one it handles.
bool gemv_fits(int64_t M, int64_t N, int64_t K, int64_t G, bool wt = false);
hipError_t launch_gemv(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                       int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream, Dump dump = Dump(),
                       bool wt = false);

// Quantize + W4A4 GEMM in one kernel: the one-row kernel above, quantizing x
// in its prologue (G in {32, 64, 128, 256, 512}, G < K).  Y as
// launch_quantize followed by launch_gemm gives, bit for bit, and Aq / sa
// receive the same codes and scales as launch_quantize writes.
bool fused_linear_fits(int64_t M, int64_t N, int64_t K, int64_t G, bool wt = false);
hipError_t launch_linear_fused(const uint16_t* x, const uint8_t* Wq, const uint16_t* sw, int64_t M, int64_t N,
                               int64_t K, int64_t G, uint16_t* Y, uint8_t* Aq, uint16_t* sa, hipStream_t stream,
                               Dump dump = Dump(), bool wt = false);

// The 4-bit codes in FP6 e3m2 containers (6-bit fields, little-endian, 3K/4
// bytes per row) and the G = 128 GEMM on the FP6 matrix cores that reads them.
hipError_t launch_pack_fp6(const uint8_t* q4, int64_t rows, int64_t K, uint8_t* q6, hipStream_t stream);
hipError_t launch_gemm_fp6(const uint8_t* A6, const uint16_t* sa, const uint8_t* W6, const uint16_t* sw, int64_t M,
                           int64_t N, int64_t K, uint16_t* Y, hipStream_t stream);

// MX variant: SymQuant codes with power-of-two (E8M0) group scales, written as
// FP6 e3m2 codes [rows, 3K/4] and scale bytes [rows, K/G]; and the GEMM that
// applies the scales inside the block-scaled FP6 MFMA (G in 32..1024).
hipError_t launch_quant_mx(const uint16_t* x, int64_t M, int64_t K, int64_t G, uint8_t* q6, uint8_t* e,
                           hipStream_t stream);
hipError_t launch_gemm_mx(const uint8_t* A6, const uint8_t* ea, const uint8_t* W6, const uint8_t* ew, int64_t M,
                          int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream);
// The MX GEMM split over K across workgroups when its tiles leave CUs idle:
// fp32 partial planes in a caller workspace of mx_splitk_workspace_bytes
// (0: no split; launch_gemm_mx_splitk then runs launch_gemm_mx).
int64_t mx_splitk_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_gemm_mx_splitk(const uint8_t* A6, const uint8_t* ea, const uint8_t* W6, const uint8_t* ew,
                                 int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, float* part,
                                 hipStream_t stream);

}  // namespace apex4
