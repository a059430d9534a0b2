// Internal launcher interface between the C ABI front end (api.hip) and the
// kernel translation units.  Arguments are already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace apex4 {

// Activation/weight quantizer (SymQuant, b = 4).
hipError_t launch_quantize(const uint16_t* x, int64_t M, int64_t K, int64_t G,
                           uint8_t* q, uint16_t* s, hipStream_t stream);

// W4A4 GEMM.  When P is non-null the kernel dumps the exact integer group sums
// of rows [0, M) of the given operands instead of dequantizing (Y unused).
hipError_t launch_gemm(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                       const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G,
                       uint16_t* Y, int32_t* P, hipStream_t stream);

// G = 128 GEMM split over K across workgroups for shapes whose 128 x 256 tiles
// leave CUs idle: S fp32 partial planes part[S][M][N] (caller workspace of
// splitk_workspace_bytes bytes), summed in split order and rounded once.
// splitk_factor() == 1 (workspace 0) where no split applies; launch_gemm_splitk
// then runs launch_gemm.
int splitk_factor(int64_t M, int64_t N, int64_t K, int64_t G);
int64_t splitk_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_gemm_splitk(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw,
                              int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, float* part,
                              hipStream_t stream);

// Y = binary16(sum of the S fp32 planes part[S][M N]) in plane order.
hipError_t launch_splitk_reduce(const float* part, int S, int64_t MN, uint16_t* Y, hipStream_t stream);

// Compute units of the current device (cached after the first call).
int device_cu_count();

// W4A4 GEMM for few rows: weights streamed once, K split over the waves of a
// workgroup.  decode_fits() says whether the shape is one it handles.
bool decode_fits(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_gemm_decode(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                              const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G,
                              uint16_t* Y, hipStream_t stream);

// W4A4 GEMM for one row on the vector ALUs (v_dot8_i32_i4 on the packed
// codes): weight rows streamed from HBM in 1 KB runs.  gemv_fits() says
// whether the shape is one it handles.
bool gemv_fits(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_gemv(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                       int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream);

// Quantize + W4A4 GEMM in one kernel: the one-row kernel above, quantizing x
// in its prologue (G in {32, 64, 128, 256, 512}, G < K).  Y as
// launch_quantize followed by launch_gemm gives, bit for bit, and Aq / sa
// receive the same codes and scales as launch_quantize writes.
bool fused_linear_fits(int64_t M, int64_t N, int64_t K, int64_t G);
hipError_t launch_linear_fused(const uint16_t* x, const uint8_t* Wq, const uint16_t* sw, int64_t M, int64_t N,
                               int64_t K, int64_t G, uint16_t* Y, uint8_t* Aq, uint16_t* sa, hipStream_t stream);

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
