// Offline tiled weight layout for gfx950: the counterpart of the paper's
// offline weight packing (Sec. 4.4 packs the 4-bit weights once, offline, into
// the vectors its kernel loads directly).
//
// The GEMM kernels read W as 32-column MFMA fragments: in a 128-wide K stage,
// lane l takes the 32 packed bytes [64 s + 32 (l / 32), + 32) of row
// 32 t + l % 32.  Row-major storage puts those 32 rows 4 KB-ish apart, so one
// load instruction gathers 64 bytes from each of 32 rows.  The tiled layout
// stores them in the order the lanes take them:
//     W_t[t][s][j][l][16 B] = W_q[32 t + l % 32][64 s + 32 (l / 32) + 16 j .. + 16]
// (zero past N and past K/2), so a wave's fragment of a stage is one
// contiguous 2 KB block and each 16-byte load instruction reads 1 KB.
// The transform runs once per weight matrix; HBM-bound, one 16-byte piece per
// thread (reads gathered, writes coalesced).
#include <hip/hip_runtime.h>

#include "apex4_internal.h"

namespace apex4 {
namespace {

__global__ __launch_bounds__(256) void tile_weights_kernel(const uint8_t* __restrict__ Wq, int64_t N, int64_t kb,
                                                           int64_t S, uint4* __restrict__ Wt, int64_t pieces) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t o = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; o < pieces; o += stride) {
        const int64_t l = o & 63, j = (o >> 6) & 1, ts = o >> 7;
        const int64_t t = ts / S, s = ts - t * S;
        const int64_t row = 32 * t + (l & 31);
        const int64_t byte = 64 * s + 32 * (l >> 5) + 16 * j;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (row < N && byte < kb) v = *reinterpret_cast<const uint4*>(Wq + row * kb + byte);
        Wt[o] = v;
    }
}

}  // namespace

hipError_t launch_tile_weights(const uint8_t* Wq, int64_t N, int64_t K, uint8_t* Wt, hipStream_t stream) {
    const int64_t pieces = tiled_weight_bytes(N, K) / 16;
    const int64_t need = (pieces + 255) / 256;
    const int blocks = static_cast<int>(need < 16384 ? need : 16384);
    hipLaunchKernelGGL(tile_weights_kernel, dim3(blocks), dim3(256), 0, stream, Wq, N, K / 2, kstages(K),
                       reinterpret_cast<uint4*>(Wt), pieces);
    return hipGetLastError();
}

}  // namespace apex4
