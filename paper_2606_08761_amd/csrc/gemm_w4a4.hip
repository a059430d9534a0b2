// Pure W4A4 group-quantized GEMM for gfx950 (CDNA4).
//
// APEX4 Sec. 3.2.1, Eq. (group_decomposition):
//   Y = sum_g (A_g^q W_g^q) (.) (S_g^a S_g^w^T)
// with immediate per-group dequantization for groups and delayed
// dequantization for per-channel scales (Sec. 4.2).
//
// CDNA4 mapping
//   * gfx950 has no 4-bit integer matrix instruction, so the packed nibbles are
//     widened to int8 MFMA operands.  The widening keeps each nibble in the high
//     half of its byte: (w << 4) & 0xF0F0F0F0 yields the even-k codes times 16
//     and w & 0xF0F0F0F0 the odd-k codes times 16 (two VALU ops per 8 codes plus
//     one).  A and W go through the same widening, so the MFMA sees the same
//     k permutation on both sides and every group sum comes out exactly
//     256 * P; the 1/256 is folded into the weight scale (a power of two,
//     exact).
//   * v_mfma_i32_32x32x32_i8 accumulates P in int32 per group (exact:
//     |256 P| <= 256 * 64 * G < 2^31 for G <= 2^16).
//   * The i32 -> f32 conversion and the s_a * s_w scaling run on the VALU once
//     per group; for G == K they run once, after the K loop.
//   * Operands are staged HBM -> registers -> (widen) -> LDS, double-buffered,
//     so each byte is widened once per workgroup, not once per wave.
//   * LDS rows are XOR-swizzled in 16-byte chunks so that the 32 rows read by
//     one MFMA operand fetch hit distinct banks.
//   * Workgroup ids are remapped so that each XCD (8 per MI355X, separate L2)
//     works on a contiguous band of output tiles.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "apex4_internal.h"

namespace apex4 {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128;          // output tile rows (M)
constexpr int BN = 128;          // output tile columns (N)
constexpr int KS = 128;          // K elements per pipeline stage
constexpr int ROWB = KS;         // bytes of one widened int8 row in LDS
constexpr int NTHREADS = 256;    // 4 waves, 2 x 2, each owns a 64 x 64 sub-tile

struct __align__(16) Stage {
    int8_t a[BM * ROWB];
    int8_t w[BN * ROWB];
    float sa[BM];
    float sw[BN];
};

// Byte offset of 16-byte chunk `chunk` (0..7) of widened row `row`.
__device__ __forceinline__ int swz(int row, int chunk) {
    return row * ROWB + ((chunk ^ (row & 7)) << 4);
}

__device__ __forceinline__ uint4 widen_even(uint4 v) {
    return make_uint4((v.x << 4) & 0xF0F0F0F0u, (v.y << 4) & 0xF0F0F0F0u, (v.z << 4) & 0xF0F0F0F0u,
                      (v.w << 4) & 0xF0F0F0F0u);
}
__device__ __forceinline__ uint4 widen_odd(uint4 v) {
    return make_uint4(v.x & 0xF0F0F0F0u, v.y & 0xF0F0F0F0u, v.z & 0xF0F0F0F0u, v.w & 0xF0F0F0F0u);
}

__device__ __forceinline__ float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }

template <bool DUMP>
__global__ __launch_bounds__(NTHREADS, 2) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ Aq, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ Wq,
    const uint16_t* __restrict__ sw, int M, int N, int K, int G, uint16_t* __restrict__ Y,
    int32_t* __restrict__ P) {
    __shared__ Stage st[2];

    // ---- tile selection (XCD-aware) ----
    const int mt_count = (M + BM - 1) / BM;
    const int nt_count = (N + BN - 1) / BN;
    const int T = mt_count * nt_count;
    int tile = blockIdx.x;
    if ((T & 7) == 0) tile = (blockIdx.x & 7) * (T >> 3) + (blockIdx.x >> 3);
    const int m0 = (tile % mt_count) * BM;
    const int n0 = (tile / mt_count) * BN;

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, lh = lane >> 5;

    const int64_t rowbytes = K / 2;
    const int nks = K / KS;
    const int spg = G / KS;          // pipeline stages per group
    const int ng = K / G;

    // ---- global -> register prefetch of one stage ----
    uint4 ra[2], rw[2];
    uint16_t rs = 0;
    auto load_stage = [&](int ks) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int c = tid + i * NTHREADS;
            const int r = c >> 2, p = c & 3;
            const int gm = m0 + r, gn = n0 + r;
            const int64_t koff = static_cast<int64_t>(ks) * (KS / 2) + p * 16;
            ra[i] = gm < M ? *reinterpret_cast<const uint4*>(Aq + gm * rowbytes + koff) : make_uint4(0, 0, 0, 0);
            rw[i] = gn < N ? *reinterpret_cast<const uint4*>(Wq + gn * rowbytes + koff) : make_uint4(0, 0, 0, 0);
        }
        if (!DUMP && (ks + 1) % spg == 0) {
            const int g = ks / spg;
            if (tid < BM) {
                const int gm = m0 + tid;
                rs = gm < M ? sa[static_cast<int64_t>(gm) * ng + g] : 0;
            } else {
                const int gn = n0 + tid - BM;
                rs = gn < N ? sw[static_cast<int64_t>(gn) * ng + g] : 0;
            }
        }
    };
    auto store_stage = [&](int ks, int buf) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int c = tid + i * NTHREADS;
            const int r = c >> 2, p = c & 3;
            *reinterpret_cast<uint4*>(&st[buf].a[swz(r, 2 * p)]) = widen_even(ra[i]);
            *reinterpret_cast<uint4*>(&st[buf].a[swz(r, 2 * p + 1)]) = widen_odd(ra[i]);
            *reinterpret_cast<uint4*>(&st[buf].w[swz(r, 2 * p)]) = widen_even(rw[i]);
            *reinterpret_cast<uint4*>(&st[buf].w[swz(r, 2 * p + 1)]) = widen_odd(rw[i]);
        }
        if (!DUMP && (ks + 1) % spg == 0) {
            if (tid < BM) st[buf].sa[tid] = h2f(rs);
            else st[buf].sw[tid - BM] = h2f(rs) * (1.0f / 256.0f);   // undo the x16 * x16 widening
        }
    };

    i32x16 acc_i[2][2];
    f32x16 acc_f[2][2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int r = 0; r < 16; ++r) { acc_f[rb][cb][r] = 0.f; acc_i[rb][cb][r] = 0; }

    auto compute = [&](int buf, auto first_tag) {
        constexpr bool FIRST = decltype(first_tag)::value;
#pragma unroll
        for (int kk = 0; kk < KS / 32; ++kk) {
            i32x4 a[2], b[2];
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
                a[rb] = *reinterpret_cast<const i32x4*>(&st[buf].a[swz(wm * 64 + rb * 32 + l32, 2 * kk + lh)]);
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
                b[cb] = *reinterpret_cast<const i32x4*>(&st[buf].w[swz(wn * 64 + cb * 32 + l32, 2 * kk + lh)]);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    if (FIRST && kk == 0) {
                        const i32x16 zero = {};
                        acc_i[rb][cb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[rb], b[cb], zero, 0, 0, 0);
                    } else {
                        acc_i[rb][cb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[rb], b[cb], acc_i[rb][cb], 0, 0, 0);
                    }
                }
        }
    };

    // Output row (within the 32 x 32 MFMA block) of accumulator element r of this lane.
    auto out_row = [&](int r) { return 8 * (r >> 2) + 4 * lh + (r & 3); };

    auto dequant = [&](int buf) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const float swv = st[buf].sw[wn * 64 + cb * 32 + l32];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float sav = st[buf].sa[wm * 64 + rb * 32 + out_row(r)];
                    acc_f[rb][cb][r] = fmaf(static_cast<float>(acc_i[rb][cb][r]) * swv, sav, acc_f[rb][cb][r]);
                }
            }
    };

    auto dump = [&](int g) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const int gn = n0 + wn * 64 + cb * 32 + l32;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gm = m0 + wm * 64 + rb * 32 + out_row(r);
                    if (gm < M && gn < N)
                        P[(static_cast<int64_t>(gm) * N + gn) * ng + g] = acc_i[rb][cb][r] >> 8;
                }
            }
    };

    // ---- main loop over K ----
    load_stage(0);
    store_stage(0, 0);
    __syncthreads();
    for (int ks = 0; ks < nks; ++ks) {
        const int buf = ks & 1;
        if (ks + 1 < nks) load_stage(ks + 1);
        if (ks % spg == 0) compute(buf, std::true_type{});
        else compute(buf, std::false_type{});
        if ((ks + 1) % spg == 0) {
            if constexpr (DUMP) dump(ks / spg);
            else dequant(buf);
        }
        if (ks + 1 < nks) store_stage(ks + 1, buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: binary32 -> binary16 (RNE) ----
    if constexpr (!DUMP) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const int gn = n0 + wn * 64 + cb * 32 + l32;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gm = m0 + wm * 64 + rb * 32 + out_row(r);
                    if (gm < M && gn < N)
                        Y[static_cast<int64_t>(gm) * N + gn] = __half_as_ushort(__float2half_rn(acc_f[rb][cb][r]));
                }
            }
    }
}

}  // namespace

hipError_t launch_gemm(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw,
                       int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, int32_t* P,
                       hipStream_t stream) {
    const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    if (tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(tiles)), block(NTHREADS);
    if (P) {
        hipLaunchKernelGGL(w4a4_gemm_kernel<true>, grid, block, 0, stream, Aq, sa, Wq, sw,
                           static_cast<int>(M), static_cast<int>(N), static_cast<int>(K), static_cast<int>(G),
                           Y, P);
    } else {
        hipLaunchKernelGGL(w4a4_gemm_kernel<false>, grid, block, 0, stream, Aq, sa, Wq, sw,
                           static_cast<int>(M), static_cast<int>(N), static_cast<int>(K), static_cast<int>(G),
                           Y, P);
    }
    return hipGetLastError();
}

}  // namespace apex4
