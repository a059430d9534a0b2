// W4A4 group GEMM on the FP6 matrix cores of gfx950 (CDNA4 numerics variant).
//
// The same computation as the INT8 path (APEX4 Sec. 3.2.1, Eq.
// group_decomposition), with the 4-bit codes held in FP6 e3m2 containers:
//   * Every code q in [-8, 7] is exact in e3m2 (1 sign, 3 exponent, 2 mantissa
//     bits, bias 3), products are exact (|q_a q_w| <= 64) and the fp32
//     accumulation of a group is exact (every partial sum is an integer below
//     2^24), so the group sums are the same integers as on the INT8 path.
//   * v_mfma_scale_f32_32x32x64_f8f6f4 with both operands FP6 (format 3) and
//     unit E8M0 block scales runs at twice the INT8 MFMA rate and takes the
//     packed 6-bit codes as stored: no nibble widening.  Each group starts from
//     a zero accumulator, so D is the group sum P as an exact float, and the
//     dequantization t = fl(P s_a), acc = fma_mix(t, s_w, acc) takes the same
//     two roundings as the INT8 path: Y is the same bits.
//   * FP6 row layout (apex4_pack_fp6): code k of a row at bits [6k, 6k + 6) of
//     the row's 3K/4 bytes, little-endian.  A 128-wide stage is 96 bytes of a
//     row; lane half h holds its bytes [48h, 48h + 48): codes [64h, 64h + 64),
//     the first 32 for MFMA kk = 0 and the rest for kk = 1.  Both operands use
//     this order, so every MFMA pairs matching k, and each lane reads its 48
//     bytes with three 16-byte LDS reads.
//   * Schedule: the ping-pong of the INT8 G = 128 kernel (gemm_w4a4.hip), 128 x
//     256 tiles, 8 waves of 128 x 32; per wave and stage 8 MFMAs instead of 16.
//   * Measured on MI355X (M = 2048, N = K = 8192) this kernel takes about 1.1x
//     the time of the INT8 one.  Halving the MFMA time moves the bound to the
//     LDS: per stage each wave reads 15 KB of operands (the whole 128-row
//     activation tile and its 32 weight rows), 60 KB for the four waves of a
//     phase, about 470 cycles at 128 bytes per clock against 256 cycles of
//     MFMA work; the dequantization VALU work is unchanged.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "apex4_internal.h"

namespace apex4 {
namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KS6 = 128;                      // K per stage
constexpr int SROW6 = KS6 * 6 / 8;            // 96 bytes of one row per stage
constexpr int AROW6 = SROW6 + 16;             // padded LDS row: 28 dwords, 16 rows x 16 bytes hit distinct banks
constexpr int FMT_E3M2 = 3;                   // f8f6f4 operand format: FP6 e3m2
constexpr int SCALE_ONE = 127;                // E8M0 2^0

__device__ __forceinline__ float h2f6(uint16_t b) { return __half2float(__ushort_as_half(b)); }

template <int B, int E, typename F>
__device__ __forceinline__ void static_for6(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for6<B + 1, E>(f);
    }
}

// e3m2 code of the two's-complement nibble v: magnitudes 0..8 are
// 0, 12, 16, 18, 20, 21, 22, 23, 24; negative values set bit 5.
__device__ __forceinline__ uint32_t e3m2_of_nibble(uint32_t v) {
    // bytes 0..7: codes of nibbles 0..7 (q = 0..7); bytes 8..15: nibbles 8..15 (q = -8..-1)
    constexpr uint64_t LO = 0x17161514'12100C00ull;
    constexpr uint64_t HI = 0x2C303234'35363738ull;
    const uint64_t tab = (v & 8) ? HI : LO;
    return static_cast<uint32_t>(tab >> (8 * (v & 7))) & 0x3Fu;
}

// 16 codes (8 bytes of packed nibbles) per thread -> 12 bytes of e3m2 codes.
__global__ __launch_bounds__(256) void pack_fp6_kernel(const uint8_t* __restrict__ q4, int64_t units, int64_t upr,
                                                       int64_t K, uint8_t* __restrict__ q6) {
    for (int64_t u = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; u < units;
         u += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t row = u / upr, j = u - row * upr;
        const uint2 v = *reinterpret_cast<const uint2*>(q4 + row * (K / 2) + 8 * j);
        uint32_t out[3] = {0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const uint32_t nib = ((i < 8 ? v.x : v.y) >> (4 * (i & 7))) & 0xFu;
            const uint32_t c = e3m2_of_nibble(nib);
            const int bit = 6 * i;
            out[bit >> 5] |= c << (bit & 31);
            if ((bit & 31) > 26) out[(bit >> 5) + 1] |= c >> (32 - (bit & 31));
        }
        uint32_t* dst = reinterpret_cast<uint32_t*>(q6 + row * (3 * K / 4) + 12 * j);
        dst[0] = out[0];
        dst[1] = out[1];
        dst[2] = out[2];
    }
}

struct Stage6 {
    uint8_t a[128 * AROW6];  // 128 activation rows x 96 bytes
    uint8_t w[256 * AROW6];  // 256 weight rows x 96 bytes
    uint16_t scale[512];     // [0, 128) s_a rows, [128, 384) s_w columns, rest unused
};
static_assert(sizeof(Stage6) == 44032, "Stage6 layout");

// G = 128, 128 x 256 tiles, ping-pong between the wave groups X (0-3) and Y
// (4-7) as in w4a4_gemm_pp_kernel; see there for the slot schedule and why the
// LDS buffers are never written while read.  Unlike there, the weights also go
// through LDS: read straight into the MFMA layout, each lane would fetch three
// 16-byte pieces of 32 rows 3K/4 bytes apart, which measured 1.5x slower for
// the whole kernel; staged, six lanes read one row's 96 contiguous bytes.
__global__ __launch_bounds__(512, 1) void w4a4_gemm_fp6_kernel(
    const uint8_t* __restrict__ A6, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ W6,
    const uint16_t* __restrict__ sw, int M, int N, int K, uint16_t* __restrict__ Y) {
    constexpr int BM = 128, BN = 256, MI = 4;
    __shared__ Stage6 st[2];

    // tile selection (XCD-aware, as the INT8 kernels)
    const int mt_count = (M + BM - 1) / BM;
    const int nt_count = (N + BN - 1) / BN;
    const int T = mt_count * nt_count;
    int mt, nt;
    if ((mt_count & 7) == 0 && (nt_count & 7) == 0) {
        const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
        const int npx = nt_count >> 3;
        const int band = j / (8 * npx), r = j % (8 * npx);
        mt = band * 8 + (r & 7);
        nt = x * npx + (r >> 3);
    } else {
        int tile = blockIdx.x;
        if ((T & 7) == 0) tile = (blockIdx.x & 7) * (T >> 3) + (blockIdx.x >> 3);
        mt = tile % mt_count;
        nt = tile / mt_count;
    }
    const int m0 = mt * BM, n0 = nt * BN;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const bool grp_y = wave >= 4;
    const int l32 = lane & 31, lh = lane >> 5;
    const int nks = K / KS6;
    const int ng = K / 128;
    const uint32_t rowb = static_cast<uint32_t>(3 * K / 4);  // bytes per FP6 row

    // A staging: 1536 chunks of 8 bytes per stage, three per thread (chunk
    // tid + 512 i: row c / 12, byte 8 (c % 12)); kept in scalars, not arrays,
    // which the compiler would move to LDS
    auto a_g = [&](int c) { return static_cast<uint32_t>(min(m0 + c / 12, M - 1)) * rowb + 8 * (c % 12); };
    auto a_l = [&](int c) { return (c / 12) * AROW6 + 8 * (c % 12); };
    const uint32_t ag0 = a_g(tid), ag1 = a_g(tid + 512), ag2 = a_g(tid + 1024);
    const int al0 = a_l(tid), al1 = a_l(tid + 512), al2 = a_l(tid + 1024);
    const bool is_a = tid < BM;
    const int srow = is_a ? min(m0 + tid, M - 1) : min(n0 + min(tid - BM, BN - 1), N - 1);
    const uint16_t* sc_base = is_a ? sa : sw;
    const uint32_t sc_off = static_cast<uint32_t>(srow) * static_cast<uint32_t>(ng);
    // W staging: 1536 chunks of 16 bytes per stage, three per thread (chunk
    // tid + 512 i: row c / 6, byte 16 (c % 6))
    auto w_g = [&](int c) { return static_cast<uint32_t>(min(n0 + c / 6, N - 1)) * rowb + 16 * (c % 6); };
    auto w_l = [&](int c) { return (c / 6) * AROW6 + 16 * (c % 6); };
    const uint32_t wg0 = w_g(tid), wg1 = w_g(tid + 512), wg2 = w_g(tid + 1024);
    const int wl0 = w_l(tid), wl1 = w_l(tid + 512), wl2 = w_l(tid + 1024);

    uint2 ra0, ra1, ra2;
    uint4 rw0, rw1, rw2;
    uint16_t rsc;
    auto load_a = [&](int ks) __attribute__((always_inline)) {
        ks = min(ks, nks - 1);
        const uint8_t* base = A6 + static_cast<int64_t>(ks) * SROW6;
        ra0 = *reinterpret_cast<const uint2*>(base + ag0);
        ra1 = *reinterpret_cast<const uint2*>(base + ag1);
        ra2 = *reinterpret_cast<const uint2*>(base + ag2);
        const uint8_t* wbase = W6 + static_cast<int64_t>(ks) * SROW6;
        rw0 = *reinterpret_cast<const uint4*>(wbase + wg0);
        rw1 = *reinterpret_cast<const uint4*>(wbase + wg1);
        rw2 = *reinterpret_cast<const uint4*>(wbase + wg2);
        rsc = sc_base[sc_off + static_cast<uint32_t>(ks)];
    };
    auto store_a = [&](int buf) __attribute__((always_inline)) {
        *reinterpret_cast<uint2*>(&st[buf].a[al0]) = ra0;
        *reinterpret_cast<uint2*>(&st[buf].a[al1]) = ra1;
        *reinterpret_cast<uint2*>(&st[buf].a[al2]) = ra2;
        *reinterpret_cast<uint4*>(&st[buf].w[wl0]) = rw0;
        *reinterpret_cast<uint4*>(&st[buf].w[wl1]) = rw1;
        *reinterpret_cast<uint4*>(&st[buf].w[wl2]) = rw2;
        st[buf].scale[tid] = rsc;
    };
    // FP6 operand of MFMA kk from 48 bytes: dwords [6 kk, 6 kk + 6); the two
    // upper dwords are not read for FP6 operands
    auto operand = [](const uint4 (&q)[3], int kk) __attribute__((always_inline)) {
        i32x8 o;
        if (kk == 0) {
            o[0] = static_cast<int>(q[0].x); o[1] = static_cast<int>(q[0].y);
            o[2] = static_cast<int>(q[0].z); o[3] = static_cast<int>(q[0].w);
            o[4] = static_cast<int>(q[1].x); o[5] = static_cast<int>(q[1].y);
        } else {
            o[0] = static_cast<int>(q[1].z); o[1] = static_cast<int>(q[1].w);
            o[2] = static_cast<int>(q[2].x); o[3] = static_cast<int>(q[2].y);
            o[4] = static_cast<int>(q[2].z); o[5] = static_cast<int>(q[2].w);
        }
        o[6] = 0;
        o[7] = 0;
        return o;
    };

    f32x16 acc[MI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
    f32x16 D[MI];
    uint2 swh[4];
    float sav[MI];
    const f32x16 zero = {};

    auto mfma_phase = [&](int s, auto PAR) __attribute__((always_inline)) {
        constexpr int par = decltype(PAR)::value;
        const int c = BM + wave * 32 + 4 * lh;
#pragma unroll
        for (int q = 0; q < 4; ++q) swh[q] = *reinterpret_cast<const uint2*>(&st[par].scale[c + 8 * q]);
#pragma unroll
        for (int i = 0; i < MI; ++i) sav[i] = h2f6(st[par].scale[i * 32 + l32]);
        __builtin_amdgcn_sched_barrier(0);
        // block by block, both MFMAs of a block back to back (the second takes
        // the first's result: dependent MFMAs issue without a gap); the next
        // block's 48 bytes are read while one block's MFMAs run
        uint4 wf[3], af[2][3];
        auto frag = [&](int i, uint4 (&f)[3]) __attribute__((always_inline)) {
            const uint8_t* p = &st[par].a[(i * 32 + l32) * AROW6 + 48 * lh];
#pragma unroll
            for (int q = 0; q < 3; ++q) f[q] = *reinterpret_cast<const uint4*>(p + 16 * q);
        };
        {
            const uint8_t* p = &st[par].w[(wave * 32 + l32) * AROW6 + 48 * lh];
#pragma unroll
            for (int q = 0; q < 3; ++q) wf[q] = *reinterpret_cast<const uint4*>(p + 16 * q);
        }
        frag(0, af[0]);
        static_for6<0, MI>([&](auto II) __attribute__((always_inline)) {
            constexpr int i = decltype(II)::value;
            if constexpr (i + 1 < MI) frag(i + 1, af[(i + 1) & 1]);
            D[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(operand(wf, 0), operand(af[i & 1], 0), zero,
                                                                   FMT_E3M2, FMT_E3M2, 0, SCALE_ONE, 0, SCALE_ONE);
            D[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(operand(wf, 1), operand(af[i & 1], 1), D[i],
                                                                   FMT_E3M2, FMT_E3M2, 0, SCALE_ONE, 0, SCALE_ONE);
        });
        // keep that order: reads of the weights and block 0, then (reads of
        // block i + 1, two MFMAs)
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
        static_for6<0, MI - 1>([&](auto) __attribute__((always_inline)) {
            __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        });
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    };
    auto dequant_phase = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < MI; ++i) asm volatile("" : "+v"(D[i]));
#pragma unroll
        for (int i = 0; i < MI; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint32_t pair = (r & 2) ? swh[r >> 2].y : swh[r >> 2].x;
                const uint16_t hw = (r & 1) ? static_cast<uint16_t>(pair >> 16) : static_cast<uint16_t>(pair & 0xFFFFu);
                const float t = D[i][r] * sav[i];
                acc[i][r] = fmaf(t, h2f6(hw), acc[i][r]);
            }
        }
    };
    auto stage_next = [&](int t) __attribute__((always_inline)) {
        store_a(t & 1);
        load_a(t + 1);
    };

    using C0 = std::integral_constant<int, 0>;
    using C1 = std::integral_constant<int, 1>;
    load_a(0);
    store_a(0);
    load_a(1);
    __syncthreads();
    if (grp_y) {
        stage_next(1);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
    }
    const int ahead = grp_y ? 2 : 1;
    auto pin = [](auto& v) __attribute__((always_inline)) { asm volatile("" : "+v"(v)); };
    auto body = [&](int s, auto PAR) __attribute__((always_inline)) {
        mfma_phase(s, PAR);
#pragma unroll
        for (int i = 0; i < MI; ++i) pin(D[i]);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        dequant_phase();
#pragma unroll
        for (int i = 0; i < MI; ++i) pin(acc[i]);
        stage_next(s + ahead);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
    };
    int s = 0;
    for (; s + 2 <= nks; s += 2) {
        body(s, C0{});
        body(s + 1, C1{});
    }
    if (s < nks) body(s, C0{});
    if (!grp_y) __syncthreads();

#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int gm = m0 + i * 32 + l32;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t h01 = __half_as_ushort(__float2half_rn(acc[i][4 * q + 0])) |
                                 (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(acc[i][4 * q + 1]))) << 16);
            const uint32_t h23 = __half_as_ushort(__float2half_rn(acc[i][4 * q + 2])) |
                                 (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(acc[i][4 * q + 3]))) << 16);
            const int gn = n0 + wave * 32 + 8 * q + 4 * lh;
            if (gm < M) {
                uint16_t* dst = Y + static_cast<int64_t>(gm) * N + gn;
                if ((N & 3) == 0 && gn + 3 < N) {
                    *reinterpret_cast<uint2*>(dst) = make_uint2(h01, h23);
                } else {
                    if (gn + 0 < N) dst[0] = static_cast<uint16_t>(h01 & 0xFFFFu);
                    if (gn + 1 < N) dst[1] = static_cast<uint16_t>(h01 >> 16);
                    if (gn + 2 < N) dst[2] = static_cast<uint16_t>(h23 & 0xFFFFu);
                    if (gn + 3 < N) dst[3] = static_cast<uint16_t>(h23 >> 16);
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_pack_fp6(const uint8_t* q4, int64_t rows, int64_t K, uint8_t* q6, hipStream_t stream) {
    const int64_t upr = K / 16, units = rows * upr;
    if (units == 0) return hipSuccess;
    const int64_t need = (units + 255) / 256;
    const int blocks = static_cast<int>(need < (1 << 20) ? need : (1 << 20));
    hipLaunchKernelGGL(pack_fp6_kernel, dim3(blocks), dim3(256), 0, stream, q4, units, upr, K, q6);
    return hipGetLastError();
}

hipError_t launch_gemm_fp6(const uint8_t* A6, const uint16_t* sa, const uint8_t* W6, const uint16_t* sw, int64_t M,
                           int64_t N, int64_t K, uint16_t* Y, hipStream_t stream) {
    const int64_t tiles = ((M + 127) / 128) * ((N + 255) / 256);
    if (tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(w4a4_gemm_fp6_kernel, dim3(static_cast<unsigned>(tiles)), dim3(512), 0, stream, A6, sa, W6, sw,
                       static_cast<int>(M), static_cast<int>(N), static_cast<int>(K), Y);
    return hipGetLastError();
}

}  // namespace apex4
