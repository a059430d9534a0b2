// MX numerics variant: 4-bit symmetric codes with power-of-two group scales,
// applied inside the block-scaled FP6 matrix instruction of gfx950.
//
// APEX4 (Sec. 3.2.1, Eq. SymQuant) scales each group by S = max|X_g| / 7 in
// FP16, and every group's integer sum then needs its own dequantization on the
// vector ALUs (Eq. group_decomposition) -- the cost the paper is about.  Here
// the scale is the smallest power of two that covers the group,
// 2^E with E = min{e : max|X_g| <= 7 * 2^e}, stored as an E8M0 byte (E + 127).
// v_mfma_scale_f32_32x32x64_f8f6f4 multiplies each lane's 32 FP6 values by its
// own E8M0 scale, so with groups aligned to 32-value blocks the whole
// sum_g 2^(Ea + Ew) P_g is one chain of MFMAs with a single fp32 accumulator:
// no per-group VALU work at all, for any G that is a multiple of 32 (the paper
// notes that block-scaled FP4 on newer NVIDIA parts likewise needs no separate
// dequantization, Sec. 2.2).  This changes the method's scales; the FP16-scale
// path stays the reference.
//
//   * quant_mx_kernel: one lane per 32-value block; the B = G / 32 lanes of a
//     group (consecutive, aligned, in one wave) combine their maxima with
//     cross-lane shuffles.  Codes are written as FP6 e3m2 (code k of a row at
//     bits [6k, 6k + 6), 3K/4 bytes per row), scales as E8M0 bytes [rows, K/G].
//   * w4a4_gemm_mx_kernel: 256 x 256 tiles of 2 x 4 waves of 128 x 64 where
//     they fill the CUs, else 128 x 256 tiles of 8 waves of 128 x 32; both
//     operands staged through LDS (16-byte chunks, six lanes per row-stage),
//     one barrier per 128-wide stage.  Lane half h of MFMA kk holds the
//     stage's codes [64h + 32kk, + 32) of its row, on both operands (as the
//     FP6 kernel), so a lane's block lies in one group and its scale byte is
//     block 2h + kk of the stage's four block scales (selected with the MFMA's
//     op_sel).  Shapes that leave CUs idle may split K across workgroups into
//     fp32 partial tiles (launch_gemm_mx_splitk, caller workspace), summed by
//     the split-K reduction of the INT8 path.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "apex4_internal.h"

namespace apex4 {
namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int MX_SROW = 96;        // FP6 bytes of one row per 128-wide stage
constexpr int MX_LROW = 112;       // padded LDS row (28 dwords)
constexpr int MX_FMT = 3;          // f8f6f4 operand format: FP6 e3m2

// e3m2 code of q in [-8, 7]: magnitudes 0..8 are 0, 12, 16, 18, 20, 21, 22, 23, 24; sign is bit 5
__device__ __forceinline__ uint32_t e3m2_of(int q) {
    constexpr uint64_t POS = 0x17161514'12100C00ull;   // q = 0..7
    constexpr uint64_t NEG = 0x2C303234'35363738ull;   // q = -8..-1, by q + 8
    return static_cast<uint32_t>(((q >= 0 ? POS : NEG) >> (8 * (q & 7))) & 0x3Fu);
}

// One lane per 32-value block of a row; B = G / 32 lanes per group.
template <int B>
__global__ __launch_bounds__(256) void quant_mx_kernel(const uint16_t* __restrict__ x, int64_t nblocks, int bpr,
                                                       int K, uint8_t* __restrict__ q6, uint8_t* __restrict__ e) {
    const int64_t b = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (b >= nblocks) return;  // whole groups: nblocks and the group starts are multiples of B
    const int64_t row = b / bpr;
    const int blk = static_cast<int>(b - row * bpr);
    const uint4* src = reinterpret_cast<const uint4*>(x + row * K + 32 * blk);
    uint32_t h[16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint4 v = src[i];
        h[4 * i] = v.x;
        h[4 * i + 1] = v.y;
        h[4 * i + 2] = v.z;
        h[4 * i + 3] = v.w;
    }
    // largest magnitude: for finite binary16 the order of |x| is that of its low 15 bits
    uint32_t amax = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) amax = max(amax, max(h[i] & 0x7FFFu, (h[i] >> 16) & 0x7FFFu));
#pragma unroll
    for (int o = 1; o < B; o <<= 1) amax = max(amax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(amax), o)));
    // E = min{e : amax <= 7 * 2^e}: with amax = f 2^k, f in [0.5, 1), it is k - 3
    // when f <= 7/8 and k - 2 otherwise (both comparisons exact)
    int E = 0;
    if (amax != 0) {
        int k;
        const float f = frexpf(__half2float(__ushort_as_half(static_cast<uint16_t>(amax))), &k);
        E = f <= 0.875f ? k - 3 : k - 2;
    }
    uint32_t out[6] = {0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 32; ++j) {
        const uint16_t bits = static_cast<uint16_t>(h[j >> 1] >> (16 * (j & 1)));
        // x 2^-E is exact, rintf rounds half to even; |q| <= 7 by the choice of E
        const float v = ldexpf(__half2float(__ushort_as_half(bits)), -E);
        const int q = max(-8, min(7, static_cast<int>(rintf(v))));
        const uint32_t c = e3m2_of(q);
        const int bit = 6 * j;
        out[bit >> 5] |= c << (bit & 31);
        if ((bit & 31) > 26) out[(bit >> 5) + 1] |= c >> (32 - (bit & 31));
    }
    uint2* dst = reinterpret_cast<uint2*>(q6 + row * (3 * static_cast<int64_t>(K) / 4) + 24 * blk);
    dst[0] = make_uint2(out[0], out[1]);
    dst[1] = make_uint2(out[2], out[3]);
    dst[2] = make_uint2(out[4], out[5]);
    if (blk % B == 0) e[row * (bpr / B) + blk / B] = static_cast<uint8_t>(E + 127);
}

template <int BM>
struct StageMX {
    uint8_t a[BM * MX_LROW];
    uint8_t w[256 * MX_LROW];
    uint32_t sa[BM];   // four block scales (bytes 0..3 = blocks 0..3 of the stage) per activation row
    uint32_t sw[256];  // the same per weight row
};

template <int B, typename F>
__device__ __forceinline__ void static_for_mx(F&& f) {
    if constexpr (B > 0) {
        static_for_mx<B - 1>(f);
        f(std::integral_constant<int, B - 1>{});
    }
}

// The stage's block scales of one row, as loaded from its E8M0 scale row
// (GB = G / 32 blocks per group): four bytes (GB = 1), two (GB = 2) or the
// group's one byte.  Only expand_scales touches the value, when it is stored to
// LDS a stage later: arithmetic right after the load would make the wave wait
// for it there (1.4x the kernel time at G = 128, M = 2048, N = K = 8192).
template <int GB>
__device__ __forceinline__ uint32_t load_scales(const uint8_t* __restrict__ erow, int s) {
    if constexpr (GB == 1) return *reinterpret_cast<const uint32_t*>(erow + 4 * s);
    else if constexpr (GB == 2) return *reinterpret_cast<const uint16_t*>(erow + 2 * s);
    else return erow[(4 * s) / GB];
}
// ... as four block-scale bytes (byte b = block b of the stage)
template <int GB>
__device__ __forceinline__ uint32_t expand_scales(uint32_t v) {
    if constexpr (GB == 1) {
        return v;
    } else if constexpr (GB == 2) {
        const uint32_t b0 = v & 0xFFu, b1 = (v >> 8) & 0xFFu;
        return b0 | (b0 << 8) | (b1 << 16) | (b1 << 24);
    } else {
        return (v & 0xFFu) * 0x01010101u;
    }
}

// WM = 1: 128 x 256 tiles, 8 waves of 128 x 32; WM = 2: 256 x 256 tiles, 2 x 4
// waves of 128 x 64 (two column blocks per wave share each activation
// fragment: 40 % fewer LDS bytes per MFMA, half the staging per output).
template <int GB, int WM>
__global__ __launch_bounds__(512, 1) void w4a4_gemm_mx_kernel(
    const uint8_t* __restrict__ A6, const uint8_t* __restrict__ ea, const uint8_t* __restrict__ W6,
    const uint8_t* __restrict__ ew, int M, int N, int K, uint16_t* __restrict__ Y, int nks_split,
    float* __restrict__ part) {
    constexpr int BM = 128 * WM, BN = 256, MI = 4, NJ = WM, WN = 8 / WM;
    constexpr int ACH = (BM * 6 + 511) / 512;  // 16-byte activation chunks per thread and stage
    __shared__ StageMX<BM> st[2];

    // tile selection (XCD-aware, as the other tile kernels)
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
    const int wm = wave / WN, wn = wave % WN;
    const int l32 = lane & 31, lh = lane >> 5;
    // K range: stages [kofs, kofs + nks) of this workgroup's split (blockIdx.y)
    const int nks = nks_split;
    const int kofs = static_cast<int>(blockIdx.y) * nks_split;
    const uint32_t rowb = static_cast<uint32_t>(3 * K / 4);
    const int ng = K / (32 * GB);

    // staging, per stage: activations BM * 6 chunks of 16 bytes (chunk tid + 512 i:
    // row c / 6, byte 16 (c % 6); with WM = 1 waves 0-3 take two and 4-7 one),
    // weights 1536 (three per thread), scales one row per thread below BM + 256.
    // Offsets are kept in scalars, not arrays, which the compiler would move to LDS.
    auto a_g = [&](int c) { return static_cast<uint32_t>(min(m0 + c / 6, M - 1)) * rowb + 16 * (c % 6); };
    auto w_g = [&](int c) { return static_cast<uint32_t>(min(n0 + c / 6, N - 1)) * rowb + 16 * (c % 6); };
    auto l_of = [&](int c) { return (c / 6) * MX_LROW + 16 * (c % 6); };
    const bool a1 = tid + 512 < BM * 6, a2 = ACH > 2 && tid + 1024 < BM * 6;
    const uint32_t ag0 = a_g(tid), ag1 = a_g(a1 ? tid + 512 : tid), ag2 = a_g(a2 ? tid + 1024 : tid);
    const int al0 = l_of(tid), al1 = l_of(a1 ? tid + 512 : tid), al2 = l_of(a2 ? tid + 1024 : tid);
    const uint32_t wg0 = w_g(tid), wg1 = w_g(tid + 512), wg2 = w_g(tid + 1024);
    const int wl0 = l_of(tid), wl1 = l_of(tid + 512), wl2 = l_of(tid + 1024);
    const bool sc_a = tid < BM, sc_w = tid >= BM && tid < BM + BN;
    const uint8_t* erow = sc_a ? ea + static_cast<int64_t>(min(m0 + tid, M - 1)) * ng
                               : ew + static_cast<int64_t>(min(n0 + min(tid - BM, BN - 1), N - 1)) * ng;

    uint4 ra0, ra1, ra2, rw0, rw1, rw2;
    uint32_t rsc = 0;
    auto load = [&](int s) __attribute__((always_inline)) {
        s = min(s, nks - 1) + kofs;
        const uint8_t* abase = A6 + static_cast<int64_t>(s) * MX_SROW;
        ra0 = *reinterpret_cast<const uint4*>(abase + ag0);
        if (a1) ra1 = *reinterpret_cast<const uint4*>(abase + ag1);
        if (a2) ra2 = *reinterpret_cast<const uint4*>(abase + ag2);
        const uint8_t* wbase = W6 + static_cast<int64_t>(s) * MX_SROW;
        rw0 = *reinterpret_cast<const uint4*>(wbase + wg0);
        rw1 = *reinterpret_cast<const uint4*>(wbase + wg1);
        rw2 = *reinterpret_cast<const uint4*>(wbase + wg2);
        if (sc_a || sc_w) rsc = load_scales<GB>(erow, s);
    };
    auto store = [&](int buf) __attribute__((always_inline)) {
        *reinterpret_cast<uint4*>(&st[buf].a[al0]) = ra0;
        if (a1) *reinterpret_cast<uint4*>(&st[buf].a[al1]) = ra1;
        if (a2) *reinterpret_cast<uint4*>(&st[buf].a[al2]) = ra2;
        *reinterpret_cast<uint4*>(&st[buf].w[wl0]) = rw0;
        *reinterpret_cast<uint4*>(&st[buf].w[wl1]) = rw1;
        *reinterpret_cast<uint4*>(&st[buf].w[wl2]) = rw2;
        if (sc_a) st[buf].sa[tid] = expand_scales<GB>(rsc);
        if (sc_w) st[buf].sw[tid - BM] = expand_scales<GB>(rsc);
    };
    // FP6 operand of MFMA kk from a lane's 48 bytes: dwords [6 kk, 6 kk + 6)
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

    f32x16 D[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) D[i][j][r] = 0.f;

    auto compute = [&](int buf) __attribute__((always_inline)) {
        uint4 wf[NJ][3], af[2][3];
        int scw[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int wr = wn * 32 * NJ + j * 32 + l32;
            const uint8_t* wp = &st[buf].w[wr * MX_LROW + 48 * lh];
#pragma unroll
            for (int q = 0; q < 3; ++q) wf[j][q] = *reinterpret_cast<const uint4*>(wp + 16 * q);
            // this lane's two block scales (kk = 0, 1) in bytes 0 and 1
            scw[j] = static_cast<int>(st[buf].sw[wr] >> (16 * lh));
        }
        int sca[MI];
#pragma unroll
        for (int i = 0; i < MI; ++i) sca[i] = static_cast<int>(st[buf].sa[wm * 128 + i * 32 + l32] >> (16 * lh));
        auto frag = [&](int i, uint4 (&f)[3]) __attribute__((always_inline)) {
            const uint8_t* p = &st[buf].a[(wm * 128 + i * 32 + l32) * MX_LROW + 48 * lh];
#pragma unroll
            for (int q = 0; q < 3; ++q) f[q] = *reinterpret_cast<const uint4*>(p + 16 * q);
        };
        frag(0, af[0]);
        static_for_mx<MI>([&](auto II) __attribute__((always_inline)) {
            constexpr int i = decltype(II)::value;
            if constexpr (i + 1 < MI) frag(i + 1, af[(i + 1) & 1]);
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                D[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                    operand(wf[j], 0), operand(af[i & 1], 0), D[i][j], MX_FMT, MX_FMT, 0, scw[j], 0, sca[i]);
                D[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                    operand(wf[j], 1), operand(af[i & 1], 1), D[i][j], MX_FMT, MX_FMT, 1, scw[j], 1, sca[i]);
            }
        });
    };

    // double-buffered pipeline, one barrier per stage: stage s + 1 goes from
    // registers to the other buffer and stage s + 2 is fetched while stage s
    // is multiplied
    load(0);
    store(0);
    load(1);
    __syncthreads();
    for (int s = 0; s < nks; ++s) {
        if (s + 1 < nks) store((s + 1) & 1);
        load(s + 2);
        compute(s & 1);
        __syncthreads();
    }

    // epilogue: lane holds row m and columns 8q + 4h + (0..3), q = 0..3, of each
    // block; a split writes its fp32 partial tile to part[split][m][n] instead
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int gm = m0 + wm * 128 + i * 32 + l32;
        if (gm >= M) continue;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (part) {
                    const int gn = n0 + wn * 32 * NJ + j * 32 + 8 * q + 4 * lh;
                    float* dst = part + static_cast<int64_t>(blockIdx.y) * M * N + static_cast<int64_t>(gm) * N + gn;
                    if ((N & 3) == 0 && gn + 3 < N) {
                        *reinterpret_cast<float4*>(dst) = make_float4(D[i][j][4 * q], D[i][j][4 * q + 1],
                                                                      D[i][j][4 * q + 2], D[i][j][4 * q + 3]);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (gn + e < N) dst[e] = D[i][j][4 * q + e];
                    }
                    continue;
                }
                const uint32_t h01 = __half_as_ushort(__float2half_rn(D[i][j][4 * q + 0])) |
                                     (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(D[i][j][4 * q + 1]))) << 16);
                const uint32_t h23 = __half_as_ushort(__float2half_rn(D[i][j][4 * q + 2])) |
                                     (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(D[i][j][4 * q + 3]))) << 16);
                const int gn = n0 + wn * 32 * NJ + j * 32 + 8 * q + 4 * lh;
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

template <int B>
hipError_t launch_quant_mx_b(const uint16_t* x, int64_t M, int64_t K, uint8_t* q6, uint8_t* e, hipStream_t stream) {
    const int64_t bpr = K / 32, nblocks = M * bpr;
    const int64_t wgs = (nblocks + 255) / 256;
    if (wgs > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(quant_mx_kernel<B>, dim3(static_cast<unsigned>(wgs)), dim3(256), 0, stream, x, nblocks,
                       static_cast<int>(bpr), static_cast<int>(K), q6, e);
    return hipGetLastError();
}

// Split factor over K for the 128 x 256 tiling when it leaves CUs idle: the
// largest S in {2, 4, 8} with tiles * S <= CUs, S dividing the stage count and
// at least 4 stages per split; 1 where no split applies or the 256 x 256
// tiling already fills the CUs.
int mx_split_factor(int64_t M, int64_t N, int64_t K) {
    const int64_t cus = device_cu_count();
    if (((M + 255) / 256) * ((N + 255) / 256) >= cus) return 1;
    const int64_t tiles = ((M + 127) / 128) * ((N + 255) / 256);
    const int64_t nks = K / 128;
    int S = 1;
    for (int c = 2; c <= 8; c *= 2)
        if (tiles * c <= cus && nks % c == 0 && nks / c >= 4) S = c;
    return S;
}

template <int GB>
hipError_t launch_gemm_mx_g(const uint8_t* A6, const uint8_t* ea, const uint8_t* W6, const uint8_t* ew, int64_t M,
                            int64_t N, int64_t K, uint16_t* Y, int S, float* part, hipStream_t stream) {
    const int nks = static_cast<int>(K / 128);
    // 256-row tiles where they still give every CU a workgroup
    const int64_t big = ((M + 255) / 256) * ((N + 255) / 256);
    if (S == 1 && big >= device_cu_count()) {
        if (big > 0x7FFFFFFF) return hipErrorInvalidValue;
        hipLaunchKernelGGL((w4a4_gemm_mx_kernel<GB, 2>), dim3(static_cast<unsigned>(big)), dim3(512), 0, stream, A6, ea,
                           W6, ew, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K), Y, nks,
                           static_cast<float*>(nullptr));
        return hipGetLastError();
    }
    const int64_t tiles = ((M + 127) / 128) * ((N + 255) / 256);
    if (tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((w4a4_gemm_mx_kernel<GB, 1>), dim3(static_cast<unsigned>(tiles), static_cast<unsigned>(S)),
                       dim3(512), 0, stream, A6, ea, W6, ew, static_cast<int>(M), static_cast<int>(N),
                       static_cast<int>(K), Y, nks / S, S > 1 ? part : static_cast<float*>(nullptr));
    return hipGetLastError();
}

hipError_t gemm_mx_dispatch(const uint8_t* A6, const uint8_t* ea, const uint8_t* W6, const uint8_t* ew, int64_t M,
                            int64_t N, int64_t K, int64_t G, uint16_t* Y, int S, float* part, hipStream_t stream) {
    switch (G) {
        case 32: return launch_gemm_mx_g<1>(A6, ea, W6, ew, M, N, K, Y, S, part, stream);
        case 64: return launch_gemm_mx_g<2>(A6, ea, W6, ew, M, N, K, Y, S, part, stream);
        case 128: return launch_gemm_mx_g<4>(A6, ea, W6, ew, M, N, K, Y, S, part, stream);
        case 256: return launch_gemm_mx_g<8>(A6, ea, W6, ew, M, N, K, Y, S, part, stream);
        case 512: return launch_gemm_mx_g<16>(A6, ea, W6, ew, M, N, K, Y, S, part, stream);
        case 1024: return launch_gemm_mx_g<32>(A6, ea, W6, ew, M, N, K, Y, S, part, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_quant_mx(const uint16_t* x, int64_t M, int64_t K, int64_t G, uint8_t* q6, uint8_t* e,
                           hipStream_t stream) {
    switch (G) {
        case 32: return launch_quant_mx_b<1>(x, M, K, q6, e, stream);
        case 64: return launch_quant_mx_b<2>(x, M, K, q6, e, stream);
        case 128: return launch_quant_mx_b<4>(x, M, K, q6, e, stream);
        case 256: return launch_quant_mx_b<8>(x, M, K, q6, e, stream);
        case 512: return launch_quant_mx_b<16>(x, M, K, q6, e, stream);
        case 1024: return launch_quant_mx_b<32>(x, M, K, q6, e, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm_mx(const uint8_t* A6, const uint8_t* ea, const uint8_t* W6, const uint8_t* ew, int64_t M,
                          int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream) {
    return gemm_mx_dispatch(A6, ea, W6, ew, M, N, K, G, Y, 1, nullptr, stream);
}

int64_t mx_splitk_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G) {
    (void)G;
    const int S = M > 0 ? mx_split_factor(M, N, K) : 1;
    return S > 1 ? static_cast<int64_t>(S) * M * N * static_cast<int64_t>(sizeof(float)) : 0;
}

hipError_t launch_gemm_mx_splitk(const uint8_t* A6, const uint8_t* ea, const uint8_t* W6, const uint8_t* ew,
                                 int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, float* part,
                                 hipStream_t stream) {
    const int S = mx_split_factor(M, N, K);
    if (S < 2) return launch_gemm_mx(A6, ea, W6, ew, M, N, K, G, Y, stream);
    const hipError_t e = gemm_mx_dispatch(A6, ea, W6, ew, M, N, K, G, Y, S, part, stream);
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(part, S, M * N, Y, stream);
}

}  // namespace apex4
