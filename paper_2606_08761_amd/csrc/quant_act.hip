// Per-token, per-group SymQuant (b = 4) for gfx950.
//
// APEX4 Sec. 3.2.1, Eq. (SymQuant): S_g = max|X_g| / 7 and
// X_g^q = clamp(round(X_g / S_g), -8, 7); activations are quantized online
// (Sec. 4.4), weights offline with the same formula (Alg. 1).
//
// The kernel is HBM-bound (2 bytes read, 0.5 byte written per element): one
// coalesced 16-byte load per lane per 8 elements, U independent loads in
// flight per lane, no re-reads.  Arithmetic:
//   amax  = max |x|             packed u16 max of the binary16 magnitudes
//                               (exact; magnitudes order like their bits)
//   S16   = binary16(amax * fl(1/7))
//                               equal to the binary16 RNE of the exact
//                               amax / 7 for every binary16 amax (checked
//                               exhaustively on the host)
//   t     = x * rcp(S16)        within 2^-19 of x / S16 (1-ulp reciprocal),
//                               while a non-tie quotient is >= 2^-14 from a
//                               half-integer
//   code  = RNE(clamp(t, -8, 7)) t + 1.5 * 2^23 rounds to the nearest even
//                               integer and leaves its two's-complement nibble
//                               in the low bits; clamping first is equivalent
//                               to clamping the rounded value
//   ties  the exact residual x - code * S16 (one fma) flags a quotient that is
//         exactly k + 1/2; such slots are redone with the even neighbour.
// A zero S16 (amax <= 3 * 2^-24) gives zero codes.  Binary16 subnormals are
// kept (no flush to zero).
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "apex4_internal.h"

namespace apex4 {
namespace {

__device__ __forceinline__ float h2f(uint32_t bits16) {
    return __half2float(__ushort_as_half(static_cast<unsigned short>(bits16)));
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Largest binary16 magnitude of 8 values, as its bit pattern.
__device__ __forceinline__ uint32_t absmax8_bits(const uint4 v) {
    const uint32_t w[4] = {v.x & 0x7FFF7FFFu, v.y & 0x7FFF7FFFu, v.z & 0x7FFF7FFFu, v.w & 0x7FFF7FFFu};
    u16x2 m = __builtin_bit_cast(u16x2, w[0]);
#pragma unroll
    for (int i = 1; i < 4; ++i) m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, w[i]));
    return m.x > m.y ? m.x : m.y;
}

constexpr float RND_MAGIC = 12582912.0f;  // 1.5 * 2^23

// 8 binary16 values -> 8 codes packed low nibble first.  *near_tie is set when
// some t = x / S16 (approximately) lies within 2^-15 of a half-integer; an exact
// tie always sets it (|t - x/S16| < 2^-19) and such slots are recomputed
// exactly.  Clamped elements have t == round(t) and never set it, which is
// right: clamping t first already gives the clamped code.
__device__ __forceinline__ uint32_t pack8_fast(const uint4 v, float inv, bool* near_tie) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t y[8];
    float dev = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float x = h2f((i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xFFFFu));
        const float t = __builtin_amdgcn_fmed3f(fmaf(x, inv, 0.f), -8.f, 7.f);  // one fma_mix from binary16
        const float r = t + RND_MAGIC;                // RNE to an integer, code in the low bits
        dev = fmaxf(dev, fabsf(t - (r - RND_MAGIC)));  // exact: distance of t to its rounding
        y[i] = __float_as_uint(r);
    }
    *near_tie = dev >= 0.5f - 0x1p-15f;
    // byte j = code(2j) | code(2j+1) << 4, then 4 bytes -> one dword
    uint32_t b[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = ((y[2 * j + 1] & 0xFu) << 4) | (y[2 * j] & 0xFu);
    return __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[3], b[2], 0x0c0c0400u), __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u),
                                 0x05040100u);
}

// One code, exact at ties (the even neighbour).
__device__ __forceinline__ uint32_t code_tie(float x, float s, float inv) {
    float q = rintf(__builtin_amdgcn_fmed3f(x * inv, -8.f, 7.f));
    const float d = fmaf(-q, s, x);
    if (fabsf(d) == 0.5f * s && (static_cast<int>(q) & 1)) q = fminf(fmaxf(q + ((d > 0.f) ? 1.f : -1.f), -8.f), 7.f);
    return static_cast<uint32_t>(static_cast<int>(q)) & 0xFu;
}

__device__ __noinline__ uint32_t pack8_ties(const uint4 v, float s, float inv) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t out = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        out |= code_tie(h2f((i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xFFFFu)), s, inv) << (4 * i);
    return out;
}

__device__ __forceinline__ uint32_t pack8(const uint4 v, float s, float inv) {
    if (s == 0.f) return 0u;
    bool near_tie;
    const uint32_t out = pack8_fast(v, inv, &near_tie);
    return near_tie ? pack8_ties(v, s, inv) : out;
}

// Max of the amax bit patterns over L consecutive lanes (L a power of two <= 64).
template <int L>
__device__ __forceinline__ uint32_t group_max(uint32_t a) {
    auto mx = [](uint32_t p, uint32_t q) { return p > q ? p : q; };
    if constexpr (L >= 2) a = mx(a, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(a), 0xB1, 0xF, 0xF, false)));   // xor 1
    if constexpr (L >= 4) a = mx(a, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(a), 0x4E, 0xF, 0xF, false)));   // xor 2
    if constexpr (L >= 8) a = mx(a, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(a), 0x141, 0xF, 0xF, false)));  // half-row mirror
    if constexpr (L >= 16) a = mx(a, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(a), 0x140, 0xF, 0xF, false))); // row mirror
    if constexpr (L >= 32) a = mx(a, static_cast<uint32_t>(__shfl_xor(static_cast<int>(a), 16, 64)));
    if constexpr (L >= 64) a = mx(a, static_cast<uint32_t>(__shfl_xor(static_cast<int>(a), 32, 64)));
    return a;
}

// Scale of a group from its amax bit pattern; returns S16 as binary32.
__device__ __forceinline__ float scale_of(uint32_t amax_bits, uint16_t* s16_bits) {
    const __half s16 = __float2half_rn(h2f(amax_bits) * (1.0f / 7.0f));
    *s16_bits = __half_as_ushort(s16);
    return __half2float(s16);
}

__device__ __forceinline__ float inv_of(float s) { return s != 0.f ? __builtin_amdgcn_rcpf(s) : 0.f; }

// Groups of G = 8 * L elements, L in {4, 8, 16, 32, 64} lanes per group.
// A "slot" is 8 consecutive binary16 values (16 bytes).  Slots are numbered
// row-major over the whole matrix; a group is L consecutive slots and never
// straddles a row because K/8 is a multiple of L.  Each lane handles U slots
// one grid stride apart; every lane of a group is active together (nslots and
// the stride are multiples of L and group starts are L-aligned), so the
// xor-shuffle reduction stays inside the group.
template <int L, int U>
__global__ __launch_bounds__(256) void quant_small_kernel(const uint4* __restrict__ x,
                                                          int64_t nslots,
                                                          uint32_t* __restrict__ q,
                                                          uint16_t* __restrict__ s) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; base < nslots;
         base += stride * U) {
        // x is read exactly once: nontemporal loads keep it from displacing the
        // codes and scales, which the GEMM reads next (about 10 % faster)
        uint4 v[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const int64_t slot = base + j * stride;
            v[j] = make_uint4(0u, 0u, 0u, 0u);
            if (slot < nslots) {
                const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(x) + slot);
                v[j] = make_uint4(t[0], t[1], t[2], t[3]);
            }
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const int64_t slot = base + j * stride;
            const uint32_t am = group_max<L>(absmax8_bits(v[j]));
            uint16_t sbits;
            const float sf = scale_of(am, &sbits);
            const uint32_t packed = pack8(v[j], sf, inv_of(sf));
            if (slot < nslots) {
                q[slot] = packed;
                if ((slot & (L - 1)) == 0) s[slot / L] = sbits;
            }
        }
    }
}

// Large groups (G >= 1024, including per-channel G == K): one workgroup per
// (row, group).  Pass 1 reduces amax over the group, pass 2 re-reads the
// group (from cache) and writes the codes.
__global__ __launch_bounds__(256) void quant_large_kernel(const uint4* __restrict__ x,
                                                          int64_t slots_per_group,
                                                          uint32_t* __restrict__ q,
                                                          uint16_t* __restrict__ s) {
    __shared__ uint32_t red[4];
    const int64_t grp = blockIdx.x;
    const uint4* xg = x + grp * slots_per_group;
    uint32_t* qg = q + grp * slots_per_group;
    uint32_t am = 0;
    for (int64_t i = threadIdx.x; i < slots_per_group; i += 256) {
        const uint32_t a = absmax8_bits(xg[i]);
        am = am > a ? am : a;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(am), off, 64));
        am = am > o ? am : o;
    }
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = am;
    __syncthreads();
    am = red[0] > red[1] ? red[0] : red[1];
    am = am > red[2] ? am : red[2];
    am = am > red[3] ? am : red[3];
    uint16_t sbits;
    const float sf = scale_of(am, &sbits);
    const float inv = inv_of(sf);
    for (int64_t i = threadIdx.x; i < slots_per_group; i += 256) qg[i] = pack8(xg[i], sf, inv);
    if (threadIdx.x == 0) s[grp] = sbits;
}

constexpr int QUANT_UNROLL = 2;

template <int L>
hipError_t launch_small(const uint16_t* x, int64_t nslots, uint8_t* q, uint16_t* s, hipStream_t st) {
    const int64_t blocks_needed = (nslots + 256 * QUANT_UNROLL - 1) / (256 * QUANT_UNROLL);
    const int blocks = static_cast<int>(blocks_needed < (1 << 20) ? blocks_needed : (1 << 20));
    hipLaunchKernelGGL((quant_small_kernel<L, QUANT_UNROLL>), dim3(blocks), dim3(256), 0, st,
                       reinterpret_cast<const uint4*>(x), nslots, reinterpret_cast<uint32_t*>(q), s);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const uint16_t* x, int64_t M, int64_t K, int64_t G, uint8_t* q,
                           uint16_t* s, hipStream_t stream) {
    const int64_t nslots = M * (K / 8);
    switch (G) {
        case 32: return launch_small<4>(x, nslots, q, s, stream);
        case 64: return launch_small<8>(x, nslots, q, s, stream);
        case 128: return launch_small<16>(x, nslots, q, s, stream);
        case 256: return launch_small<32>(x, nslots, q, s, stream);
        case 512: return launch_small<64>(x, nslots, q, s, stream);
        default: break;
    }
    const int64_t groups = M * (K / G);
    if (groups > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(quant_large_kernel, dim3(static_cast<unsigned>(groups)), dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(x), G / 8, reinterpret_cast<uint32_t*>(q), s);
    return hipGetLastError();
}

}  // namespace apex4
