// SymQuant (b = 4) arithmetic shared by the quantizer kernels and the fused
// quantize + GEMM decode path, so both produce the same codes and scales bit
// for bit.  APEX4 Sec. 3.2.1, Eq. (SymQuant): S_g = max|X_g| / 7 and
// X_g^q = clamp(round(X_g / S_g), -8, 7).  The arithmetic and why it is exact
// are described at the top of quant_act.hip.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace apex4 {
namespace quant {
namespace {   // internal linkage in every translation unit that includes it

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

}  // namespace
}  // namespace quant
}  // namespace apex4
