// Per-token, per-group SymQuant (b = 4) for gfx950.
//
// APEX4 Sec. 3.2.1, Eq. (SymQuant): S_g = max|X_g| / 7 and
// X_g^q = clamp(round(X_g / S_g), -8, 7); activations are quantized online
// (Sec. 4.4), weights offline with the same formula (Alg. 1).
//
// The kernel is HBM-bound (2 bytes read, 0.5 byte written per element), so the
// design goal is one coalesced 16-byte load per lane per 8 elements and no
// re-reads.  Arithmetic, all in binary32:
//   amax    = max |x|                        exact (binary16 values)
//   S16     = binary16(amax / 7)             correctly rounded division, then
//                                            one RNE conversion; equal to the
//                                            RNE of the exact quotient because
//                                            amax/7 never lies on or within a
//                                            binary32 ulp of a binary16 midpoint
//   code    = clamp(RNE(x / S16), -8, 7)     from t = x * (1/S16): t is within
//                                            10 * 2^-23 of x/S16, while any
//                                            non-tie quotient is >= 2^-14 from a
//                                            half-integer, so rint(t) is right
//                                            except at exact ties; the exact
//                                            residual fma(-q, S16, x) detects a
//                                            tie and picks the even neighbour.
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

// One code from x, the binary16 scale s (as binary32, nonzero) and inv = 1/s.
__device__ __forceinline__ uint32_t code_of(float x, float s, float inv) {
    float q = rintf(x * inv);
    const float d = fmaf(-q, s, x);        // exact: x - q*s
    const float h = 0.5f * s;
    if (fabsf(d) == h) {                   // exact tie: choose the even neighbour
        const int qi = static_cast<int>(q);
        if (qi & 1) q += (d > 0.f) ? 1.f : -1.f;
    }
    q = fminf(fmaxf(q, -8.f), 7.f);
    return static_cast<uint32_t>(static_cast<int>(q)) & 0xFu;
}

__device__ __forceinline__ float absmax8(const uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m = fmaxf(m, fabsf(h2f(w[i] & 0xFFFFu)));
        m = fmaxf(m, fabsf(h2f(w[i] >> 16)));
    }
    return m;
}

// 8 binary16 values -> 8 codes packed low nibble first into one dword.
__device__ __forceinline__ uint32_t pack8(const uint4 v, float s, float inv) {
    if (s == 0.f) return 0u;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t out = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        out |= code_of(h2f(w[i] & 0xFFFFu), s, inv) << (8 * i);
        out |= code_of(h2f(w[i] >> 16), s, inv) << (8 * i + 4);
    }
    return out;
}

__device__ __forceinline__ float scale_of(float amax, uint16_t* s16_bits) {
    const __half s16 = __float2half_rn(amax / 7.0f);
    *s16_bits = __half_as_ushort(s16);
    return __half2float(s16);
}

// Groups of G = 8 * L elements, L in {4, 8, 16, 32, 64} lanes per group.
// A "slot" is 8 consecutive binary16 values (16 bytes).  Slots are numbered
// row-major over the whole matrix; a group is L consecutive slots and never
// straddles a row because K/8 is a multiple of L.  Every lane of a group is
// active together (nslots is a multiple of L and group starts are L-aligned),
// so the xor-shuffle reduction stays inside the group.
template <int L>
__global__ __launch_bounds__(256) void quant_small_kernel(const uint4* __restrict__ x,
                                                          int64_t nslots,
                                                          uint32_t* __restrict__ q,
                                                          uint16_t* __restrict__ s) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t slot = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; slot < nslots;
         slot += stride) {
        const uint4 v = x[slot];
        float amax = absmax8(v);
#pragma unroll
        for (int off = L / 2; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, L));
        uint16_t sbits;
        const float sf = scale_of(amax, &sbits);
        const float inv = (sf != 0.f) ? 1.0f / sf : 0.f;
        q[slot] = pack8(v, sf, inv);
        if ((slot & (L - 1)) == 0) s[slot / L] = sbits;
    }
}

// Large groups (G >= 1024, including per-channel G == K): one workgroup per
// (row, group).  Pass 1 reduces amax over the group, pass 2 re-reads the
// group (from cache) and writes the codes.
__global__ __launch_bounds__(256) void quant_large_kernel(const uint4* __restrict__ x,
                                                          int64_t slots_per_group,
                                                          uint32_t* __restrict__ q,
                                                          uint16_t* __restrict__ s) {
    __shared__ float red[4];
    const int64_t grp = blockIdx.x;
    const uint4* xg = x + grp * slots_per_group;
    uint32_t* qg = q + grp * slots_per_group;
    float amax = 0.f;
    for (int64_t i = threadIdx.x; i < slots_per_group; i += 256) amax = fmaxf(amax, absmax8(xg[i]));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    uint16_t sbits;
    const float sf = scale_of(amax, &sbits);
    const float inv = (sf != 0.f) ? 1.0f / sf : 0.f;
    for (int64_t i = threadIdx.x; i < slots_per_group; i += 256) qg[i] = pack8(xg[i], sf, inv);
    if (threadIdx.x == 0) s[grp] = sbits;
}

template <int L>
hipError_t launch_small(const uint16_t* x, int64_t nslots, uint8_t* q, uint16_t* s, hipStream_t st) {
    const int64_t blocks_needed = (nslots + 255) / 256;
    const int blocks = static_cast<int>(blocks_needed < 65536 ? blocks_needed : 65536);
    hipLaunchKernelGGL(quant_small_kernel<L>, dim3(blocks), dim3(256), 0, st,
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
