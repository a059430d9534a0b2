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
#include "quant_core.h"

namespace apex4 {
namespace {

using namespace quant;

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

template <int L, int U>
hipError_t launch_small_u(const uint16_t* x, int64_t nslots, uint8_t* q, uint16_t* s, hipStream_t st) {
    const int64_t blocks_needed = (nslots + 256 * U - 1) / (256 * U);
    const int blocks = static_cast<int>(blocks_needed < (1 << 20) ? blocks_needed : (1 << 20));
    hipLaunchKernelGGL((quant_small_kernel<L, U>), dim3(blocks), dim3(256), 0, st, reinterpret_cast<const uint4*>(x),
                       nslots, reinterpret_cast<uint32_t*>(q), s);
    return hipGetLastError();
}

// Two slots per lane once there are enough of them to fill the chip (MI355X:
// 5-15 % faster from M = 2048, K = 8192 up); below that one slot per lane,
// twice the workgroups (10-15 % faster at M = 16 .. 256, K = 8192).
constexpr int64_t QUANT_U2_SLOTS = int64_t{1} << 20;

template <int L>
hipError_t launch_small(const uint16_t* x, int64_t nslots, uint8_t* q, uint16_t* s, hipStream_t st) {
    if (nslots >= QUANT_U2_SLOTS) return launch_small_u<L, 2>(x, nslots, q, s, st);
    return launch_small_u<L, 1>(x, nslots, q, s, st);
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
