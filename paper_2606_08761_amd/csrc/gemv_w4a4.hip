// W4A4 group GEMM for a single activation row (single-token decode) on gfx950,
// on the vector ALUs instead of the matrix cores.
//
// Same result as the tiled kernel (APEX4 Sec. 3.2.1, Eq. group_decomposition):
// Y[0, n] = sum_g s_a[g] s_w[n, g] sum_{k in g} A_q[k] W_q[n, k].  At one row
// the work is a matrix-vector product bound by streaming W from HBM, so the
// design is about the load stream, not the contraction:
//   * v_dot8_i32_i4 multiplies 8 packed signed nibbles of A with the 8 nibbles
//     of W at the same k and adds the products: the packed codes are used as
//     stored, with no unpacking.
//   * A wave streams whole weight rows.  One load instruction covers 1 KB of
//     one row (64 lanes x 16 bytes, contiguous), so lane l of chunk c holds the
//     32 codes k in [2048 c + 32 l, 2048 c + 32 l + 32), all in one group
//     (every supported G is a multiple of 32).  Each wave keeps its whole share
//     of rows (up to 16 loads per lane) in flight at once, and the workgroups
//     are small (4 waves) so that many waves per CU keep the HBM queue full.
//   * The lane's 32-code partial sum is exact in int32 (|p| <= 2048).  It is
//     dequantized right away with its group's scales, t = p s_a, acc += t s_w
//     (binary32; splitting a group into 32-code partials changes only the fp32
//     rounding, never the exact group sum).
//   * A's codes and scales (as binary32) sit in LDS, staged once per
//     workgroup while the first weight loads are in flight; every wave reads
//     the 16 bytes matching its weight load.
//   * A row's 64 lane partials are summed in a fixed butterfly order and
//     rounded once to binary16.
//   * Fused linear (FUSE, G <= 512): the kernel takes the binary16 row x
//     instead of its codes and quantizes it into LDS in the prologue with the
//     quantizer's own arithmetic (quant_core.h: same codes and scales, bit for
//     bit); workgroup 0 also writes them to the caller's work buffers.
//   * Tiled weights (w4a4_gemv_tiled_kernel): W in the tiled layout
//     (apex4_internal.h), where a 1 KB run holds 16 bytes of each of 32 rows:
//     a workgroup takes one 32-row tile and its 8 waves split the tile's 1 KB
//     runs; lanes l and l + 32 hold the same row, so a row's sum is one
//     shuffle, then the waves' partials are added in a fixed order in LDS.
//   * Two rows (tiled weights, R = 2): every weight run is multiplied with
//     both activation rows (both in LDS), so the weights are still read once;
//     the VALU work doubles.  Measured on MI355X against the MFMA few-row
//     kernel at M = 2 (tiled weights, rotated, graph replay): 7-12 % faster at
//     N = 10240 and 28672 or K = 28672, even at N = K = 8192; at M = 3..4 the
//     four-row form was 5-17 % slower and at M = 8 40-55 %, so only M = 2
//     takes it.
//   * DUMP (rows [pm0, pm0 + pmr) of the R): every lane's exact 32-code partial
//     sum is added with an integer atomic into the zeroed P[pmr][N][K/G],
//     giving the exact group sums whatever the order; sa == nullptr (codes
//     only) skips the scales and Y.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "apex4_internal.h"
#include "quant_core.h"

namespace apex4 {
namespace {

constexpr int GV_WAVES = 4;     // waves per workgroup
constexpr int GV_NT = 64 * GV_WAVES;
constexpr int GV_LOADS = 16;    // 16-byte weight loads in flight per lane
constexpr int GV_CHUNK = 1024;  // bytes of a weight row per load instruction
constexpr int GV_FQ = 4;        // fused prologue: 16-byte loads of x in flight per thread
constexpr int GV_MAX_LDS = 64 * 1024;

__device__ __forceinline__ float gv_h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }

// Sum over the 64 lanes of a wave in a fixed order (every lane gets the sum).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) v += __shfl_xor(v, d, 64);
    return v;
}

// A's codes (K/2 bytes) into gv_lds and s_a as binary32 [K/G] into sa_lds, by
// the NT threads of a workgroup: copied from Aq / sa, or (FUSE) quantized from
// the binary16 row x with the quantizer's arithmetic (quant_core.h: the same
// codes and scales, bit for bit), which workgroup 0 also writes to aq_out /
// sa_out.  QL = G / 8: slots of 8 values per group (FUSE only).
template <bool FUSE, int QL, int NT>
__device__ __forceinline__ void gv_stage_a(uint4* gv_lds, float* sa_lds, const uint8_t* __restrict__ Aq,
                                           const uint16_t* __restrict__ sa, bool have_sc, int K, int ng,
                                           const uint16_t* __restrict__ x, uint8_t* __restrict__ aq_out,
                                           uint16_t* __restrict__ sa_out) {
    const int tid = threadIdx.x;
    [[maybe_unused]] const int kb = K / 2;
    if constexpr (FUSE) {
        // SymQuant of x in slots of 8 values (slot s: k in [8 s, 8 s + 8)),
        // QL consecutive slots per group.  Slot base + tid + u NT is
        // lane-consecutive, so a group is QL neighbouring lanes of one wave,
        // all active (slots past K load zeros: code 0, scale 0).
        const int nslots = K / 8;
        uint4 v[GV_FQ];
        auto load_x = [&](int base) __attribute__((always_inline)) {
#pragma unroll
            for (int u = 0; u < GV_FQ; ++u) {
                const int s = base + tid + u * NT;
                v[u] = s < nslots ? *reinterpret_cast<const uint4*>(x + static_cast<int64_t>(s) * 8) : make_uint4(0u, 0u, 0u, 0u);
            }
        };
        load_x(0);
        for (int base = 0; base < nslots; base += GV_FQ * NT) {
            uint32_t packed[GV_FQ];
            uint16_t sbits[GV_FQ];
#pragma unroll
            for (int u = 0; u < GV_FQ; ++u) {
                if (base + u * NT < nslots) {  // uniform: thread 0 has a slot
                    const uint32_t am = quant::group_max<QL>(quant::absmax8_bits(v[u]));
                    const float sf = quant::scale_of(am, &sbits[u]);
                    packed[u] = quant::pack8(v[u], sf, quant::inv_of(sf));
                }
            }
            if (base + GV_FQ * NT < nslots) load_x(base + GV_FQ * NT);
#pragma unroll
            for (int u = 0; u < GV_FQ; ++u) {
                const int s = base + tid + u * NT;
                if (s < nslots) {
                    reinterpret_cast<uint32_t*>(gv_lds)[s] = packed[u];
                    const bool lead = (s & (QL - 1)) == 0;
                    if (lead) sa_lds[s / QL] = gv_h2f(sbits[u]);
                    if (blockIdx.x == 0) {
                        reinterpret_cast<uint32_t*>(aq_out)[s] = packed[u];
                        if (lead) sa_out[s / QL] = sbits[u];
                    }
                }
            }
        }
    } else {
        for (int i = tid; i < kb / 16; i += NT) gv_lds[i] = reinterpret_cast<const uint4*>(Aq)[i];
        if (have_sc)
            for (int i = tid; i < ng; i += NT) sa_lds[i] = gv_h2f(sa[i]);
    }
}

// Wave w of workgroup b owns weight rows n0 .. n0 + rpw - 1,
// n0 = (b * GV_WAVES + w) * rpw, and walks its (row, chunk) pairs row-major in
// batches of GV_LOADS loads.  lgG: log2(G), or 31 for G = K (one group).
// QL = G / 8: slots of 8 values per group (FUSE only).
template <bool FUSE, int QL, bool DUMP>
__global__ __launch_bounds__(GV_NT) void w4a4_gemv_kernel(
    const uint8_t* __restrict__ Aq, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ Wq,
    const uint16_t* __restrict__ sw, int N, int K, int G, int lgG, int rpw, uint16_t* __restrict__ Y,
    const uint16_t* __restrict__ x, uint8_t* __restrict__ aq_out, uint16_t* __restrict__ sa_out,
    int32_t* __restrict__ P, int pmr) {
    const bool have_sc = FUSE || !DUMP || sa != nullptr;  // uniform
    // A's codes (K/2 bytes), then s_a as binary32 [K/G]
    extern __shared__ uint4 gv_lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kb = K / 2;                            // bytes per row
    const int nch = (kb + GV_CHUNK - 1) / GV_CHUNK;  // chunks per row
    const int ng = K / G;
    const int n0 = (static_cast<int>(blockIdx.x) * GV_WAVES + wave) * rpw;
    const int units = rpw * nch;
    float* sa_lds = reinterpret_cast<float*>(gv_lds + kb / 16);

    uint4 w[GV_LOADS];
    uint16_t sws[GV_LOADS];
    // loads of pairs f0 .. f0 + GV_LOADS - 1 (pairs past the wave's share, rows
    // past N and bytes past the row end load nothing)
    auto issue = [&](int f0) __attribute__((always_inline)) {
        int r = f0 / nch, c = f0 - r * nch;
#pragma unroll
        for (int j = 0; j < GV_LOADS; ++j) {
            const int n = n0 + r;
            const int off = c * GV_CHUNK + 16 * lane;
            const bool ok = f0 + j < units && n < N && off < kb;
            w[j] = ok ? *reinterpret_cast<const uint4*>(Wq + static_cast<int64_t>(n) * kb + off) : make_uint4(0u, 0u, 0u, 0u);
            sws[j] = (ok && have_sc) ? sw[static_cast<int64_t>(n) * ng + ((2 * off) >> lgG)] : static_cast<uint16_t>(0);
            if (++c == nch) {
                c = 0;
                ++r;
            }
        }
    };

    if (n0 < N) issue(0);
    // A's codes and scales into LDS while the first weight loads are in flight
    gv_stage_a<FUSE, QL, GV_NT>(gv_lds, sa_lds, Aq, sa, have_sc, K, ng, x, aq_out, sa_out);
    __syncthreads();
    if (n0 >= N) return;  // after the only barrier

    float acc = 0.f;
    for (int f0 = 0; f0 < units; f0 += GV_LOADS) {
        if (f0 > 0) issue(f0);
        int r = f0 / nch, c = f0 - r * nch;
#pragma unroll
        for (int j = 0; j < GV_LOADS; ++j) {
            if (f0 + j < units) {  // uniform
                const int off = c * GV_CHUNK + 16 * lane;
                if (off < kb) {
                    const uint4 a = gv_lds[off >> 4];
                    int p = __builtin_amdgcn_sdot8(static_cast<int>(a.x), static_cast<int>(w[j].x), 0, false);
                    p = __builtin_amdgcn_sdot8(static_cast<int>(a.y), static_cast<int>(w[j].y), p, false);
                    p = __builtin_amdgcn_sdot8(static_cast<int>(a.z), static_cast<int>(w[j].z), p, false);
                    p = __builtin_amdgcn_sdot8(static_cast<int>(a.w), static_cast<int>(w[j].w), p, false);
                    if constexpr (DUMP) {
                        const int n = n0 + r;
                        if (pmr > 0 && n < N) atomicAdd(&P[static_cast<int64_t>(n) * ng + ((2 * off) >> lgG)], p);
                    }
                    if (have_sc) {
                        const float t = static_cast<float>(p) * sa_lds[(2 * off) >> lgG];
                        acc = fmaf(t, gv_h2f(sws[j]), acc);
                    }
                }
                if (c == nch - 1) {  // row n0 + r complete (uniform)
                    const float s = wave_sum(acc);
                    const int n = n0 + r;
                    if (have_sc && lane == 0 && n < N) Y[n] = __half_as_ushort(__float2half_rn(s));
                    acc = 0.f;
                }
            }
            if (++c == nch) {
                c = 0;
                ++r;
            }
        }
    }
}

constexpr int GT_WAVES = 8;  // tiled: waves per workgroup (one 32-row tile)
constexpr int GT_NT = 64 * GT_WAVES;
constexpr int GT_MAX_LDS = 128 * 1024 + 1024;  // dynamic LDS of the tiled kernel (the static part is 1 KB)
constexpr int GT_SWP = 16;                      // weight scales per thread loaded ahead (K/G <= 256 in full)

// One row against tiled weights.  Workgroup t owns rows 32 t .. 32 t + 31; its
// wave w takes the tile's 1 KB runs q = w, w + GT_WAVES, ... (run q = stage
// q / 2, half q % 2), GV_LOADS at a time; lane l holds row 32 t + l % 32 and the
// 32 codes at packed bytes 64 (q / 2) + 32 (l / 32) + 16 (q % 2).  G >= 128, so
// a run lies in one group, g = 128 (q / 2) / G for every lane: the tile's
// weight scales are staged in LDS group-major ([K/G][32], one coalesced pass)
// and a run reads 32 consecutive ones.
// R activation rows (1, or 2 without FUSE): A rows r at gv_lds + r K/32,
// their scales at sa_lds + r K/G; rows past M repeat row M - 1 (never stored).
template <bool FUSE, int QL, bool DUMP, int R = 1>
__global__ __launch_bounds__(GT_NT) void w4a4_gemv_tiled_kernel(
    const uint8_t* __restrict__ Aq, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ Wt,
    const uint16_t* __restrict__ sw, int M, int N, int K, int G, int lgG, uint16_t* __restrict__ Y,
    const uint16_t* __restrict__ x, uint8_t* __restrict__ aq_out, uint16_t* __restrict__ sa_out,
    int32_t* __restrict__ P, int pm0, int pmr) {
    static_assert(R == 1 || !FUSE, "the fused prologue quantizes one row");
    static_assert(R <= GT_WAVES, "one wave per output row in the final sum");
    const bool have_sc = FUSE || !DUMP || sa != nullptr;  // uniform
    extern __shared__ uint4 gv_lds[];
    __shared__ float red[GT_WAVES][R][32];
    const int tid = threadIdx.x, lane = tid & 63, lh = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kb = K / 2, kv = kb / 16;
    const int ng = K / G;
    const int nq = 2 * static_cast<int>(kstages(K));  // 1 KB runs per tile
    const int row = 32 * static_cast<int>(blockIdx.x) + (lane & 31);
    const bool row_ok = row < N;
    const int nmine = nq > wave ? (nq - wave + GT_WAVES - 1) / GT_WAVES : 0;  // runs of this wave (uniform)
    const uint8_t* wbase = Wt + static_cast<int64_t>(blockIdx.x) * nq * 1024 + 16 * lane;
    float* sa_lds = reinterpret_cast<float*>(gv_lds + R * kv);
    uint16_t* sw_lds = reinterpret_cast<uint16_t*>(sa_lds + R * ng);  // [K/G][32]
    // packed byte of A matching the lane's 16 weight bytes in run q
    auto a_off = [&](int q) { return 64 * (q >> 1) + 32 * lh + 16 * (q & 1); };

    uint4 w[GV_LOADS];
    // runs i0 .. i0 + GV_LOADS - 1 of this wave (the zero padding past K and N
    // loads like any other byte)
    auto issue = [&](int i0) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < GV_LOADS; ++j) {
            const int q = wave + (i0 + j) * GT_WAVES;
            w[j] = i0 + j < nmine ? *reinterpret_cast<const uint4*>(wbase + static_cast<int64_t>(q) * 1024)
                                  : make_uint4(0u, 0u, 0u, 0u);
        }
    };

    issue(0);
    // the tile's weight scales: the first GT_SWP per thread are loaded before A
    // is staged and stored after, so their latency overlaps it; rows past N
    // stage zeros (their sums are never stored)
    const int64_t r0 = 32 * static_cast<int64_t>(blockIdx.x);
    const int nsw = have_sc ? 32 * ng : 0;
    auto sw_at = [&](int i) {
        const int r = i / ng, g = i - r * ng;
        return r0 + r < N ? sw[(r0 + r) * ng + g] : static_cast<uint16_t>(0);
    };
    uint16_t swv[GT_SWP];
#pragma unroll
    for (int u = 0; u < GT_SWP; ++u) swv[u] = tid + u * GT_NT < nsw ? sw_at(tid + u * GT_NT) : static_cast<uint16_t>(0);
    if constexpr (R == 1) {
        gv_stage_a<FUSE, QL, GT_NT>(gv_lds, sa_lds, Aq, sa, have_sc, K, ng, x, aq_out, sa_out);
    } else {
        for (int i = tid; i < R * kv; i += GT_NT) {
            const int r = i / kv, c = i - r * kv;
            gv_lds[i] = reinterpret_cast<const uint4*>(Aq + static_cast<int64_t>(min(r, M - 1)) * kb)[c];
        }
        if (have_sc)
            for (int i = tid; i < R * ng; i += GT_NT) {
                const int r = i / ng, g = i - r * ng;
                sa_lds[i] = gv_h2f(sa[static_cast<int64_t>(min(r, M - 1)) * ng + g]);
            }
    }
#pragma unroll
    for (int u = 0; u < GT_SWP; ++u) {
        const int i = tid + u * GT_NT;
        if (i < nsw) sw_lds[(i % ng) * 32 + i / ng] = swv[u];
    }
    for (int i = tid + GT_SWP * GT_NT; i < nsw; i += GT_NT) sw_lds[(i % ng) * 32 + i / ng] = sw_at(i);
    __syncthreads();

    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
    for (int i0 = 0; i0 < nmine; i0 += GV_LOADS) {
        if (i0 > 0) issue(i0);
#pragma unroll
        for (int j = 0; j < GV_LOADS; ++j) {
            if (i0 + j < nmine) {  // uniform
                const int off = a_off(wave + (i0 + j) * GT_WAVES);
                if (off < kb) {
                    const int g = (2 * off) >> lgG;
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        const uint4 a = gv_lds[r * kv + (off >> 4)];
                        int p = __builtin_amdgcn_sdot8(static_cast<int>(a.x), static_cast<int>(w[j].x), 0, false);
                        p = __builtin_amdgcn_sdot8(static_cast<int>(a.y), static_cast<int>(w[j].y), p, false);
                        p = __builtin_amdgcn_sdot8(static_cast<int>(a.z), static_cast<int>(w[j].z), p, false);
                        p = __builtin_amdgcn_sdot8(static_cast<int>(a.w), static_cast<int>(w[j].w), p, false);
                        if constexpr (DUMP) {
                            if (row_ok && r >= pm0 && r < pm0 + pmr)
                                atomicAdd(&P[(static_cast<int64_t>(r - pm0) * N + row) * ng + g], p);
                        }
                        if (have_sc) {
                            const float t = static_cast<float>(p) * sa_lds[r * ng + g];
                            acc[r] = fmaf(t, gv_h2f(sw_lds[g * 32 + (lane & 31)]), acc[r]);
                        }
                    }
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        acc[r] += __shfl_xor(acc[r], 32, 64);  // the row's two lane halves
        if (lane < 32) red[wave][r][lane] = acc[r];
    }
    __syncthreads();
    // wave r adds row r's eight wave partials in wave order
    if (wave < R && wave < M && lane < 32 && have_sc && row_ok) {
        float v = red[0][wave][lane];
#pragma unroll
        for (int u = 1; u < GT_WAVES; ++u) v += red[u][wave][lane];
        Y[static_cast<int64_t>(wave) * N + row] = __half_as_ushort(__float2half_rn(v));
    }
}

size_t gemv_lds_bytes(int64_t K, int64_t G) { return static_cast<size_t>(K / 2) + 4 * static_cast<size_t>(K / G); }
// tiled, R rows: R rows of codes and scales plus the tile's weight scales, binary16 [K/G][32]
size_t gemv_tiled_lds_bytes(int64_t K, int64_t G, int R = 1) {
    return R * gemv_lds_bytes(K, G) + 64 * static_cast<size_t>(K / G);
}

// Rows per wave and workgroups: fill the load batch, but keep at least 8 waves
// per CU when N allows.
struct GemvGrid {
    int64_t rpw, grid;
};
GemvGrid gemv_grid(int64_t N, int64_t K) {
    const int64_t nch = (K / 2 + GV_CHUNK - 1) / GV_CHUNK;
    int64_t rpw = GV_LOADS / nch;
    const int64_t spread = N / (8 * static_cast<int64_t>(device_cu_count()));
    if (rpw > spread) rpw = spread;
    if (rpw < 1) rpw = 1;
    const int64_t waves = (N + rpw - 1) / rpw;
    return {rpw, (waves + GV_WAVES - 1) / GV_WAVES};
}

template <bool FUSE, int QL, int R = 1>
hipError_t launch_gemv_t(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t N,
                         int64_t K, int64_t G, uint16_t* Y, const uint16_t* x, uint8_t* aq_out, uint16_t* sa_out,
                         Dump dump, bool wt, hipStream_t stream, int64_t M = 1) {
    int lgG = 31;
    if (G != K)
        for (lgG = 5; (int64_t{1} << lgG) < G; ++lgG) {
        }
    const size_t lds = gemv_lds_bytes(K, G);
    const int n = static_cast<int>(N), k = static_cast<int>(K), g = static_cast<int>(G);
    if (dump.P) {
        // 32-code partial sums are added atomically into a zeroed window
        const hipError_t e = launch_fill_i32(dump.P, static_cast<int64_t>(dump.mr) * N * (K / G), 0, stream);
        if (e != hipSuccess) return e;
    }
    if (wt) {
        const dim3 gd(static_cast<unsigned>((N + 31) / 32)), bd(GT_NT);
        const size_t lds_t = gemv_tiled_lds_bytes(K, G, R);
        // above 64 KB of dynamic LDS the kernel must allow it (at most
        // GT_MAX_LDS where the fits functions hold)
        static std::atomic<uint64_t> lds_allowed[2] = {{0}, {0}};
        const void* kf = dump.P ? reinterpret_cast<const void*>(w4a4_gemv_tiled_kernel<FUSE, QL, true, R>)
                                : reinterpret_cast<const void*>(w4a4_gemv_tiled_kernel<FUSE, QL, false, R>);
        const hipError_t ea = allow_dynamic_lds(kf, GT_MAX_LDS, lds_allowed[dump.P ? 1 : 0]);
        if (ea != hipSuccess) return ea;
        if (lds_t > GT_MAX_LDS) return hipErrorInvalidValue;
        const int m = static_cast<int>(M);
        if (dump.P)
            hipLaunchKernelGGL((w4a4_gemv_tiled_kernel<FUSE, QL, true, R>), gd, bd, lds_t, stream, Aq, sa, Wq, sw, m, n,
                               k, g, lgG, Y, x, aq_out, sa_out, dump.P, dump.m0, dump.mr);
        else
            hipLaunchKernelGGL((w4a4_gemv_tiled_kernel<FUSE, QL, false, R>), gd, bd, lds_t, stream, Aq, sa, Wq, sw, m,
                               n, k, g, lgG, Y, x, aq_out, sa_out, static_cast<int32_t*>(nullptr), 0, 0);
        return hipGetLastError();
    }
    if constexpr (R != 1) return hipErrorInvalidValue;  // several rows: tiled weights only
    const GemvGrid gg = gemv_grid(N, K);
    const dim3 gd(static_cast<unsigned>(gg.grid)), bd(GV_NT);
    const int rpw = static_cast<int>(gg.rpw);
    if (dump.P)
        hipLaunchKernelGGL((w4a4_gemv_kernel<FUSE, QL, true>), gd, bd, lds, stream, Aq, sa, Wq, sw, n, k, g, lgG, rpw, Y, x,
                           aq_out, sa_out, dump.P, dump.mr);
    else
        hipLaunchKernelGGL((w4a4_gemv_kernel<FUSE, QL, false>), gd, bd, lds, stream, Aq, sa, Wq, sw, n, k, g, lgG, rpw, Y,
                           x, aq_out, sa_out, static_cast<int32_t*>(nullptr), 0);
    return hipGetLastError();
}

// Workgroups of a one-row launch (row-major: rows-per-wave grid; tiled: one per 32 rows).
int64_t gemv_workgroups(int64_t N, int64_t K, bool wt) { return wt ? (N + 31) / 32 : gemv_grid(N, K).grid; }

}  // namespace

bool gemv_fits(int64_t M, int64_t N, int64_t K, int64_t G, bool wt) {
    const bool g_ok = G == K || G == 32 || G == 64 || G == 128 || G == 256 || G == 512 || G == 1024;
    if (M == 2)  // two rows: tiled weights (G >= 128), both rows in LDS
        return wt && N >= 1 && g_ok && G >= 128 && gemv_tiled_lds_bytes(K, G, 2) <= GT_MAX_LDS;
    return M == 1 && N >= 1 && g_ok && gemv_lds_bytes(K, G) <= GV_MAX_LDS;
}

hipError_t launch_gemv(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                       int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream, Dump dump, bool wt) {
    if (!gemv_fits(M, N, K, G, wt) || (wt && G < 128)) return hipErrorInvalidValue;
    if (M == 2)
        return launch_gemv_t<false, 1, 2>(Aq, sa, Wq, sw, N, K, G, Y, nullptr, nullptr, nullptr, dump, wt, stream, M);
    return launch_gemv_t<false, 1>(Aq, sa, Wq, sw, N, K, G, Y, nullptr, nullptr, nullptr, dump, wt, stream);
}

// Every workgroup quantizes all of x, so the fused prologue's total work is
// (workgroups x K): up to 2^23 it is cheaper than a second launch (measured on
// MI355X: 0.8 - 1.4 us faster at N = 1024 .. 10240, K = 8192), beyond it the
// separate quantizer wins (0.9 us at N = 28672, 12 us at N = 8192, K = 28672).
constexpr int64_t GV_FUSE_WORK = int64_t{1} << 23;
// Tiled weights: 8-wave workgroups, and the fused form only paid up to
// 256 x 8192 (MI355X: about even at N = 8192, K = 8192; 10 us slower at
// N = 10240 and 20 us at N = 28672 than the quantizer and the GEMM).
constexpr int64_t GT_FUSE_WORK = int64_t{1} << 21;

bool fused_linear_fits(int64_t M, int64_t N, int64_t K, int64_t G, bool wt) {
    return M == 1 && gemv_fits(M, N, K, G) && (G == 32 || G == 64 || G == 128 || G == 256 || G == 512) && G < K &&
           !(wt && G < 128) && gemv_workgroups(N, K, wt) * K <= (wt ? GT_FUSE_WORK : GV_FUSE_WORK);
}

hipError_t launch_linear_fused(const uint16_t* x, const uint8_t* Wq, const uint16_t* sw, int64_t M, int64_t N, int64_t K,
                               int64_t G, uint16_t* Y, uint8_t* Aq, uint16_t* sa, hipStream_t stream, Dump dump,
                               bool wt) {
    if (!fused_linear_fits(M, N, K, G, wt)) return hipErrorInvalidValue;
    const uint8_t* no_aq = nullptr;
    const uint16_t* no_sa = nullptr;
    switch (G) {
        case 32: return launch_gemv_t<true, 4>(no_aq, no_sa, Wq, sw, N, K, G, Y, x, Aq, sa, dump, wt, stream);
        case 64: return launch_gemv_t<true, 8>(no_aq, no_sa, Wq, sw, N, K, G, Y, x, Aq, sa, dump, wt, stream);
        case 128: return launch_gemv_t<true, 16>(no_aq, no_sa, Wq, sw, N, K, G, Y, x, Aq, sa, dump, wt, stream);
        case 256: return launch_gemv_t<true, 32>(no_aq, no_sa, Wq, sw, N, K, G, Y, x, Aq, sa, dump, wt, stream);
        default: return launch_gemv_t<true, 64>(no_aq, no_sa, Wq, sw, N, K, G, Y, x, Aq, sa, dump, wt, stream);
    }
}

}  // namespace apex4
