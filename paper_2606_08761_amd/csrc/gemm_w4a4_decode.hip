// W4A4 group GEMM for few rows (M <= 32: decode and small batches) on gfx950.
//
// Same result as the tiled kernel (APEX4 Sec. 3.2.1, Eq. group_decomposition),
// organised for the memory-bound regime, where the weights are streamed from HBM
// once and the HBM queue is kept full.
//   * Work unit: 32 output columns ("tile") by every row.  Workgroups are
//     persistent (at most one per CU) and walk the tiles blockIdx.x,
//     blockIdx.x + gridDim.x, ...  Their 8 waves split the 128-wide K stages
//     round-robin (wave w takes stages w, w + 8, ...), so neighbouring waves read
//     neighbouring 64-byte runs of every weight row.
//   * Each wave streams (tile, stage) pairs through a ring of PF stages of packed
//     weights and activations held in registers.  The ring runs
//     across tile boundaries, so the next tile's loads are in flight while a tile
//     is reduced and stored.  Every wave walks the same number of stages per
//     tile: stages past K are re-reads of the last one with weight 0, which
//     keeps the per-tile barriers uniform.
//   * Per stage, four v_mfma_i32_32x32x32_i8 with the activations as the first
//     operand (lane l holds output column l % 32 and 16 rows) give exactly
//     256 x the stage's partial group sum.  The partial is dequantized right away
//     with its group's scales.  Dequantization is linear in P, so splitting a
//     group into 128-wide partials changes only the fp32 rounding, never the
//     exact group sum.  Every partial satisfies |256 P| <= 2^21, so the
//     1.5 * 2^23 accumulator bias gives the float conversion for free at every G.
//     The weight scale is one value per lane.  The activation scales of all rows
//     and groups (at most 32 * K/G binary16) sit in LDS for the whole kernel
//     (for the stream-K form with fewer tiles than workgroups, per segment).
//   * Groups of 32 or 64 (GPS = 4 or 2 groups per 128-wide stage): each MFMA
//     must stay inside one group, so lane half h of MFMA kk covers
//     k in [32 kk + 16 h, 32 kk + 16 h + 16) (packed bytes 16 kk + 8 h .. + 7)
//     for both operands, and every group's MFMAs start from the bias and are
//     dequantized with that group's scales.
//   * The 8 partial fp32 tiles are summed through LDS in a fixed order and
//     rounded once to binary16.
//   * K need not be a multiple of 128 (G in {32, 64} or G = K): the last stage
//     is then partial and its missing codes load as zeros; its missing groups
//     are skipped.
//   * Tiled weights (wt, G >= 128 or G = K): a wave's 32-column fragment of a
//     stage is one contiguous 2 KB block (each 16-byte load instruction reads
//     1 KB), instead of 64 bytes from each of 32 rows (measured on MI355X with
//     the weights rotated past the 256 MB cache: 5-20 % less time at
//     M = 8..32, N = 8192..57344).
//   * Activations in LDS (ALDS): when K % 512 == 0 and the M packed rows fit
//     beside the scales, the workgroup stages them in LDS once, straight from
//     global memory (global_load_lds, no registers; 16-byte chunks swizzled
//     per row so the rows of a fragment read spread over the banks), and each
//     stage reads its fragment there instead of from global memory.  Every
//     wave otherwise re-reads the activations for each of its tiles, as many
//     requests as the weights (measured on MI355X: 8-23 % of the time at
//     M = 16..32).
//   * The 8 partial fp32 tiles are reduced through LDS in passes of 8 output
//     registers per lane (two passes at M > 16), which keeps the reduction
//     buffer at 16 KB.
//   * Scales are staged into LDS with consecutive lanes on consecutive rows of
//     one 16-byte vector, so a wave's 2-byte stores land in consecutive places
//     of a group (one group stride apart they would all hit one bank), and a
//     stage reads all its groups' scales before its MFMAs.
//   * Stream-K (workspace entry points): where the round-robin walk leaves
//     CUs idle in its last round and the tiles are long, the workgroups keep
//     the full rounds and split the remaining tiles' (tile, stage) units into
//     equal runs; a tile cut between workgroups has its fp32 parts added in
//     segment order, through the workspace, by the workgroup that counts its
//     last part.  With fewer tiles than workgroups the scales are staged per
//     segment, only for the groups it covers.
//   * DUMP: each stage's exact partial group sums of rows [pm0, pm0 + pmr) are
//     added with integer atomics into the zeroed P[pmr][N][K/G] (the sum over a
//     group's stages is exact in any order); sa == nullptr skips the scales
//     and Y.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "apex4_internal.h"

namespace apex4 {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int NWAVE = 8;
constexpr int COLS = 32;
constexpr int ROWS = 32;
constexpr int MAX_SC_LDS = 60 * 1024;         // bytes of each staged scale block ([K/G][32] binary16)
constexpr int RED_ROWS = 8;                    // output registers per lane reduced per pass
constexpr int LDS_TOTAL = 160 * 1024;          // LDS per workgroup on gfx950
constexpr int MAX_DYN_LDS = LDS_TOTAL - NWAVE * RED_ROWS * 64 * 4 - 256;   // scales (+ activations); 256 B for small statics
constexpr int DECODE_PF = 6;                   // stages in flight per wave
constexpr uint32_t MAGIC_BITS = 0x4B400000u;  // binary32 1.5 * 2^23
constexpr float MAGIC = 12582912.0f;

__device__ __forceinline__ float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }
__device__ __forceinline__ uint32_t even_w(uint32_t w) { return (w << 4) & 0xF0F0F0F0u; }
__device__ __forceinline__ uint32_t odd_w(uint32_t w) { return w & 0xF0F0F0F0u; }
__device__ __forceinline__ i32x4 frag2(uint32_t w0, uint32_t w1) {
    i32x4 r;
    r[0] = static_cast<int>(even_w(w0));
    r[1] = static_cast<int>(odd_w(w0));
    r[2] = static_cast<int>(even_w(w1));
    r[3] = static_cast<int>(odd_w(w1));
    return r;
}

// MROWS in {8, 16, 32}: the rows that can hold outputs (M <= MROWS); only they
// are dequantized and reduced.  PF: stages in flight per wave.  GPS: groups per
// 128-wide stage (1 for G >= 128, 2 for G = 64, 4 for G = 32).  Lane l holds
// rows 8 (r / 4) + 4 (l / 32) + r % 4 for r < MROWS / 2.
// TAIL: K % 128 != 0, the last stage is partial and its loads are masked
// (only then: the masks cost selects on every load).
// SK (stream-K, caller workspace): the workgroups first take the whole tiles
// of the full rounds round robin, then equal runs of the tile-major (tile,
// stage) units of the S = ntiles mod grid remaining tiles, so such a tile may be
// cut between two or more of them; each writes its reduced fp32 part of a cut
// tile to part[tile - (ntiles - S)][segment][MROWS/2][64] and counts it in the
// tile's counter (zeroed before the launch); the workgroup that counts the
// tile's last part adds the parts in segment order and stores Y.
template <int MROWS, int PF, int GPS, bool DUMP, bool TAIL, bool ALDS, bool SK>
__global__ __launch_bounds__(64 * NWAVE, 1) void w4a4_decode_kernel(
    const uint8_t* __restrict__ Aq, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ Wq,
    const uint16_t* __restrict__ sw, int M, int N, int K, int G, uint16_t* __restrict__ Y,
    int32_t* __restrict__ P, int pm0, int pmr, int wt, float* part, int* cnt,
    int segmax) {
    const bool have_sc = !DUMP || sa != nullptr;  // uniform
    const bool tiled = GPS == 1 && wt != 0;       // uniform
    constexpr int NR = MROWS / 2;      // output registers per lane that matter
    constexpr int RR = NR < RED_ROWS ? NR : RED_ROWS;
    __shared__ float red[NWAVE][RR][64];
    // [K/G][32] twice: activation scale of row r and group g at g * 32 + r, then
    // the weight scale of the current tile's column c and group g at g * 32 + c;
    // then (ALDS) the packed activation rows 0 .. M-1 (swizzled 16-byte chunks)
    extern __shared__ uint16_t sas[];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int l32 = lane & 31, lh = lane >> 5;
    const int nks = (K + 127) / 128;  // the last stage may be partial
    const int kb = K / 2;
    const int ng = K / G;
    // group of stage s (GPS == 1): s >> lg; first group of stage s (GPS > 1): s * GPS
    const int lg = (G == K) ? 31 : (G <= 128 ? 0 : (G == 256 ? 1 : (G == 512 ? 2 : 3)));
    constexpr int KPG = 4 / GPS;       // MFMAs per group and stage
    const int ntiles = (N + COLS - 1) / COLS;
    // The workgroup walks segments: stage ranges [seg_lo, seg_hi) of one tile.
    // Round robin: whole tiles b, b + grid, ...  Stream-K: the whole tiles of the
    // ntiles / grid full rounds round robin, then the units [u0, u1) of the
    // remaining tiles' tile-major (tile, stage) units.
    const int grid = static_cast<int>(gridDim.x), wg = static_cast<int>(blockIdx.x);
    const int full = SK ? ntiles / grid : 0;
    const int sk_t0 = full * grid;  // first stream-K tile
    const int64_t units = static_cast<int64_t>(ntiles - sk_t0) * nks;
    // the first skg workgroups share the stream-K units, at least one stage per wave each
    const int64_t upw = units / NWAVE;
    const int skg = SK ? static_cast<int>(upw < grid ? (upw > 1 ? upw : 1) : grid) : grid;
    const int64_t u0 = SK && wg < skg ? units * wg / skg : 0;
    const int64_t u1 = SK && wg < skg ? units * (wg + 1) / skg : 0;
    const int sk_first = sk_t0 + static_cast<int>(u0 / nks);
    const int my_segs = SK ? full + (u1 > u0 ? static_cast<int>((u1 - 1) / nks - u0 / nks) + 1 : 0)
                           : (wg < ntiles ? (ntiles - 1 - wg) / grid + 1 : 0);
    auto tile_of = [&](int k) { return (!SK || k < full) ? wg + k * grid : sk_first + (k - full); };
    // Only the first and the last stream-K segment can be cut: their stage
    // bounds, and for each cut one the slot of its part and the tile's count of
    // parts (the workgroups whose ranges meet the tile), are fixed here once.
    const bool has_sk = SK && my_segs > full;
    const int first_lo = has_sk ? static_cast<int>(u0 - static_cast<int64_t>(sk_first - sk_t0) * nks) : 0;
    const int last_hi = has_sk ? static_cast<int>(u1 - static_cast<int64_t>(tile_of(my_segs - 1) - sk_t0) * nks) : nks;
    auto seg_lo = [&](int k) { return (SK && k == full) ? first_lo : 0; };
    auto seg_hi = [&](int k) { return (SK && k == my_segs - 1 && k >= full) ? last_hi : nks; };
    // the workgroup whose stream-K range holds unit u (the largest w with
    // floor(units w / skg) <= u)
    auto wg_of = [&](int64_t u) { return static_cast<int>(((u + 1) * skg + units - 1) / units) - 1; };
    bool cut_c[2] = {false, false};
    int cut_k[2] = {-1, -1}, cut_nseg[2] = {0, 0};
    int64_t cut_slot[2] = {0, 0};
    if (has_sk) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int k = c == 0 ? full : my_segs - 1;
            cut_c[c] = (c == 0 || k != full) && (seg_lo(k) != 0 || seg_hi(k) != nks);
            if (cut_c[c]) {
                const int64_t tu0 = static_cast<int64_t>(tile_of(k) - sk_t0) * nks;
                const int w0 = wg_of(tu0);
                cut_k[c] = k;
                cut_nseg[c] = wg_of(tu0 + nks - 1) - w0 + 1;
                cut_slot[c] = (static_cast<int64_t>(tile_of(k) - sk_t0) * segmax + (wg - w0)) * (NR * 64);
            }
        }
    }
    // stages per wave of segment k (every wave walks them all; the last may be null)
    auto seg_n = [&](int k) { return (seg_hi(k) - seg_lo(k) + NWAVE - 1) / NWAVE; };
    int total = 0;
    for (int k = 0; k < my_segs; ++k) total += seg_n(k);

    // Scales staged in LDS, group-major ([K/G][32]): the activation scales of
    // rows 0..31 (rows past M clamped; their outputs are never stored) for the
    // whole kernel, and the weight scales of the current tile's 32 columns
    // (columns past N clamped).  Rows of 8k scales are read as 16-byte vectors,
    // four per thread with every load issued before the LDS stores, so a staging
    // pass costs one load latency.
    uint16_t* wsc = sas + ng * ROWS;
    // staged activation chunk c of row r sits at 16-byte place r * K/32 + (c ^ (r & 15))
    // (K % 512 == 0), so the 16 rows of a fragment read hit 16 different bank groups
    uint8_t* alds = reinterpret_cast<uint8_t*>(sas + 2 * ng * ROWS);
    constexpr int NT = 64 * NWAVE;
    // groups [glo, ghi) of one or two [32][K/G] blocks (row r at base +
    // min(r, rmax) * K/G) into LDS group-major; a pass covers four 16-byte
    // vectors per thread (two of each block), all loads issued before the
    // stores.  Consecutive lanes take consecutive rows of one vector, so each
    // 2-byte LDS store of a wave covers 32 consecutive places of a group (row
    // index fastest there), not 64 places one group-stride apart in one bank.
    auto stage = [&](const uint16_t* b0, int rmax0, uint16_t* d0, const uint16_t* b1, int rmax1, uint16_t* d1, int glo,
                     int ghi) __attribute__((always_inline)) {
        const bool two = b1 != nullptr;
        if ((ng & 7) == 0) {
            const int vlo = glo >> 3, nv = ((ghi + 7) >> 3) - vlo;  // vectors per row in the range
            const int step = (two ? 2 : 4) * NT;
            for (int i0 = tid; i0 < ROWS * nv; i0 += step) {
                uint4 v[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int b = two ? (u >> 1) : 0;
                    const int i = i0 + (two ? (u & 1) : u) * NT;
                    if (i < ROWS * nv) {
                        const int r = i & (ROWS - 1), c = vlo + i / ROWS;
                        v[u] = *reinterpret_cast<const uint4*>((b ? b1 : b0) + static_cast<int64_t>(min(r, b ? rmax1 : rmax0)) * ng + 8 * c);
                    }
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int b = two ? (u >> 1) : 0;
                    const int i = i0 + (two ? (u & 1) : u) * NT;
                    if (i < ROWS * nv) {
                        const int r = i & (ROWS - 1), c = vlo + i / ROWS;
                        const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
                        uint16_t* d = b ? d1 : d0;
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            d[(8 * c + e) * ROWS + r] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
                    }
                }
            }
        } else {
            const int ngr = ghi - glo;
            for (int b = 0; b < (two ? 2 : 1); ++b)
                for (int i = tid; i < ngr * ROWS; i += NT) {
                    const int r = i & (ROWS - 1), g = glo + i / ROWS;
                    (b ? d1 : d0)[g * ROWS + r] = (b ? b1 : b0)[static_cast<int64_t>(min(r, b ? rmax1 : rmax0)) * ng + g];
                }
        }
    };
    auto tile_col0 = [&](int k) { return tile_of(k) * COLS; };
    auto stage_wscales = [&](int t) __attribute__((always_inline)) {
        const int c0 = tile_col0(t);
        stage(sw + static_cast<int64_t>(c0) * ng, N - 1 - c0, wsc, nullptr, 0, nullptr, 0, ng);
    };
    // The next tile's weight scales, when they fit two 16-byte vectors per
    // thread (K/G <= 256, a multiple of 8): loaded into registers when a tile
    // starts and written to LDS when it ends, so the tile boundary waits for no
    // scale load.
    // Stream-K with no full round (fewer tiles than workgroups): a workgroup
    // walks one or two short segments, so both scale blocks are staged per
    // segment, only for the groups its stages cover.
    const bool pure = SK && full == 0;
    auto seg_glo = [&](int k) { return GPS > 1 ? seg_lo(k) * GPS : (seg_lo(k) >> lg); };
    auto seg_ghi = [&](int k) { return GPS > 1 ? min(ng, seg_hi(k) * GPS) : ((seg_hi(k) - 1) >> lg) + 1; };
    auto stage_both = [&](int k) __attribute__((always_inline)) {
        const int c0 = tile_col0(k);
        stage(sa, M - 1, sas, sw + static_cast<int64_t>(c0) * ng, N - 1 - c0, wsc, pure ? seg_glo(k) : 0,
              pure ? seg_ghi(k) : ng);
    };
    const bool pf_sc = (ng & 7) == 0 && ng <= 256 && !pure;
    uint4 nsc[2];
    auto prefetch_wscales = [&](int t) __attribute__((always_inline)) {
        const int c0 = tile_col0(t), nv = ng >> 3;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int i = tid + u * 64 * NWAVE;
            if (i < ROWS * nv) {
                const int r = i & (ROWS - 1), c = i / ROWS;
                nsc[u] = *reinterpret_cast<const uint4*>(sw + static_cast<int64_t>(min(c0 + r, N - 1)) * ng + 8 * c);
            }
        }
    };
    auto store_wscales = [&]() __attribute__((always_inline)) {
        const int nv = ng >> 3;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int i = tid + u * 64 * NWAVE;
            if (i < ROWS * nv) {
                const int r = i & (ROWS - 1), c = i / ROWS;
                const uint32_t w[4] = {nsc[u].x, nsc[u].y, nsc[u].z, nsc[u].w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    wsc[(8 * c + e) * ROWS + r] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
            }
        }
    };

    // per-lane byte offsets; every load adds a wave-uniform base (stage and group)
    constexpr uint32_t HOFF = GPS > 1 ? 8 : 32;   // byte offset of lane half 1 within a stage
    const uint32_t a_voff = static_cast<uint32_t>(min(l32, M - 1)) * static_cast<uint32_t>(K / 2) + HOFF * lh;
    uint32_t w_voff = 0;
    auto set_tile = [&](int t) {
        if (tiled) {
            w_voff = static_cast<uint32_t>(tile_col0(t) / COLS) * static_cast<uint32_t>(nks) * 2048u + 16u * lane;
        } else {
            const int n = min(tile_col0(t) + l32, N - 1);
            w_voff = static_cast<uint32_t>(n) * static_cast<uint32_t>(K / 2) + HOFF * lh;
        }
    };
    // weight stage and half strides (row-major: 64 and 16 bytes; tiled: 2 KB and 1 KB)
    const int w_sstride = tiled ? 2048 : 64, w_jstride = tiled ? 1024 : 16;

    // ring of in-flight stages; (lt, li) is the next (segment, stage) to load.  No
    // load is issued past the last stage.
    uint4 rw[PF][2], ra[ALDS ? 1 : PF][2];
    int lt = 0, li = 0;
    // 32 packed bytes of one lane for a stage: two 16-byte runs (GPS == 1), or
    // four 8-byte pieces 16 apart (one per MFMA) when groups are finer than a stage
    // lim: packed bytes of the stage inside the row (64 unless it is the partial
    // last stage); pieces past it load as zeros
    auto load32 = [&](const uint8_t* p, uint4 (&r)[2], int lim, int jstride) __attribute__((always_inline)) {
        const bool full = lim >= 64;
        if constexpr (GPS == 1) {
            const int h = static_cast<int>(HOFF) * lh;
            r[0] = (full || h < lim) ? *reinterpret_cast<const uint4*>(p) : make_uint4(0u, 0u, 0u, 0u);
            r[1] = (full || h + 16 < lim) ? *reinterpret_cast<const uint4*>(p + jstride) : make_uint4(0u, 0u, 0u, 0u);
        } else {
            const int h = static_cast<int>(HOFF) * lh;
            const uint2 z = make_uint2(0u, 0u);
            const uint2 q0 = (full || h < lim) ? *reinterpret_cast<const uint2*>(p) : z;
            const uint2 q1 = (full || h + 16 < lim) ? *reinterpret_cast<const uint2*>(p + 16) : z;
            const uint2 q2 = (full || h + 32 < lim) ? *reinterpret_cast<const uint2*>(p + 32) : z;
            const uint2 q3 = (full || h + 48 < lim) ? *reinterpret_cast<const uint2*>(p + 48) : z;
            r[0] = make_uint4(q0.x, q0.y, q1.x, q1.y);
            r[1] = make_uint4(q2.x, q2.y, q3.x, q3.y);
        }
    };
    int l_lo = 0, l_hi = 0, l_n = 0;  // bounds of segment lt
    auto load = [&](int j) {
        const int s = min(l_lo + wave + NWAVE * li, l_hi - 1);
        const uint8_t* wb = Wq + static_cast<int64_t>(s) * w_sstride;
        const uint8_t* ab = Aq + static_cast<int64_t>(s) * 64;
        const int lim = TAIL ? kb - s * 64 : 64;
        load32(wb + w_voff, rw[j], tiled ? 64 : lim, w_jstride);  // the tiled layout is zero padded
        if constexpr (!ALDS) load32(ab + a_voff, ra[j], lim, 16);
        else (void)ab;
        if (++li == l_n) {
            if (lt + 1 < my_segs) {
                li = 0;
                set_tile(++lt);
                l_lo = seg_lo(lt), l_hi = seg_hi(lt), l_n = seg_n(lt);
            } else {
                li = l_n - 1;
            }
        }
    };

    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;

    // the first stages' loads go out before the scale staging, whose waits then
    // overlap them: one memory round trip before the first stage is processed
    if (total > 0) {
        set_tile(0);
        l_lo = seg_lo(0), l_hi = seg_hi(0), l_n = seg_n(0);
#pragma unroll
        for (int j = 0; j < PF; ++j) load(j);
    }
    // ALDS: the packed activation rows go straight into LDS (global_load_lds,
    // 1 KB per wave instruction: 16 bytes per lane at consecutive places), in
    // the swizzled order of alds_slot; the waits come with the scale staging's
    const int cpr = kb / 16;  // 16-byte chunks per activation row
    if constexpr (ALDS) {
        const int nch = M * cpr;
        for (int b = wave; b * 64 < nch; b += NWAVE) {  // wave-uniform
            const int slot = min(b * 64 + lane, nch - 1);  // the last block's spare lanes repeat a chunk
            const int r = slot / cpr, c = (slot - r * cpr) ^ (r & 15);
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(Aq + static_cast<int64_t>(r) * kb + 16 * c),
                (__attribute__((address_space(3))) void*)(alds + b * 1024), 16, 0, 0);
        }
    }
    // activation scales of rows 0 .. 31 (rows past M clamped) and the first
    // tile's weight scales, their loads in flight together
    if (have_sc) {
        if (my_segs > 0) stage_both(0);
        if (pf_sc && my_segs > 1) prefetch_wscales(1);
    }
    if constexpr (ALDS) __builtin_amdgcn_s_waitcnt(0);  // this wave's LDS loads have landed
    __syncthreads();  // activation scales, the first tile's weight scales (and activations) staged

    int pi = 0;  // stage-in-segment of the next processed stage
    int pt = 0;  // segment of the next processed stage
    int p_lo = 0, p_hi = 0, p_n = 0;
    if (my_segs > 0) p_lo = seg_lo(0), p_hi = seg_hi(0), p_n = seg_n(0);
    auto process = [&](int j) {
        const int s_raw = p_lo + wave + NWAVE * pi;
        const bool live = s_raw < p_hi;
        const int s = min(s_raw, p_hi - 1);
        // The stage's scales are read first, so that their LDS latency overlaps
        // the fragment reads and the contraction instead of following each
        // group's MFMAs (a partial last stage's missing groups read a staged
        // group and are skipped below).
        float s1v[GPS];
        uint2 sah[GPS][NR / 4];
        if (have_sc) {
#pragma unroll
            for (int gi = 0; gi < GPS; ++gi) {
                const int g = GPS == 1 ? (s >> lg) : s * GPS + gi;
                const int gc = g < ng ? g : ng - 1;
                const float w1 = h2f(wsc[gc * ROWS + l32]) * (1.0f / 256.0f);
                s1v[gi] = live ? w1 : 0.f;
#pragma unroll
                for (int q4 = 0; q4 < NR / 4; ++q4)
                    sah[gi][q4] = *reinterpret_cast<const uint2*>(&sas[gc * ROWS + 8 * q4 + 4 * lh]);
            }
        }
        i32x4 bw[4], af[4];
        uint4 la[2];
        if constexpr (ALDS) {
            // this lane's 32 packed activation bytes of stage s (row min(l32, M - 1)):
            // chunks 4s + 2h, 4s + 2h + 1 (one group per stage), or 8 bytes at
            // offset 8h of chunks 4s .. 4s + 3 (finer groups)
            const int r = min(l32, M - 1);
            const uint8_t* row = alds + r * cpr * 16;
            auto chunk = [&](int c) __attribute__((always_inline)) { return row + 16 * (c ^ (r & 15)); };
            if constexpr (GPS == 1) {
                la[0] = *reinterpret_cast<const uint4*>(chunk(4 * s + 2 * lh));
                la[1] = *reinterpret_cast<const uint4*>(chunk(4 * s + 2 * lh + 1));
            } else {
                const uint2 q0 = *reinterpret_cast<const uint2*>(chunk(4 * s) + 8 * lh);
                const uint2 q1 = *reinterpret_cast<const uint2*>(chunk(4 * s + 1) + 8 * lh);
                const uint2 q2 = *reinterpret_cast<const uint2*>(chunk(4 * s + 2) + 8 * lh);
                const uint2 q3 = *reinterpret_cast<const uint2*>(chunk(4 * s + 3) + 8 * lh);
                la[0] = make_uint4(q0.x, q0.y, q1.x, q1.y);
                la[1] = make_uint4(q2.x, q2.y, q3.x, q3.y);
            }
        }
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const uint4& v = rw[j][kk >> 1];
            const uint4& u = ALDS ? la[kk >> 1] : ra[j][kk >> 1];
            bw[kk] = (kk & 1) ? frag2(v.z, v.w) : frag2(v.x, v.y);
            af[kk] = (kk & 1) ? frag2(u.z, u.w) : frag2(u.x, u.y);
        }
#pragma unroll
        for (int gi = 0; gi < GPS; ++gi) {
            const int g = GPS == 1 ? (s >> lg) : s * GPS + gi;
            i32x16 d;
#pragma unroll
            for (int r = 0; r < 16; ++r) d[r] = static_cast<int>(MAGIC_BITS);
#pragma unroll
            for (int q = 0; q < KPG; ++q)
                d = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[gi * KPG + q], bw[gi * KPG + q], d, 0, 0, 0);
            if (g >= ng) continue;  // past the last group (partial last stage)
            if constexpr (DUMP) {
                const int col = tile_col0(pt) + l32;
                if (live && col < N) {
#pragma unroll
                    for (int r = 0; r < NR; ++r) {
                        const int row = 8 * (r >> 2) + 4 * lh + (r & 3);
                        if (row >= pm0 && row < pm0 + pmr)
                            atomicAdd(&P[(static_cast<int64_t>(row - pm0) * N + col) * ng + g],
                                      (d[r] - static_cast<int>(MAGIC_BITS)) >> 8);
                    }
                }
                if (!have_sc) continue;
            }
            const float s1 = s1v[gi];
            const float nb = -MAGIC * s1;
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                const uint32_t pair = (r & 2) ? sah[gi][r >> 2].y : sah[gi][r >> 2].x;
                const uint16_t h = (r & 1) ? static_cast<uint16_t>(pair >> 16) : static_cast<uint16_t>(pair & 0xFFFFu);
                const float tt = fmaf(__int_as_float(d[r]), s1, nb);
                acc[r] = fmaf(tt, h2f(h), acc[r]);
            }
        }
    };

    __shared__ int sk_last;
    // reduce the 8 partial tiles of segment k, store (or, for a cut tile, write
    // the part to the workspace), clear the accumulator, and stage the next
    // segment's weight scales (every wave is past segment k's stages after the
    // first barrier; the second publishes the new scales)
    auto finish_tile = [&](int k) {
        const int n0 = tile_of(k) * COLS;
        const bool cut = SK && ((cut_c[0] && k == cut_k[0]) || (cut_c[1] && k == cut_k[1]));  // uniform
        const int64_t slot = (SK && k == cut_k[0]) ? cut_slot[0] : cut_slot[1];
#pragma unroll
        for (int r0 = 0; r0 < NR; r0 += RR) {
#pragma unroll
            for (int r = 0; r < RR; ++r) red[wave][r][lane] = acc[r0 + r];
            __syncthreads();
            if (r0 == 0 && have_sc && k + 1 < my_segs) {
                if (pf_sc) store_wscales();
                else if (pure) stage_both(k + 1);
                else stage_wscales(k + 1);
            }
            for (int o = tid; o < RR * 64; o += 64 * NWAVE) {
                const int r = r0 + (o >> 6), ln = o & 63;
                float v = 0.f;
#pragma unroll
                for (int w = 0; w < NWAVE; ++w) v += red[w][r - r0][ln];
                const int row = 8 * (r >> 2) + 4 * (ln >> 5) + (r & 3);
                const int col = n0 + (ln & 31);
                if (cut) {
                    if (have_sc)
                        __hip_atomic_store(&part[slot + r * 64 + ln], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                } else if (have_sc && row < M && col < N) {
                    Y[static_cast<int64_t>(row) * N + col] = __half_as_ushort(__float2half_rn(v));
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    };

    for (int q0 = 0; q0 < total; q0 += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            if (q0 + j < total) {  // uniform across the workgroup
                process(j);
                if (q0 + j + PF < total) load(j);
                if (++pi == p_n) {
                    finish_tile(pt++);
                    pi = 0;
                    if (pt < my_segs) p_lo = seg_lo(pt), p_hi = seg_hi(pt), p_n = seg_n(pt);
                    if (have_sc && pf_sc && pt + 1 < my_segs) prefetch_wscales(pt + 1);
                }
            }
        }
    }

    // Count the parts of the cut tiles; the workgroup that counts a tile's last
    // part adds all its parts in segment order and stores Y.  The parts are
    // written and read with device-scope atomic accesses, which go to the point
    // where every XCD's L2 sees them; they are complete (vmcnt 0, then the
    // barrier) before the count is added, and the last workgroup reads them only
    // after its count returned, so no L2 write-back or invalidate is needed.
    if constexpr (SK) {
        if (have_sc && (cut_c[0] || cut_c[1])) {
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                if (!cut_c[c]) continue;  // uniform
                const int tile = tile_of(cut_k[c]), nseg = cut_nseg[c];
                if (tid == 0)
                    sk_last = __hip_atomic_fetch_add(&cnt[tile - sk_t0], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                              nseg - 1;
                __syncthreads();
                if (sk_last) {
                    float* tp = part + static_cast<int64_t>(tile - sk_t0) * segmax * (NR * 64);
                    for (int o = tid; o < NR * 64; o += 64 * NWAVE) {
                        const int r = o >> 6, ln = o & 63;
                        const int row = 8 * (r >> 2) + 4 * (ln >> 5) + (r & 3);
                        const int col = tile * COLS + (ln & 31);
                        // eight loads in flight, added in segment order
                        float v = 0.f;
                        for (int q0 = 0; q0 < nseg; q0 += 8) {
                            float t[8];
#pragma unroll
                            for (int j = 0; j < 8; ++j)
                                t[j] = q0 + j < nseg ? __hip_atomic_load(&tp[static_cast<int64_t>(q0 + j) * (NR * 64) + o],
                                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                                     : 0.f;
#pragma unroll
                            for (int j = 0; j < 8; ++j)
                                if (q0 + j < nseg) v = q0 + j == 0 ? t[j] : v + t[j];
                        }
                        if (row < M && col < N) Y[static_cast<int64_t>(row) * N + col] = __half_as_ushort(__float2half_rn(v));
                    }
                }
                __syncthreads();  // sk_last is read before the next count writes it
            }
        }
    }
}

// Bytes of staged scales, and of staged activation rows (whole 1 KB blocks)
// when they fit (ALDS; K % 512 == 0 for the swizzle, so never a partial stage).
int64_t decode_scale_lds(int64_t K, int64_t G) { return 2 * (K / G) * ROWS * static_cast<int64_t>(sizeof(uint16_t)); }

// Stream-K form (workspace), over the S tiles past the full rounds: counters
// [S] (padded to 256 bytes), then the parts [S][segmax][MROWS/2][64] fp32.
// grid == 0: not used.
struct DecodeSK {
    float* part = nullptr;
    int* cnt = nullptr;
    int segmax = 0;
    int grid = 0;
};
struct DecodeSKPlan {
    int grid, segmax;
    int64_t cnt_bytes, bytes;
};
// Round robin gives some workgroups one tile more than others.  The stream-K
// form is taken where it was measured faster: the last round leaves more than a
// tenth of the CUs idle, and the tiles are long: below one tile per CU, at
// least 128 stage-groups (K/128 stages times 128/G groups per stage) and, with
// half the CUs or more busy, at least 192 stages (K >= 24576); from one tile
// per CU on, at least 192 stages.  Below that, a tile's round robin time
// is near the kernel's fixed latency, which the stream-K form's counter clear,
// count and fix-up only add to.  The first skg workgroups (all, unless there
// are fewer than 8 units per workgroup) share the units, so each gets at least
// one stage per wave; a tile's count of parts is the count of them whose
// ranges meet it.
DecodeSKPlan decode_sk_plan(int64_t M, int64_t N, int64_t K, int64_t G) {
    const int64_t ntiles = (N + COLS - 1) / COLS, nks = kstages(K), cus = device_cu_count();
    const int64_t rounds = (ntiles + cus - 1) / cus;
    const int64_t gps = G < 128 ? 128 / G : 1;
    if (rounds * cus * 10 <= ntiles * 11) return {0, 0, 0, 0};
    if (ntiles < cus ? (nks * gps < 128 || (ntiles * 2 >= cus && nks < 192)) : nks < 192) return {0, 0, 0, 0};
    const int64_t skt = ntiles - ntiles / cus * cus;  // tiles past the full rounds
    const int64_t units = skt * nks;
    const int64_t upw = units / NWAVE;
    const int64_t skg = upw < cus ? (upw > 1 ? upw : 1) : cus;
    const int64_t grid = ntiles >= cus ? cus : skg;
    if (ntiles / grid * grid != ntiles - skt) return {0, 0, 0, 0};  // the kernel's full rounds (ntiles / grid)
    const int64_t lmin = units / skg;                               // units per workgroup, at least
    const int64_t span = (nks - 1) / lmin + 2;                      // workgroups one tile can span, at most
    const int64_t segmax = span < skg ? span : skg;
    const int64_t mrows = M <= 8 ? 8 : (M <= 16 ? 16 : 32);
    const int64_t cnt_bytes = (skt * 4 + 255) / 256 * 256;
    return {static_cast<int>(grid), static_cast<int>(segmax), cnt_bytes, cnt_bytes + skt * segmax * (mrows / 2) * 64 * 4};
}
int64_t decode_a_lds(int64_t M, int64_t K) { return (M * (K / 2) + 1023) / 1024 * 1024; }
bool decode_alds(int64_t M, int64_t K, int64_t G) {
    return K % 512 == 0 && decode_a_lds(M, K) + decode_scale_lds(K, G) <= MAX_DYN_LDS;
}

template <int MROWS, int PF, int GPS, bool DUMP, bool TAIL, bool ALDS, bool SK>
hipError_t launch_decode_k(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                           int64_t N, int64_t K, int64_t G, uint16_t* Y, Dump dump, bool wt, hipStream_t stream,
                           DecodeSK sk) {
    static std::atomic<uint64_t> lds_allowed{0};
    const hipError_t e = allow_dynamic_lds(
        reinterpret_cast<const void*>(w4a4_decode_kernel<MROWS, PF, GPS, DUMP, TAIL, ALDS, SK>), MAX_DYN_LDS,
        lds_allowed);
    if (e != hipSuccess) return e;
    const int64_t tiles = (N + COLS - 1) / COLS;
    const int64_t grid = SK ? sk.grid : (tiles < device_cu_count() ? tiles : device_cu_count());
    const size_t lds = static_cast<size_t>(decode_scale_lds(K, G) + (ALDS ? decode_a_lds(M, K) : 0));
    const dim3 gd(static_cast<unsigned>(grid)), bd(64 * NWAVE);
    const int m = static_cast<int>(M), n = static_cast<int>(N), k = static_cast<int>(K), g = static_cast<int>(G);
    hipLaunchKernelGGL((w4a4_decode_kernel<MROWS, PF, GPS, DUMP, TAIL, ALDS, SK>), gd, bd, lds, stream, Aq, sa, Wq, sw,
                       m, n, k, g, Y, dump.P, dump.m0, dump.mr, wt ? 1 : 0, sk.part, sk.cnt, sk.segmax);
    return hipGetLastError();
}

template <int PF, int GPS, bool DUMP, bool TAIL>
hipError_t launch_decode_pf(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                            int64_t N, int64_t K, int64_t G, uint16_t* Y, Dump dump, bool wt, hipStream_t stream,
                            DecodeSK sk) {
    // staging the activations costs one up-front read of them per workgroup,
    // which pays once a wave walks at least 16 stages (several tiles or a long
    // K); below that the per-stage loads overlap better (MI355X: N = K = 8192,
    // one tile per workgroup, 3-9 % slower staged; 8-16 % faster at N = 28672
    // and 57344)
    const int64_t tiles = (N + COLS - 1) / COLS, cus = device_cu_count();
    const int64_t wave_stages = sk.grid ? (tiles * kstages(K) / sk.grid + NWAVE - 1) / NWAVE
                                        : (tiles + cus - 1) / cus * ((K / 128 + NWAVE - 1) / NWAVE);
    const bool alds = !TAIL && wave_stages >= 16 && decode_alds(M, K, G);
#define APEX4_DECODE_SK(R, A)                                                                                          \
    return sk.grid ? launch_decode_k<R, PF, GPS, DUMP, TAIL, A, true>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk) \
                   : launch_decode_k<R, PF, GPS, DUMP, TAIL, A, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk)
#define APEX4_DECODE_ROWS(R)                                                                                           \
    if (alds) { APEX4_DECODE_SK(R, !TAIL); }                                                                           \
    APEX4_DECODE_SK(R, false)
    if (M <= 8) {
        APEX4_DECODE_ROWS(8);
    }
    if (M <= 16) {
        APEX4_DECODE_ROWS(16);
    }
    APEX4_DECODE_ROWS(32);
#undef APEX4_DECODE_ROWS
#undef APEX4_DECODE_SK
}

template <int PF, int GPS>
hipError_t launch_decode_g(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                           int64_t N, int64_t K, int64_t G, uint16_t* Y, Dump dump, bool wt, hipStream_t stream,
                           DecodeSK sk) {
    const bool tail = K % 128 != 0;
    if (!dump.P)
        return tail ? launch_decode_pf<PF, GPS, false, true>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk)
                    : launch_decode_pf<PF, GPS, false, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk);
    // partial sums are added atomically into a zeroed window
    const hipError_t e = launch_fill_i32(dump.P, static_cast<int64_t>(dump.mr) * N * (K / G), 0, stream);
    if (e != hipSuccess) return e;
    return tail ? launch_decode_pf<PF, GPS, true, true>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk)
                : launch_decode_pf<PF, GPS, true, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk);
}

}  // namespace

int device_cu_count() {
    static int n = 0;  // benign race: every caller computes the same value
    if (n == 0) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            n = v;
        else
            return 256;
    }
    return n;
}

bool decode_fits(int64_t M, int64_t N, int64_t K, int64_t G) {
    const bool g_ok = G == K || G == 32 || G == 64 || G == 128 || G == 256 || G == 512 || G == 1024;
    return M >= 1 && M <= ROWS && N >= 1 && g_ok && (K / G) * ROWS * 2 <= MAX_SC_LDS;
}

int64_t decode_split_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G) {
    return decode_fits(M, N, K, G) ? decode_sk_plan(M, N, K, G).bytes : 0;
}

hipError_t launch_gemm_decode(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw,
                              int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream, Dump dump,
                              bool wt, void* workspace) {
    if (!decode_fits(M, N, K, G)) return hipErrorInvalidValue;
    if (wt && G < 128) return hipErrorInvalidValue;  // the tiled layout serves one group per stage or more
    DecodeSK sk;
    if (workspace) {
        const DecodeSKPlan pl = decode_sk_plan(M, N, K, G);
        if (pl.grid) {
            sk.cnt = static_cast<int*>(workspace);
            sk.part = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + pl.cnt_bytes);
            sk.segmax = pl.segmax;
            sk.grid = pl.grid;
            const hipError_t e = launch_fill_i32(sk.cnt, pl.cnt_bytes / 4, 0, stream);
            if (e != hipSuccess) return e;
        }
    }
    // four group sums per stage hold more registers: a shorter ring keeps G = 32 spill-free
    if (G == 32) return launch_decode_g<DECODE_PF - 2, 4>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, false, stream, sk);
    if (G == 64) return launch_decode_g<DECODE_PF, 2>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, false, stream, sk);
    return launch_decode_g<DECODE_PF, 1>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, sk);
}

}  // namespace apex4
