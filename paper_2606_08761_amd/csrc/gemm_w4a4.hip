// Pure W4A4 group-quantized GEMM for gfx950 (CDNA4).
//
// APEX4 Sec. 3.2.1, Eq. (group_decomposition):
//   Y = sum_g (A_g^q W_g^q) (.) (S_g^a S_g^w^T)
// with immediate per-group dequantization for groups and delayed
// dequantization for per-channel scales (Sec. 4.2).
//
// CDNA4 mapping
//   * No 4-bit integer matrix instruction exists on gfx950, so packed nibbles
//     are widened to int8 MFMA operands: (w << 4) & 0xF0F0F0F0 gives the
//     even-position codes times 16, w & 0xF0F0F0F0 the odd-position codes times
//     16 (three VALU ops per 8 codes).  A and W are widened the same way, so
//     every MFMA sums products of matching k and each group sum comes out as
//     exactly 256 P; the 1/256 is folded into the activation scale (a power of
//     two, exact).
//   * v_mfma_i32_32x32x32_i8 accumulates 256 P in int32 per group (exact:
//     |256 P| <= 2^14 G < 2^31 for G <= 2^16).
//   * The MFMA is fed W as its first operand and A as its second, so a 32 x 32
//     result block is Y^T: lane l holds output row m = l % 32 and 16 output
//     columns.  The activation scale is then one value per lane.
//   * Dequantization, binary32 on the VALU, once per group and output element.
//     For G <= 256 the first MFMA of a group starts from the bit pattern of
//     1.5 * 2^23 instead of 0, so the int32 result read as binary32 is
//     1.5 * 2^23 + 256 P exactly (|256 P| <= 2^22), and
//         t   = fma(D, s_a/256, -1.5 * 2^23 * s_a/256)      (= fl(P s_a))
//         acc = fma(t, s_w, acc)          (s_w binary16 through v_fma_mix_f32)
//     i.e. two VALU ops with no int -> float conversion.  Larger groups and
//     per-channel scales use float(D) instead of the bias.
//   * Staging.  The activation tile is shared by all waves of a workgroup: it
//     goes HBM -> registers (one stage ahead) -> widen -> LDS (double-buffered,
//     rows padded to 144 bytes so 8 or 16 consecutive rows at the same chunk
//     hit distinct banks and every fragment offset is an immediate).  Each
//     wave owns distinct weight columns, so the weight fragments go straight
//     from global memory into registers (one stage ahead) and are widened there;
//     the weights never touch LDS.
//   * K slots.  In a 128-wide K stage, lane half h of MFMA kk covers
//     k in [64 h + 16 kk, 64 h + 16 kk + 16): the packed dwords at byte
//     32 h + 8 kk of the row, widened as even(w0), odd(w0), even(w1), odd(w1).
//     A lane's weight bytes for a stage are one contiguous 32-byte run.  For
//     G < 128 each MFMA must stay inside one group, so lane half h of MFMA kk
//     covers k in [32 kk + 16 h, 32 kk + 16 h + 16) (packed byte 16 kk + 8 h).
//   * Groups.  G in {32, 64}: 4 or 2 whole groups per stage, each dequantized
//     after its 1 or 2 MFMAs.  G == 128: one group per stage, each block's group
//     sum is dequantized right after its four MFMAs.  G in {256, 512, 1024}: group sums
//     persist over the stages of a group.  G == K: sums persist over all of K
//     and the scales are applied once in the epilogue.
//   * Workgroup ids are remapped so that each XCD (8 per MI355X, each with its
//     own L2) works on a compact block of output tiles (8 m-tiles by a band of
//     n-tiles at a time).
//   * G in {128, 256} on 128 x 256 tiles runs w4a4_gemm_pp_kernel: the same
//     wave tile and arithmetic, with the two waves of each SIMD running their
//     MFMA and dequant phases half a stage apart (described at the kernel).  Small tiles
//     (64 x 128) may split K over two wave groups (KSPLIT) and keep PF stages
//     of loads in flight.
//   * Split-K across workgroups (launch_gemm_splitk, caller workspace): when
//     the tiles leave CUs idle, the kernel runs on a tiles x S grid, each
//     workgroup over S-th of the stages (whole groups), and writes its partial
//     tile (fp32; exact int32 for G == K); a second kernel adds the S partials
//     in range order and rounds once.
//   * K % 128 != 0 (K % 32 == 0; G in {32, 64} or G == K): the last stage is
//     partial.  Its loads are masked to the row's end (lanes past it hold
//     zero codes, which add nothing) and its missing groups are skipped.
//   * Tiled weights (wt): W may come in the offline tiled layout, 32-row tiles
//     by 128-wide K stages with each lane's 32 bytes of a stage stored
//     contiguously ([N/32][K/128][2][64 lanes][16 B], zero padded), so that a
//     wave's weight fragment for a stage is one contiguous 2 KB block.  Only
//     the weight addressing changes (per-lane base, stage and half strides).
//   * Dump (tests and diagnostics): the same kernels, instantiated with DUMP,
//     also write the exact group sums of a row window, taken from the int32
//     MFMA results before dequantization; the kernel choice (plan_gemm) is the
//     one the production call makes.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "apex4_internal.h"

namespace apex4 {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KS = 128;                       // K elements per pipeline stage
constexpr int KK = KS / 32;                   // MFMAs per 32 x 32 block per stage
constexpr int AROW = KS + 16;                 // padded bytes of one widened LDS row
constexpr uint32_t MAGIC_BITS = 0x4B400000u;  // binary32 1.5 * 2^23
constexpr float MAGIC = 12582912.0f;

enum Mode : int {
    kRotate = 0,    // G <= 128: whole groups per stage
    kPersist = 1,   // G in {256, 512, 1024}: group sums persist over the stages of a group
    kChannel = 2,   // G == K: one scale per row and column, applied in the epilogue
};

template <int BM, int NT, int GPS>
struct Stage {
    int8_t a[BM * AROW];
    uint16_t scale[GPS][NT];   // per group of the stage: [0, BM) s_a rows; [BM, BM + BN) s_w columns
};

__device__ __forceinline__ float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }
__device__ __forceinline__ uint32_t even_w(uint32_t w) { return (w << 4) & 0xF0F0F0F0u; }
__device__ __forceinline__ uint32_t odd_w(uint32_t w) { return w & 0xF0F0F0F0u; }

// 16 int8 MFMA operand values from two packed dwords (16 codes).
__device__ __forceinline__ i32x4 frag2(uint32_t w0, uint32_t w1) {
    i32x4 r;
    r[0] = static_cast<int>(even_w(w0));
    r[1] = static_cast<int>(odd_w(w0));
    r[2] = static_cast<int>(even_w(w1));
    r[3] = static_cast<int>(odd_w(w1));
    return r;
}

// Compile-time loop: f(integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

__device__ __forceinline__ i32x16 splat16(int v) {
    i32x16 r;
#pragma unroll
    for (int i = 0; i < 16; ++i) r[i] = v;
    return r;
}

// One workgroup computes a BM x BN tile with KSPLIT groups of WAVES_M x
// WAVES_N waves; each wave owns MI x NJ blocks of 32 x 32 (rows x columns).
// K-group kg runs the contiguous stages [kg nks/KSPLIT, (kg+1) nks/KSPLIT)
// with LDS buffers of its own, in step with the others (shared barriers); at
// the end the groups' partial tiles are added through LDS in a fixed order.
//
// DUMP: the kernel also writes the exact group sums of rows [pm0, pm0 + pmr)
// to P[pmr][N][K/G] as each group completes (the Y path is unchanged; with
// sa == nullptr the scales are not read and Y is not written).
//
// TAIL: K is not a multiple of 128 (groups of 32 or 64, or G = K): the last
// stage is partial, its missing codes load as zeros, which add nothing to any
// sum, and its missing groups are neither dequantized nor dumped.  Only the
// TAIL instantiations carry the masks: with them in the steady-state code
// the register allocation spilled (up to 900 bytes per lane at G = 32).
template <int WAVES_M, int WAVES_N, int MI, int NJ, int MODE, bool MAGIC_OK, int GPS, int PF, int KSPLIT, bool DUMP,
          bool TAIL>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N * KSPLIT, 1) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ Aq, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ Wq,
    const uint16_t* __restrict__ sw, int M, int N, int K, int G, uint16_t* __restrict__ Y,
    int32_t* __restrict__ P, int pm0, int pmr, int nks_split, void* __restrict__ part, int wt) {
    constexpr int NT = 64 * WAVES_M * WAVES_N;
    constexpr int BM = WAVES_M * MI * 32, BN = WAVES_N * NJ * 32;
    constexpr int A_CH = BM * 4 / NT;                 // 16-byte packed activation chunks per thread
    constexpr bool ROTATE = MODE == kRotate;
    constexpr bool NEED_ACC = (MODE == kRotate || MODE == kPersist);
    constexpr bool FINE = GPS > 1;                    // G < 128: GPS whole groups per stage
    constexpr int KPG = KK / GPS;                     // MFMAs per group and block
    static_assert(A_CH * NT == BM * 4, "tile / thread mismatch");
    static_assert(BM + BN <= NT, "one staged scale per thread");
    static_assert(!FINE || MODE == kRotate, "fine groups rotate");
    __shared__ Stage<BM, NT, GPS> st[2][KSPLIT];
    const bool have_sc = !DUMP || sa != nullptr;  // uniform

    // ---- tile selection (XCD-aware) ----
    // Workgroup b runs on XCD b & 7 (round-robin dispatch), each XCD with its
    // own L2.  When both tile counts are multiples of 8, XCD x owns the n-tiles
    // [x nt/8, (x+1) nt/8) and walks them in bands of 8 m-tiles, so the tiles it
    // runs at the same time share 8 m-tiles of A and their n-tiles of W (at the
    // paper shape 4 MB of A + 4 MB of W per XCD and round, instead of all 8 MB
    // of A + 2 MB of W).  Otherwise XCD x takes a contiguous run of tile ids.
    const int mt_count = (M + BM - 1) / BM;
    const int nt_count = (N + BN - 1) / BN;
    const int T = mt_count * nt_count;
    int mt, nt;
    if ((mt_count & 7) == 0 && (nt_count & 7) == 0) {
        const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
        const int npx = nt_count >> 3;          // n-tiles per XCD
        const int band = j / (8 * npx), r = j % (8 * npx);
        mt = band * 8 + (r & 7);
        nt = x * npx + (r >> 3);
    } else {
        int tile = blockIdx.x;
        if ((T & 7) == 0) tile = (blockIdx.x & 7) * (T >> 3) + (blockIdx.x >> 3);
        mt = tile % mt_count;
        nt = tile / mt_count;
    }
    const int m0 = mt * BM;
    const int n0 = nt * BN;

    const int kg = KSPLIT == 1 ? 0 : static_cast<int>(threadIdx.x) / NT;  // K-group
    const int tid = KSPLIT == 1 ? static_cast<int>(threadIdx.x) : static_cast<int>(threadIdx.x) % NT;
    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, lh = lane >> 5;
    // stages of this K-group, and its first stage: a workgroup covers
    // nks_split stages from blockIdx.y * nks_split (split-K across workgroups)
    const int nks = nks_split / KSPLIT;
    const int kbase = static_cast<int>(blockIdx.y) * nks_split + kg * nks;
    // stages per group (per-channel: one group over all stages)
    const int spg = FINE ? 1 : (MODE == kChannel ? (1 << 30) : G / KS);
    const int ng = K / G;
    const int kb = K / 2;  // packed bytes per row

    // ---- per-lane offsets (32-bit); uniform stage bases live in scalar registers.
    // Rows past M or N are clamped to the last row: they only feed outputs that
    // are never stored, so loads need no branch.
    uint32_t a_off[A_CH];
    int a_lds0[A_CH], a_lds1[A_CH];
    [[maybe_unused]] int a_pos[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
        const int c = tid + i * NT;
        const int r = c >> 2, p = c & 3;
        a_off[i] = static_cast<uint32_t>(min(m0 + r, M - 1)) * static_cast<uint32_t>(K / 2) + p * 16;
        a_pos[i] = 16 * p;  // byte of the chunk within a stage
        if constexpr (FINE) {
            // packed bytes 16p .. 16p+7 and 16p+8 .. 16p+15 are MFMA p, lane halves 0 and 1
            a_lds0[i] = r * AROW + (2 * p) * 16;
            a_lds1[i] = r * AROW + (2 * p + 1) * 16;
        } else {
            // packed dwords 4p .. 4p+3 are lane half p/2, MFMAs 2(p%2) and 2(p%2)+1
            const int c0 = 2 * (2 * (p & 1)) + (p >> 1);
            a_lds0[i] = r * AROW + c0 * 16;
            a_lds1[i] = r * AROW + (c0 + 2) * 16;
        }
    }
    // Scale staged by this thread: an activation row, a weight column, or (past
    // BM + BN) a clamped dummy that is never read.
    const uint16_t* sc_base;
    uint32_t sc_off;
    {
        const bool is_a = tid < BM;
        const int row = is_a ? min(m0 + tid, M - 1) : min(n0 + min(tid - BM, BN - 1), N - 1);
        sc_base = is_a ? sa : sw;
        sc_off = static_cast<uint32_t>(row) * static_cast<uint32_t>(ng);
    }
    // weight bytes: row-major, lane base n K/2 + 32 h, stage stride 64, halves 16
    // apart; tiled (G >= 128 only), lane base (tile stages) 2 KB + 16 lane, stage
    // stride 2 KB, halves 1 KB apart
    const bool tiled = !FINE && wt != 0;  // uniform
    const int w_sstride = tiled ? 2048 : KS / 2;
    const int w_jstride = tiled ? 1024 : 16;
    uint32_t w_off[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        if (tiled) {
            const int t = min((n0 + wn * NJ * 32 + j * 32) / 32, (N + 31) / 32 - 1);
            w_off[j] = static_cast<uint32_t>(t) * static_cast<uint32_t>(kstages(K)) * 2048u + 16u * lane;
        } else {
            const int n = min(n0 + wn * NJ * 32 + j * 32 + l32, N - 1);
            w_off[j] = static_cast<uint32_t>(n) * static_cast<uint32_t>(K / 2) + (FINE ? 8 : 32) * lh;
        }
    }

    // Global loads run PF stages ahead: stage s lives in register slot s % PF
    // (activations and their scales until stored to LDS, weights until widened).
    uint4 ra[PF][A_CH];
    uint16_t rsc[PF][GPS] = {};
    auto load_a = [&](int ks, auto SLOT) __attribute__((always_inline)) {
        constexpr int sl = decltype(SLOT)::value;
        const uint8_t* base = Aq + static_cast<int64_t>(ks) * (KS / 2);
        const int lim = kb - ks * (KS / 2);  // packed bytes of this stage inside the row (uniform)
        if (!TAIL || lim >= KS / 2) {
#pragma unroll
            for (int i = 0; i < A_CH; ++i) ra[sl][i] = *reinterpret_cast<const uint4*>(base + a_off[i]);
        } else {
#pragma unroll
            for (int i = 0; i < A_CH; ++i)
                ra[sl][i] = a_pos[i] < lim ? *reinterpret_cast<const uint4*>(base + a_off[i]) : make_uint4(0u, 0u, 0u, 0u);
        }
        if (have_sc) {
            // the GPS groups of a stage are adjacent in a scale row.  When ng is
            // a multiple of GPS every stage is whole and the row's scales are
            // aligned for one vector load; otherwise (K % 128 != 0) they are
            // read one by one, and past the last group (partial last stage)
            // they read as zero.
            const int g0 = (ks / spg) * GPS;
            const uint16_t* sp = sc_base + sc_off + static_cast<uint32_t>(g0);
            if constexpr (GPS == 1) {
                rsc[sl][0] = *sp;
            } else if (!TAIL || (ng % GPS) == 0) {
                if constexpr (GPS == 2) {
                    const uint32_t v = *reinterpret_cast<const uint32_t*>(sp);
                    rsc[sl][0] = static_cast<uint16_t>(v);
                    rsc[sl][1] = static_cast<uint16_t>(v >> 16);
                } else {
                    const uint2 v = *reinterpret_cast<const uint2*>(sp);
                    rsc[sl][0] = static_cast<uint16_t>(v.x);
                    rsc[sl][1] = static_cast<uint16_t>(v.x >> 16);
                    rsc[sl][2] = static_cast<uint16_t>(v.y);
                    rsc[sl][3] = static_cast<uint16_t>(v.y >> 16);
                }
            } else {
#pragma unroll
                for (int gi = 0; gi < GPS; ++gi) rsc[sl][gi] = g0 + gi < ng ? sp[gi] : static_cast<uint16_t>(0);
            }
        }
    };
    auto store_a = [&](int buf, auto SLOT) __attribute__((always_inline)) {
        constexpr int sl = decltype(SLOT)::value;
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            *reinterpret_cast<i32x4*>(&st[buf][kg].a[a_lds0[i]]) = frag2(ra[sl][i].x, ra[sl][i].y);
            *reinterpret_cast<i32x4*>(&st[buf][kg].a[a_lds1[i]]) = frag2(ra[sl][i].z, ra[sl][i].w);
        }
#pragma unroll
        for (int gi = 0; gi < GPS; ++gi) st[buf][kg].scale[gi][tid] = rsc[sl][gi];
    };
    // w[slot][j][kk / 2] holds the two packed dwords of MFMA kk (x, y for even kk, z, w for odd)
    uint4 w[PF][NJ][2];
    auto load_w = [&](int ks, auto SLOT) __attribute__((always_inline)) {
        constexpr int sl = decltype(SLOT)::value;
        const uint8_t* base = Wq + static_cast<int64_t>(ks) * w_sstride;
        const int lim = kb - ks * (KS / 2);  // uniform
        // full stages (and the zero-padded tiled layout) load unmasked; only a
        // partial last stage takes the per-lane masks (a branch on a uniform
        // value, so the full-stage code carries no selects)
        if (!TAIL || tiled || lim >= KS / 2) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                if constexpr (FINE) {
                    // MFMA kk, lane half h: packed bytes 16 kk + 8 h .. + 7
                    const uint8_t* q = base + w_off[j];
                    const uint2 q0 = *reinterpret_cast<const uint2*>(q);
                    const uint2 q1 = *reinterpret_cast<const uint2*>(q + 16);
                    const uint2 q2 = *reinterpret_cast<const uint2*>(q + 32);
                    const uint2 q3 = *reinterpret_cast<const uint2*>(q + 48);
                    w[sl][j][0] = make_uint4(q0.x, q0.y, q1.x, q1.y);
                    w[sl][j][1] = make_uint4(q2.x, q2.y, q3.x, q3.y);
                } else {
                    w[sl][j][0] = *reinterpret_cast<const uint4*>(base + w_off[j]);
                    w[sl][j][1] = *reinterpret_cast<const uint4*>(base + w_off[j] + w_jstride);
                }
            }
        } else {
            const uint2 z2 = make_uint2(0u, 0u);
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                if constexpr (FINE) {
                    const uint8_t* q = base + w_off[j];
                    const int h8 = 8 * lh;
                    const uint2 q0 = h8 < lim ? *reinterpret_cast<const uint2*>(q) : z2;
                    const uint2 q1 = 16 + h8 < lim ? *reinterpret_cast<const uint2*>(q + 16) : z2;
                    const uint2 q2 = 32 + h8 < lim ? *reinterpret_cast<const uint2*>(q + 32) : z2;
                    const uint2 q3 = 48 + h8 < lim ? *reinterpret_cast<const uint2*>(q + 48) : z2;
                    w[sl][j][0] = make_uint4(q0.x, q0.y, q1.x, q1.y);
                    w[sl][j][1] = make_uint4(q2.x, q2.y, q3.x, q3.y);
                } else {
                    const int h32 = 32 * lh;
                    w[sl][j][0] = h32 < lim ? *reinterpret_cast<const uint4*>(base + w_off[j]) : make_uint4(0u, 0u, 0u, 0u);
                    w[sl][j][1] = h32 + 16 < lim ? *reinterpret_cast<const uint4*>(base + w_off[j] + w_jstride)
                                                 : make_uint4(0u, 0u, 0u, 0u);
                }
            }
        }
    };

    f32x16 acc[NEED_ACC ? MI : 1][NEED_ACC ? NJ : 1];
    if constexpr (NEED_ACC) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    }
    i32x16 psum[ROTATE ? 1 : MI][ROTATE ? 1 : NJ];
    const i32x16 start = splat16(MAGIC_OK ? static_cast<int>(MAGIC_BITS) : 0);

    auto read_a = [&](int buf, int i, i32x4 (&af)[KK]) {
        const int row = wm * MI * 32 + i * 32 + l32;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            af[kk] = *reinterpret_cast<const i32x4*>(&st[buf][kg].a[row * AROW + (2 * kk + lh) * 16]);
    };
    // Weight scales of this lane's 16 columns in block j (binary16 pairs).
    auto read_sw = [&](int buf, int j, uint2 (&swh)[4], int gi = 0) {
        const int c = BM + wn * NJ * 32 + j * 32 + 4 * lh;
#pragma unroll
        for (int q = 0; q < 4; ++q) swh[q] = *reinterpret_cast<const uint2*>(&st[buf][kg].scale[gi][c + 8 * q]);
    };
    // Activation scale of this lane's row in block i, with the 1/256 of the widening.
    auto read_sa = [&](int buf, int i, int gi = 0) {
        return h2f(st[buf][kg].scale[gi][wm * MI * 32 + i * 32 + l32]) * (1.0f / 256.0f);
    };
    auto sw_at = [](const uint2 (&swh)[4], int r) {
        const uint32_t pair = (r & 2) ? swh[r >> 2].y : swh[r >> 2].x;
        return (r & 1) ? static_cast<uint16_t>(pair >> 16) : static_cast<uint16_t>(pair & 0xFFFFu);
    };
    // acc += fl(P s_a) * s_w.
    auto dequant = [&](const i32x16& D, f32x16& a, float sav, const uint2 (&swh)[4]) {
        const float nb = -MAGIC * sav;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float t;
            if constexpr (MAGIC_OK) t = fmaf(__int_as_float(D[r]), sav, nb);
            else t = static_cast<float>(D[r]) * sav;
            a[r] = fmaf(t, h2f(sw_at(swh, r)), a[r]);
        }
    };

    // Exact group sums of block (i, j) for group g into the dump window
    // (d holds 256 P, biased by 1.5 * 2^23 when MAGIC_OK).
    auto dump_block = [&](const i32x16& d, int i, int j, int g) __attribute__((always_inline)) {
        if constexpr (DUMP) {
            const int gm = m0 + wm * MI * 32 + i * 32 + l32;
            if (g < ng && gm >= pm0 && gm < pm0 + pmr) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gn = n0 + wn * NJ * 32 + j * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
                    const int v = MAGIC_OK ? (d[r] - static_cast<int>(MAGIC_BITS)) : d[r];
                    if (gn < N) P[(static_cast<int64_t>(gm - pm0) * N + gn) * ng + g] = v >> 8;
                }
            }
        }
    };

    // One K stage (global stage index gks): widen this wave's weight fragments,
    // issue the next stage's weight loads into the freed registers, then run
    // the row blocks.
    auto compute = [&](int buf, int next, int gks, auto FIRST, auto SLOT) __attribute__((always_inline)) {
        constexpr bool group_first = decltype(FIRST)::value;
        constexpr int sl = decltype(SLOT)::value;
        i32x4 bw[NJ][KK];
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const uint4& v = w[sl][j][kk >> 1];
                bw[j][kk] = (kk & 1) ? frag2(v.z, v.w) : frag2(v.x, v.y);
            }
        // keep both weight copies from being live at once (register budget)
        __builtin_amdgcn_sched_barrier(0);
        load_w(next, SLOT);
        __builtin_amdgcn_sched_barrier(0);
        uint2 swh[ROTATE ? NJ : 1][4];
        float sav[ROTATE ? MI : 1];
        if constexpr (ROTATE) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) read_sw(buf, j, swh[j]);
#pragma unroll
            for (int i = 0; i < MI; ++i) sav[i] = read_sa(buf, i);
        }
        i32x4 af[2][KK];
        read_a(buf, 0, af[0]);
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            if (i + 1 < MI) read_a(buf, i + 1, af[(i + 1) & 1]);
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                i32x16 d;
                if constexpr (ROTATE || group_first) d = start;
                else d = psum[i][j];
#pragma unroll
                for (int kk = 0; kk < KK; ++kk)
                    d = __builtin_amdgcn_mfma_i32_32x32x32_i8(bw[j][kk], af[i & 1][kk], d, 0, 0, 0);
                if constexpr (ROTATE) {
                    dump_block(d, i, j, gks);
                    dequant(d, acc[i][j], sav[i], swh[j]);
                } else {
                    psum[i][j] = d;
                }
            }
        }
    };

    // One K stage holding GPS whole groups (G < 128): for each group and row
    // block, KPG MFMAs from the bias, then dequantize (or dump) right away.
    auto compute_fine = [&](int buf, int next, int ks, auto SLOT) __attribute__((always_inline)) {
        constexpr int sl = decltype(SLOT)::value;
        i32x4 bw[NJ][KK];
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const uint4& v = w[sl][j][kk >> 1];
                bw[j][kk] = (kk & 1) ? frag2(v.z, v.w) : frag2(v.x, v.y);
            }
        __builtin_amdgcn_sched_barrier(0);
        load_w(next, SLOT);
        __builtin_amdgcn_sched_barrier(0);
        constexpr int NF = GPS * MI;
        i32x4 af[2][KPG];
        auto read_f = [&](int f, i32x4 (&dst)[KPG]) __attribute__((always_inline)) {
            const int gi = f / MI, i = f % MI;
            const int row = wm * MI * 32 + i * 32 + l32;
#pragma unroll
            for (int q = 0; q < KPG; ++q)
                dst[q] = *reinterpret_cast<const i32x4*>(&st[buf][kg].a[row * AROW + (2 * (gi * KPG + q) + lh) * 16]);
        };
        read_f(0, af[0]);
        uint2 swh[NJ][4];
        // At G = 32 an item (block f, column block j) is a single MFMA, so item
        // t + 1's MFMA is issued before item t is dequantized, into the other
        // of two result sets: the dequantization then overlaps the next MFMA
        // instead of waiting for its own (with one result set every MFMA also
        // waited for the previous dequantization to read its registers).  At
        // G = 64 (two chained MFMAs per item) a second set brought nothing, and
        // in the debug and partial-last-stage forms it only adds spills.
        if constexpr (GPS == 4 && !DUMP && !TAIL) {
            constexpr int NIT = NF * NJ;
            i32x16 dd[2];
            auto issue = [&](auto T) __attribute__((always_inline)) {
                constexpr int t = decltype(T)::value;
                constexpr int f = t / NJ, j = t % NJ, gi = f / MI;
                dd[t & 1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bw[j][gi], af[f & 1][0], start, 0, 0, 0);
            };
            issue(std::integral_constant<int, 0>());
            static_for<0, NIT>([&](auto T) __attribute__((always_inline)) {
                constexpr int t = decltype(T)::value;
                constexpr int f = t / NJ, j = t % NJ, gi = f / MI, i = f % MI;
                if constexpr (j == 0) {
                    if constexpr (f + 1 < NF) read_f(f + 1, af[(f + 1) & 1]);
                    if constexpr (i == 0) {
#pragma unroll
                        for (int jj = 0; jj < NJ; ++jj) read_sw(buf, jj, swh[jj], gi);
                    }
                }
                if constexpr (t + 1 < NIT) issue(std::integral_constant<int, t + 1>());
                dequant(dd[t & 1], acc[i][j], read_sa(buf, i, gi), swh[j]);
            });
        } else {
            static_for<0, NF>([&](auto F) __attribute__((always_inline)) {
                constexpr int f = decltype(F)::value;
                constexpr int gi = f / MI, i = f % MI;
                if constexpr (f + 1 < NF) read_f(f + 1, af[(f + 1) & 1]);
                if constexpr (i == 0) {
#pragma unroll
                    for (int j = 0; j < NJ; ++j) read_sw(buf, j, swh[j], gi);
                }
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    i32x16 d = start;
#pragma unroll
                    for (int q = 0; q < KPG; ++q)
                        d = __builtin_amdgcn_mfma_i32_32x32x32_i8(bw[j][gi * KPG + q], af[f & 1][q], d, 0, 0, 0);
                    dump_block(d, i, j, ks * GPS + gi);
                    dequant(d, acc[i][j], read_sa(buf, i, gi), swh[j]);
                }
            });
        }
    };

    // End of a group for the persistent mode.
    auto finish_group = [&](int buf, int g) __attribute__((always_inline)) {
        if constexpr (MODE == kPersist) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                uint2 swh[4];
                read_sw(buf, j, swh);
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    dump_block(psum[i][j], i, j, g);
                    dequant(psum[i][j], acc[i][j], read_sa(buf, i), swh);
                }
            }
        }
        (void)buf;
        (void)g;
    };

    // ---- main loop over K.  Stage ks lives in LDS buffer ks & 1 and, until
    // then, in register slot ks % PF; step ks issues the loads of stage ks + PF
    // into the slot stage ks frees.  Loads past the last stage are clamped to it
    // (harmless re-reads), so the rotating body is branch-free.
    auto step = [&](int ks, auto BUF, auto SLOT) __attribute__((always_inline)) {
        constexpr int buf = decltype(BUF)::value;
        constexpr int sl = decltype(SLOT)::value;
        const int ahead = kbase + min(ks + PF, nks - 1);
        load_a(ahead, SLOT);
        if constexpr (FINE) {
            compute_fine(buf, ahead, kbase + ks, SLOT);
        } else if constexpr (ROTATE) {
            compute(buf, ahead, kbase + ks, std::true_type{}, SLOT);
        } else {
            // a K-group's stages start on a group boundary (nks is a multiple of spg)
            if ((ks % spg) == 0) compute(buf, ahead, kbase + ks, std::true_type{}, SLOT);
            else compute(buf, ahead, kbase + ks, std::false_type{}, SLOT);
            if (MODE != kChannel && (ks + 1) % spg == 0) finish_group(buf, (kbase + ks) / spg);
        }
        store_a(buf ^ 1, std::integral_constant<int, (sl + 1) % PF>{});
        __syncthreads();
    };
    static_for<0, PF>([&](auto S) __attribute__((always_inline)) {
        constexpr int s0 = decltype(S)::value;
        load_a(kbase + min(s0, nks - 1), S);
        load_w(kbase + min(s0, nks - 1), S);
    });
    store_a(0, std::integral_constant<int, 0>{});
    __syncthreads();
    constexpr int U = PF == 1 ? 2 : (PF % 2 == 0 ? PF : 2 * PF);  // steps per unrolled round: lcm(2, PF)
    int ks = 0;
    for (; ks + U <= nks; ks += U)
        static_for<0, U>([&](auto S) __attribute__((always_inline)) {
            constexpr int u = decltype(S)::value;
            step(ks + u, std::integral_constant<int, u & 1>{}, std::integral_constant<int, u % PF>{});
        });
    static_for<0, U - 1>([&](auto S) __attribute__((always_inline)) {
        constexpr int u = decltype(S)::value;
        if (ks + u < nks) step(ks + u, std::integral_constant<int, u & 1>{}, std::integral_constant<int, u % PF>{});
    });

    // ---- K-groups 1 .. KSPLIT-1 hand their partial tiles to group 0, which adds
    // them in group order (fp32 sums, or the exact int32 sums of kChannel)
    if constexpr (KSPLIT > 1) {
        __shared__ int32_t red[KSPLIT - 1][NT / 64][MI * NJ * 16][64];
        if (kg > 0) {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        if constexpr (MODE == kChannel) red[kg - 1][wave][(i * NJ + j) * 16 + r][lane] = psum[i][j][r];
                        else red[kg - 1][wave][(i * NJ + j) * 16 + r][lane] = __float_as_int(acc[i][j][r]);
                    }
        }
        __syncthreads();
        if (kg > 0) return;  // after the workgroup's last barrier
#pragma unroll
        for (int k2 = 0; k2 < KSPLIT - 1; ++k2)
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int32_t v = red[k2][wave][(i * NJ + j) * 16 + r][lane];
                        if constexpr (MODE == kChannel) psum[i][j][r] += v;
                        else acc[i][j][r] += __int_as_float(v);
                    }
    }

    if constexpr (MODE == kChannel) {
        if (!part) {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j) dump_block(psum[i][j], i, j, 0);
        }
    }
    if (!have_sc) return;  // group sums only

    // ---- epilogue: lane holds row m and columns 8q + 4h + (0..3), q = 0..3.
    // The last step stored a copy of the final stage (and its scales) into the
    // buffer it did not read, so either buffer holds the final scales.
    const int lastbuf = nks & 1;
    if (part) {
        // split-K: this workgroup's partial tile, fp32 (exact int32 sums for
        // kChannel), to plane blockIdx.y of part[S][M][N]
        int32_t* pbase = static_cast<int32_t*>(part) + static_cast<int64_t>(blockIdx.y) * M * N;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int gm = m0 + wm * MI * 32 + i * 32 + l32;
            if (gm >= M) continue;
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    int32_t v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if constexpr (MODE == kChannel) v[e] = psum[i][j][4 * q + e];
                        else v[e] = __float_as_int(acc[i][j][4 * q + e]);
                    }
                    const int gn = n0 + wn * NJ * 32 + j * 32 + 8 * q + 4 * lh;
                    int32_t* dst = pbase + static_cast<int64_t>(gm) * N + gn;
                    if ((N & 3) == 0 && gn + 3 < N) {
                        *reinterpret_cast<int4*>(dst) = make_int4(v[0], v[1], v[2], v[3]);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (gn + e < N) dst[e] = v[e];
                    }
                }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int gm = m0 + wm * MI * 32 + i * 32 + l32;
        float sav = 0.f;
        if constexpr (MODE == kChannel) sav = read_sa(lastbuf, i);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            uint2 swh[4];
            if constexpr (MODE == kChannel) read_sw(lastbuf, j, swh);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = 4 * q + e;
                    if constexpr (MODE == kChannel) v[e] = static_cast<float>(psum[i][j][r]) * sav * h2f(sw_at(swh, r));
                    else v[e] = acc[i][j][r];
                }
                const uint32_t h01 = __half_as_ushort(__float2half_rn(v[0])) |
                                     (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(v[1]))) << 16);
                const uint32_t h23 = __half_as_ushort(__float2half_rn(v[2])) |
                                     (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(v[3]))) << 16);
                const int gn = n0 + wn * NJ * 32 + j * 32 + 8 * q + 4 * lh;
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
}

// G = 128 (and 256) on 128 x 256 tiles with a ping-pong schedule.
//
// Each SIMD runs one wave of group X (waves 0-3) and one of group Y (waves
// 4-7), which own the same 128 x 32 outputs per wave as the kernel above.  A
// wave's stage has an MFMA phase (widen its weights, 16 v_mfma into four
// group-sum blocks) and a dequant phase (the 4 x 16 elements of those blocks,
// 2 VALU ops each).  The groups run them half a stage apart, separated by
// workgroup barriers:
//     slot 2s:    X: MFMA phase of stage s     Y: dequant of stage s-1
//     slot 2s+1:  X: dequant of stage s        Y: MFMA phase of stage s
// (the same loop body for both groups, Y one slot behind)
// so in every slot one wave of each SIMD issues MFMAs while the other issues
// VALU work, and the SIMD can run both at once.  The group sums, scales and
// the order in which groups are added are those of the kernel above, so the
// results are the same bits.
//   * A (widened) and the stage's scales are double-buffered in LDS; stage s
//     sits in buffer s & 1.  X's threads stage rows 0-63 of A and scale slots
//     0-255, Y's threads rows 64-127 and slots 256-511, each in its own
//     dequant slot: X writes stage s+1 in slot 2s+1, Y in slot 2s.  Neither
//     buffer is written while it is read (buffer s & 1 is read in slots 2s and
//     2s+1 and next written in slots 2s+2 and 2s+3).
//   * A wave reads its stage's scales in its MFMA phase, so its dequant phase
//     only touches registers.
//   * A thread's next global loads are issued as soon as their registers are
//     free: weights of stage s + 1 right after stage s's are widened, its A
//     chunk of stage s + 2 right after stage s + 1's is stored (two slots of
//     cover each).
//   * SPG: stages per group (1 for G = 128, 2 for G = 256).  The group's
//     stages accumulate into the same sums from the bias (|256 P| <= 2^22 at
//     G = 256, so the bias still converts exactly); only its last stage reads
//     the scales and has a dequant phase, which is skipped in the others, as
//     the kernel above does in its persistent mode.
//   * DUMP: the group sums of rows [pm0, pm0 + pmr) also go to P[pmr][N][K/G]
//     in the dequant phase (sa == nullptr: no scales read, no Y written).
template <bool DUMP, int SPG>
__global__ __launch_bounds__(512, 1) void w4a4_gemm_pp_kernel(
    const uint8_t* __restrict__ Aq, const uint16_t* __restrict__ sa, const uint8_t* __restrict__ Wq,
    const uint16_t* __restrict__ sw, int M, int N, int K, uint16_t* __restrict__ Y, int nks_split,
    float* __restrict__ part, int32_t* __restrict__ P, int pm0, int pmr, int wt) {
    constexpr int NT = 512, BM = 128, BN = 256, MI = 4;
    __shared__ Stage<BM, NT, 1> st[2];
    const bool have_sc = !DUMP || sa != nullptr;  // uniform

    // tile selection: as the kernel above
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
    const bool grp_y = wave >= 4;  // uniform per wave
    const int l32 = lane & 31, lh = lane >> 5;
    // K range: stages [kofs, kofs + nks) of this workgroup's split (blockIdx.y)
    const int nks = nks_split;
    const int kofs = static_cast<int>(blockIdx.y) * nks_split;
    const int ng = K / (KS * SPG);

    // this thread's 16-byte chunk of A per stage and its widened LDS places
    const int ar = tid >> 2, ap = tid & 3;
    const uint32_t a_off = static_cast<uint32_t>(min(m0 + ar, M - 1)) * static_cast<uint32_t>(K / 2) + ap * 16;
    const int c0 = 2 * (2 * (ap & 1)) + (ap >> 1);
    const int a_lds0 = ar * AROW + c0 * 16, a_lds1 = ar * AROW + (c0 + 2) * 16;
    // this thread's scale slot: an activation row, a weight column or a dummy
    const bool is_a = tid < BM;
    const int srow = is_a ? min(m0 + tid, M - 1) : min(n0 + min(tid - BM, BN - 1), N - 1);
    const uint16_t* sc_base = is_a ? sa : sw;
    const uint32_t sc_off = static_cast<uint32_t>(srow) * static_cast<uint32_t>(ng);
    // weights: row-major or tiled, as in the kernel above
    const uint32_t w_off =
        wt ? static_cast<uint32_t>(min(nt * 8 + wave, (N + 31) / 32 - 1)) * static_cast<uint32_t>(K / KS) * 2048u + 16u * lane
           : static_cast<uint32_t>(min(n0 + wave * 32 + l32, N - 1)) * static_cast<uint32_t>(K / 2) + 32 * lh;
    const int w_sstride = wt ? 2048 : KS / 2, w_jstride = wt ? 1024 : 16;

    uint4 ra;
    uint16_t rsc;
    uint4 w[2];
    auto load_a = [&](int ks) __attribute__((always_inline)) {
        ks = min(ks, nks - 1) + kofs;
        ra = *reinterpret_cast<const uint4*>(Aq + static_cast<int64_t>(ks) * (KS / 2) + a_off);
        rsc = have_sc ? sc_base[sc_off + static_cast<uint32_t>(ks / SPG)] : static_cast<uint16_t>(0);
    };
    auto store_a = [&](int buf) __attribute__((always_inline)) {
        *reinterpret_cast<i32x4*>(&st[buf].a[a_lds0]) = frag2(ra.x, ra.y);
        *reinterpret_cast<i32x4*>(&st[buf].a[a_lds1]) = frag2(ra.z, ra.w);
        st[buf].scale[0][tid] = rsc;
    };
    auto load_w = [&](int ks) __attribute__((always_inline)) {
        ks = min(ks, nks - 1) + kofs;
        const uint8_t* base = Wq + static_cast<int64_t>(ks) * w_sstride + w_off;
        w[0] = *reinterpret_cast<const uint4*>(base);
        w[1] = *reinterpret_cast<const uint4*>(base + w_jstride);
    };

    f32x16 acc[MI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
    i32x16 D[MI];
    uint2 swh[4];
    float sav[MI];
    const i32x16 start = splat16(static_cast<int>(MAGIC_BITS));

    // MFMA phase of stage s (LDS buffer and register slot s & 1)
    auto mfma_phase = [&](int s, int par, auto FIRST, auto LAST) __attribute__((always_inline)) {
        constexpr bool first = decltype(FIRST)::value, last = decltype(LAST)::value;
        const int c = BM + wave * 32 + 4 * lh;
        if constexpr (last) {
#pragma unroll
            for (int q = 0; q < 4; ++q) swh[q] = *reinterpret_cast<const uint2*>(&st[par].scale[0][c + 8 * q]);
#pragma unroll
            for (int i = 0; i < MI; ++i) sav[i] = h2f(st[par].scale[0][i * 32 + l32]) * (1.0f / 256.0f);
        }
        i32x4 bw[KK];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const uint4& v = w[kk >> 1];
            bw[kk] = (kk & 1) ? frag2(v.z, v.w) : frag2(v.x, v.y);
        }
        __builtin_amdgcn_sched_barrier(0);
        load_w(s + 1);
        __builtin_amdgcn_sched_barrier(0);
        // the four blocks' chains interleaved, MFMA n = (kk = n / 4, i = n % 4)
        // needs (i, kk - 1) only, four MFMAs earlier; A fragments are read LA
        // MFMAs ahead into a ring of LA + 1
        constexpr int LA = 4;
        i32x4 af[LA + 1];
        auto frag = [&](int n) __attribute__((always_inline)) {
            const int kk = n >> 2, i = n & 3;
            return *reinterpret_cast<const i32x4*>(&st[par].a[(i * 32 + l32) * AROW + (2 * kk + lh) * 16]);
        };
        static_for<0, LA>([&](auto NN) __attribute__((always_inline)) { af[decltype(NN)::value] = frag(decltype(NN)::value); });
        static_for<0, 4 * MI>([&](auto NN) __attribute__((always_inline)) {
            constexpr int n = decltype(NN)::value;
            if constexpr (n + LA < 4 * MI) af[(n + LA) % (LA + 1)] = frag(n + LA);
            constexpr int kk = n >> 2, i = n & 3;
            D[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bw[kk], af[n % (LA + 1)], (kk == 0 && first) ? start : D[i], 0, 0, 0);
        });
        // keep that order: LA fragment reads, then MFMA / next read pairs
        __builtin_amdgcn_sched_group_barrier(0x100, LA, 0);
        static_for<0, 4 * MI - LA>([&](auto) __attribute__((always_inline)) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        });
        __builtin_amdgcn_sched_group_barrier(0x008, LA, 0);
    };
    // acc += fl(P s_a) * s_w for the four blocks of the last MFMA phase (stage s)
    auto dequant_phase = [&](int s) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < MI; ++i) asm volatile("" : "+v"(D[i]));
        if constexpr (DUMP) {
            const int g = (kofs + s) / SPG;
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                const int gm = m0 + i * 32 + l32;
                if (gm >= pm0 && gm < pm0 + pmr) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int gn = n0 + wave * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
                        if (gn < N) P[(static_cast<int64_t>(gm - pm0) * N + gn) * ng + g] = (D[i][r] - static_cast<int>(MAGIC_BITS)) >> 8;
                    }
                }
            }
        }
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const float nb = -MAGIC * sav[i];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint32_t pair = (r & 2) ? swh[r >> 2].y : swh[r >> 2].x;
                const uint16_t hw = (r & 1) ? static_cast<uint16_t>(pair >> 16) : static_cast<uint16_t>(pair & 0xFFFFu);
                const float t = fmaf(__int_as_float(D[i][r]), sav[i], nb);
                acc[i][r] = fmaf(t, h2f(hw), acc[i][r]);
            }
        }
    };
    // this thread's part of stage t (in its registers) into LDS, then the
    // loads of stage t + 1
    auto stage_next = [&](int t) __attribute__((always_inline)) {
        store_a(t & 1);
        load_a(t + 1);
    };

    // prologue: stage 0 in LDS buffer 0 (every thread), stage 1 in registers
    load_w(0);
    load_a(0);
    store_a(0);
    load_a(1);
    __syncthreads();

    // Both groups run the same loop body, Y one slot behind X: Y spends slot 0
    // staging its half of stage 1, and X ends with one barrier more, so the
    // barrier counts match.  In its dequant slot of stage s, X stages its half
    // of stage s + 1 and Y its half of stage s + 2.  The compiler keeps each
    // phase between its barriers (no code motion across them).
    if (grp_y) {
        stage_next(1);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
    }
    const int ahead = grp_y ? 2 : 1;
    // The empty asm statements make the MFMA results and the accumulators
    // opaque at the barriers, so that no MFMA or dequant work is sunk past the
    // barrier that ends its phase (or hoisted above the one that starts it).
    auto pin = [](auto& v) __attribute__((always_inline)) { asm volatile("" : "+v"(v)); };
    for (int s = 0; s < nks; ++s) {
        // a group's stages accumulate into D from the bias; the group's last
        // stage reads its scales and is dequantized
        if constexpr (SPG == 1) {
            mfma_phase(s, s & 1, std::true_type(), std::true_type());
        } else {
            if (s % SPG == 0) mfma_phase(s, s & 1, std::true_type(), std::false_type());
            else mfma_phase(s, s & 1, std::false_type(), std::true_type());
        }
#pragma unroll
        for (int i = 0; i < MI; ++i) pin(D[i]);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        if (SPG == 1 || s % SPG == SPG - 1) dequant_phase(s);
#pragma unroll
        for (int i = 0; i < MI; ++i) pin(acc[i]);
        stage_next(s + ahead);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
    }
    if (!grp_y) __syncthreads();
    if (!have_sc) return;  // group sums only

    // epilogue: lane holds row m and columns 8q + 4h + (0..3), q = 0..3.
    // Split K: the fp32 partial tile goes to part[split][m][n] instead.
    if (part) {
        float* pbase = part + static_cast<int64_t>(blockIdx.y) * M * N;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int gm = m0 + i * 32 + l32;
            if (gm >= M) continue;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int gn = n0 + wave * 32 + 8 * q + 4 * lh;
                float* dst = pbase + static_cast<int64_t>(gm) * N + gn;
                if ((N & 3) == 0 && gn + 3 < N) {
                    *reinterpret_cast<float4*>(dst) =
                        make_float4(acc[i][4 * q], acc[i][4 * q + 1], acc[i][4 * q + 2], acc[i][4 * q + 3]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (gn + e < N) dst[e] = acc[i][4 * q + e];
                }
            }
        }
        return;
    }
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

template <int WAVES_M, int WAVES_N, int MI, int NJ, int MODE, bool MAGIC_OK, int GPS, int KSPLIT, bool DUMP>
hipError_t launch_k(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                    int64_t N, int64_t K, int64_t G, uint16_t* Y, Dump dump, bool wt, hipStream_t stream, int S = 1,
                    void* part = nullptr) {
    // a partial last stage only happens with groups finer than a stage or one group per row
    constexpr bool can_tail = GPS > 1 || MODE == kChannel;
    constexpr int BM = WAVES_M * MI * 32, BN = WAVES_N * NJ * 32;
    const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    if (tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    // Small tiles (one wave per SIMD) have little compute per stage to hide a
    // load behind: their loads run 4 stages ahead (measured 4-7 % faster at
    // M = 64..256, N = 8192 for G in {128, 256}, 24 % for G = K).  With G < 128
    // the deeper ring costs occupancy and time, so those keep one stage.
    constexpr int PF = (WAVES_M * WAVES_N * MI * NJ <= 8 && GPS == 1) ? 4 : 1;
    const dim3 grid(static_cast<unsigned>(tiles), static_cast<unsigned>(S)), block(64 * WAVES_M * WAVES_N * KSPLIT);
    const int m = static_cast<int>(M), n = static_cast<int>(N), k = static_cast<int>(K), g = static_cast<int>(G);
    const int nks = static_cast<int>(kstages(K) / S), w = wt ? 1 : 0;
    if (K % KS != 0) {
        if constexpr (can_tail)
            hipLaunchKernelGGL((w4a4_gemm_kernel<WAVES_M, WAVES_N, MI, NJ, MODE, MAGIC_OK, GPS, PF, KSPLIT, DUMP, true>),
                               grid, block, 0, stream, Aq, sa, Wq, sw, m, n, k, g, Y, dump.P, dump.m0, dump.mr, nks, part,
                               w);
        else
            return hipErrorInvalidValue;
    } else {
        hipLaunchKernelGGL((w4a4_gemm_kernel<WAVES_M, WAVES_N, MI, NJ, MODE, MAGIC_OK, GPS, PF, KSPLIT, DUMP, false>),
                           grid, block, 0, stream, Aq, sa, Wq, sw, m, n, k, g, Y, dump.P, dump.m0, dump.mr, nks, part, w);
    }
    return hipGetLastError();
}

// Small tiles (one wave per SIMD) split K over two wave groups when every CU
// gets at most one tile and the halves start on group boundaries: two waves
// per SIMD, half the stages each (MI355X, M = 256, N = 8192: 10 % faster at
// G = 128, 21 % at G = 256, 11 % at G = K, 28-40 % at G = 32).  With more
// tiles than CUs the 8-wave workgroups fit once per CU where the 4-wave ones
// fit twice, and the split loses (N = 10240: 9 % slower).
template <int WAVES_M, int WAVES_N, int MI, int NJ, int MODE, bool MAGIC_OK, int GPS = 1>
hipError_t launch(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                  int64_t N, int64_t K, int64_t G, uint16_t* Y, Dump dump, bool wt, hipStream_t stream, int S = 1,
                  void* part = nullptr) {
    constexpr bool small = WAVES_M * WAVES_N * MI * NJ <= 8;
    int ksplit = 1;
    if constexpr (small) {
        constexpr int BM = WAVES_M * MI * 32, BN = WAVES_N * NJ * 32;
        const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
        const int64_t stages = kstages(K);
        const int64_t spg = (MODE == kChannel || GPS > 1) ? 1 : G / KS;
        if (S == 1 && tiles <= device_cu_count() && stages % 2 == 0 && (stages / 2) % spg == 0) ksplit = 2;
    }
    // S > 1: split across workgroups, one wave group per workgroup
    if (dump.P) {
        if constexpr (small) {
            if (ksplit == 2)
                return launch_k<WAVES_M, WAVES_N, MI, NJ, MODE, MAGIC_OK, GPS, 2, true>(Aq, sa, Wq, sw, M, N, K, G, Y,
                                                                                        dump, wt, stream);
        }
        return launch_k<WAVES_M, WAVES_N, MI, NJ, MODE, MAGIC_OK, GPS, 1, true>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt,
                                                                                stream, S, part);
    }
    if constexpr (small) {
        if (ksplit == 2)
            return launch_k<WAVES_M, WAVES_N, MI, NJ, MODE, MAGIC_OK, GPS, 2, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump,
                                                                                     wt, stream);
    }
    return launch_k<WAVES_M, WAVES_N, MI, NJ, MODE, MAGIC_OK, GPS, 1, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt,
                                                                             stream, S, part);
}

// The ping-pong kernel on 128 x 256 tiles, SPG stages per group (S > 1, for
// G = 128 only: split over K, fp32 partial tiles to part).
template <int SPG>
hipError_t launch_pp(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                     int64_t N, int64_t K, uint16_t* Y, Dump dump, bool wt, hipStream_t stream, int S = 1,
                     float* part = nullptr) {
    const int64_t tiles = ((M + 127) / 128) * ((N + 255) / 256);
    if (tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(tiles), static_cast<unsigned>(S));
    const int m = static_cast<int>(M), n = static_cast<int>(N), k = static_cast<int>(K), nks = static_cast<int>(K / KS / S);
    if (dump.P)
        hipLaunchKernelGGL((w4a4_gemm_pp_kernel<true, SPG>), grid, dim3(512), 0, stream, Aq, sa, Wq, sw, m, n, k, Y, nks, part,
                           dump.P, dump.m0, dump.mr, wt ? 1 : 0);
    else
        hipLaunchKernelGGL((w4a4_gemm_pp_kernel<false, SPG>), grid, dim3(512), 0, stream, Aq, sa, Wq, sw, m, n, k, Y, nks, part,
                           static_cast<int32_t*>(nullptr), 0, 0, wt ? 1 : 0);
    return hipGetLastError();
}

}  // namespace

// Tile: 128 x 256 per workgroup, 8 waves (two per SIMD) of 128 x 32.  When that
// tiling would not give every CU a workgroup, 64 x 128 tiles with 4 waves of
// 64 x 32 (four times as many workgroups, two per CU), or 8 waves splitting K
// (see launch).  G = 128 (and G = 256 unsplit) on 128 x 256 tiles is the
// ping-pong kernel unless force_general.
template <int WAVES_N, int MI>
hipError_t launch_tiles(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw, int64_t M,
                        int64_t N, int64_t K, int64_t G, uint16_t* Y, Dump dump, bool wt, hipStream_t stream, int S = 1,
                        void* part = nullptr, bool force_general = false) {
    if (G == K) return launch<1, WAVES_N, MI, 1, kChannel, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, S, part);
    if (G == 32) return launch<1, WAVES_N, MI, 1, kRotate, true, 4>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, S, part);
    if (G == 64) return launch<1, WAVES_N, MI, 1, kRotate, true, 2>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, S, part);
    if (G == 128) {
        if constexpr (WAVES_N == 8 && MI == 4) {
            if (!force_general)
                return launch_pp<1>(Aq, sa, Wq, sw, M, N, K, Y, dump, wt, stream, S, static_cast<float*>(part));
        }
        return launch<1, WAVES_N, MI, 1, kRotate, true>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, S, part);
    }
    if (G == 256) {
        if constexpr (WAVES_N == 8 && MI == 4) {
            if (!force_general && S == 1)
                return launch_pp<2>(Aq, sa, Wq, sw, M, N, K, Y, dump, wt, stream, 1, nullptr);
        }
        return launch<1, WAVES_N, MI, 1, kPersist, true>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, S, part);
    }
    return launch<1, WAVES_N, MI, 1, kPersist, false>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, S, part);
}

namespace {

// Y = binary16(part[0] + part[1] + ... + part[S-1]), summed in split order:
// four elements per thread when M N is a multiple of 4 (16-byte aligned
// partial planes), one otherwise.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int S, int64_t MN,
                                                            uint16_t* __restrict__ Y) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    if ((MN & 3) == 0) {
        for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < MN / 4; i += stride) {
            float4 a = reinterpret_cast<const float4*>(part)[i];
            for (int sp = 1; sp < S; ++sp) {
                const float4 b = reinterpret_cast<const float4*>(part + sp * MN)[i];
                a.x += b.x;
                a.y += b.y;
                a.z += b.z;
                a.w += b.w;
            }
            const uint32_t lo = __half_as_ushort(__float2half_rn(a.x)) |
                                (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(a.y))) << 16);
            const uint32_t hi = __half_as_ushort(__float2half_rn(a.z)) |
                                (static_cast<uint32_t>(__half_as_ushort(__float2half_rn(a.w))) << 16);
            reinterpret_cast<uint2*>(Y)[i] = make_uint2(lo, hi);
        }
    } else {
        for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < MN; i += stride) {
            float a = part[i];
            for (int sp = 1; sp < S; ++sp) a += part[sp * MN + i];
            Y[i] = __half_as_ushort(__float2half_rn(a));
        }
    }
}

// Per-channel split-K: the S planes hold exact int32 sums of 256 P; their sum
// is scaled exactly as the per-channel epilogue does, so Y is the same bits as
// without the split.
// With a dump, the exact per-channel group sum (P = the planes' sum / 256) of
// rows [pm0, pm0 + pmr) also goes to P[pmr][N].
__global__ __launch_bounds__(256) void splitk_reduce_channel_kernel(const int32_t* __restrict__ part, int S, int M,
                                                                    int N, const uint16_t* __restrict__ sa,
                                                                    const uint16_t* __restrict__ sw,
                                                                    uint16_t* __restrict__ Y, int32_t* __restrict__ P,
                                                                    int pm0, int pmr) {
    const int64_t MN = static_cast<int64_t>(M) * N;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < MN; i += stride) {
        int32_t p = part[i];
        for (int sp = 1; sp < S; ++sp) p += part[sp * MN + i];
        const int64_t m = i / N, n = i - m * N;
        if (P && m >= pm0 && m < pm0 + pmr) P[(m - pm0) * N + n] = p >> 8;
        const float sav = h2f(sa[m]) * (1.0f / 256.0f);
        const float v = static_cast<float>(p) * sav * h2f(sw[n]);
        Y[i] = __half_as_ushort(__float2half_rn(v));
    }
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

}  // namespace

// Split factor over K when the tiles leave CUs idle; 1 where no split applies.
//   * G = 128: the ping-pong kernel's 128 x 256 tiles, the largest S in
//     {2, 4, 8} with tiles * S <= CUs, S dividing the stage count and at least
//     4 stages per split.  S = 2 is taken only from M = 256 on: below that the
//     128-row tiles are half empty and the 64 x 128 tiles of launch_gemm,
//     which already fill the CUs, were faster (MI355X, M = 64, N = 28672,
//     K = 8192: 39.5 us against 49.6 us split).
//   * Other G: the 64 x 128 tiles of four waves (two workgroups per CU), when
//     they fill at most half the CUs (above that the in-workgroup K split of
//     launch already gives every SIMD two waves): the largest S with
//     tiles * S <= 2 CUs, splits starting on group boundaries, at least 4
//     stages each.
int splitk_factor(int64_t M, int64_t N, int64_t K, int64_t G) {
    if (M <= 0 || gemv_fits(M, N, K, G) || decode_fits(M, N, K, G)) return 1;
    const int64_t cus = device_cu_count();
    const int64_t nks = kstages(K);
    if (((M + 127) / 128) * ((N + 255) / 256) >= cus) return 1;
    int S = 1;
    if (G == 128) {
        const int64_t tiles = ((M + 127) / 128) * ((N + 255) / 256);
        for (int c = 2; c <= 8; c *= 2)
            if (tiles * c <= cus && nks % c == 0 && nks / c >= 4) S = c;
        return (S == 2 && M < 256) ? 1 : S;
    }
    const int64_t tiles = ((M + 63) / 64) * ((N + 127) / 128);
    if (2 * tiles > cus) return 1;
    const int64_t spg = (G == K || G <= KS) ? 1 : G / KS;
    for (int c = 2; c <= 8; c *= 2)
        if (tiles * c <= 2 * cus && nks % c == 0 && (nks / c) % spg == 0 && nks / c >= 4) S = c;
    return S;
}

int64_t splitk_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t G) {
    // few rows: the stream-K form of the few-row kernel where it applies
    if (M > 0 && !gemv_fits(M, N, K, G) && decode_fits(M, N, K, G)) return decode_split_workspace_bytes(M, N, K, G);
    const int S = splitk_factor(M, N, K, G);
    return S > 1 ? static_cast<int64_t>(S) * M * N * 4 : 0;
}

hipError_t launch_splitk_reduce(const float* part, int S, int64_t MN, uint16_t* Y, hipStream_t stream) {
    const int64_t items = (MN & 3) == 0 ? MN / 4 : MN;
    const int64_t need = (items + 255) / 256;
    const int blocks = static_cast<int>(need < 8192 ? need : 8192);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, stream, part, S, MN, Y);
    return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t need = (n + 255) / 256;
    const int blocks = static_cast<int>(need < 8192 ? need : 8192);
    hipLaunchKernelGGL(fill_i32_kernel, dim3(blocks), dim3(256), 0, stream, p, n, v);
    return hipGetLastError();
}

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int64_t G, bool split, bool force_tile, bool wt) {
    if (split) {
        const int S = splitk_factor(M, N, K, G);
        if (S > 1) return {G == 128 && !force_tile ? kKernelPingPong : kKernelTile64, S};
    }
    if (!force_tile && gemv_fits(M, N, K, G, wt)) return {kKernelGemv, 1};
    if (!force_tile && decode_fits(M, N, K, G))
        return {split && decode_split_workspace_bytes(M, N, K, G) > 0 ? kKernelDecodeSplit : kKernelDecode, 1};
    const int64_t big_tiles = ((M + 127) / 128) * ((N + 255) / 256);
    if (big_tiles < device_cu_count()) return {kKernelTile64, 1};
    return {(G == 128 || G == 256) && !force_tile ? kKernelPingPong : kKernelTile128, 1};
}

namespace {

hipError_t launch_planned(const GemmPlan& plan, const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                          const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y,
                          hipStream_t stream, Dump dump, float* part, bool wt) {
    switch (plan.kernel) {
        case kKernelGemv: return launch_gemv(Aq, sa, Wq, sw, M, N, K, G, Y, stream, dump, wt);
        case kKernelDecode: return launch_gemm_decode(Aq, sa, Wq, sw, M, N, K, G, Y, stream, dump, wt);
        case kKernelDecodeSplit: return launch_gemm_decode(Aq, sa, Wq, sw, M, N, K, G, Y, stream, dump, wt, part);
        case kKernelTile64:
            return launch_tiles<4, 2>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, plan.splits, part);
        case kKernelTile128:
            return launch_tiles<8, 4>(Aq, sa, Wq, sw, M, N, K, G, Y, dump, wt, stream, 1, nullptr, /*force_general=*/true);
        case kKernelPingPong:
            return G == 256 ? launch_pp<2>(Aq, sa, Wq, sw, M, N, K, Y, dump, wt, stream, plan.splits, part)
                            : launch_pp<1>(Aq, sa, Wq, sw, M, N, K, Y, dump, wt, stream, plan.splits, part);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_gemm_splitk(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw,
                              int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, float* part,
                              hipStream_t stream, Dump dump, bool force_tile, bool wt) {
    const GemmPlan plan = plan_gemm(M, N, K, G, true, force_tile, wt);
    if (plan.kernel == kKernelDecodeSplit)  // the workspace holds the stream-K counters and parts
        return launch_planned(plan, Aq, sa, Wq, sw, M, N, K, G, Y, stream, dump, part, wt);
    if (plan.splits < 2) return launch_planned(plan, Aq, sa, Wq, sw, M, N, K, G, Y, stream, dump, nullptr, wt);
    const int S = plan.splits;
    // split ranges hold whole groups, so every group sum except the
    // per-channel one is dumped by the kernel that completes it
    Dump tile_dump = dump;
    if (G == K) tile_dump.P = nullptr;
    const hipError_t e = launch_planned(plan, Aq, sa, Wq, sw, M, N, K, G, Y, stream, tile_dump, part, wt);
    if (e != hipSuccess) return e;
    if (G == K) {
        const int64_t need = (M * N + 255) / 256;
        const int blocks = static_cast<int>(need < 8192 ? need : 8192);
        hipLaunchKernelGGL(splitk_reduce_channel_kernel, dim3(blocks), dim3(256), 0, stream,
                           reinterpret_cast<const int32_t*>(part), S, static_cast<int>(M), static_cast<int>(N), sa, sw,
                           Y, dump.P, dump.m0, dump.mr);
        return hipGetLastError();
    }
    return launch_splitk_reduce(part, S, M * N, Y, stream);
}

// One row (two on tiled weights): the dot-product kernel; up to 32 rows: the
// weight-streaming kernel; otherwise the tile kernels (the same choice with or
// without a dump).
hipError_t launch_gemm(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq, const uint16_t* sw,
                       int64_t M, int64_t N, int64_t K, int64_t G, uint16_t* Y, hipStream_t stream, Dump dump,
                       bool force_tile, bool wt) {
    return launch_planned(plan_gemm(M, N, K, G, false, force_tile, wt), Aq, sa, Wq, sw, M, N, K, G, Y, stream, dump,
                          nullptr, wt);
}

}  // namespace apex4
