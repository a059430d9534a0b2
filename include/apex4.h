/*
 * apex4.h -- C ABI of the MI355X (gfx950) W4A4 group-quantized GEMM library.
 *
 * Method: APEX4, "Efficient Pure W4A4 LLM Inference via Intra-SM Compute
 * Rebalancing" (arXiv 2606.08761).
 *
 * Data formats (shared by every entry point):
 *   - binary16 buffers are passed as void* and hold IEEE 754 binary16 bit
 *     patterns (torch.float16);
 *   - packed 4-bit codes are uint8 [rows, K/2], row-major, two signed codes in
 *     [-8, 7] per byte along K, low nibble = even k (Sec. 4.4 stores activations
 *     and weights as packed 4-bit vectors; this library packs both along K);
 *   - scales are binary16 [rows, K/G], row-major: one per row and K-group
 *     (Sec. 4.4: S1 for activations, S2 for weights, both FP16);
 *   - Y = A W^T: A_q is [M, K/2], W_q is [N, K/2] (nn.Linear layout), Y is
 *     binary16 [M, N], row-major.
 *
 * Ownership and execution: every pointer is caller-owned device memory.  The
 * library never allocates, frees, synchronises or keeps a pointer past the
 * call.  Outputs are fully overwritten; inputs and outputs must not alias.
 * Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and is
 * complete once that stream is synchronised.  Calls are reentrant.
 *
 * Errors: every entry point returns an apex4_status and never prints or
 * aborts.  Arguments are validated before any HIP call, in this order:
 * NULL pointers, shapes, group size, alignment, device; M == 0 is a
 * successful no-op (after validation), and buffers whose size is zero
 * (M-sized when M == 0, the group-sum dump when mr == 0) may be NULL.  A failed launch returns
 * APEX4_ERR_LAUNCH.  Nothing is written when validation fails.
 *
 * Shape rules (4-bit code entry points):  M >= 0, N >= 1, K >= 32 and
 * K % 32 == 0, K % G == 0; each packed operand of the GEMM entry points under
 * 4 GiB (M K/2 and N K/2 below 2^32 bytes).  The FP6 and MX entry points keep
 * K >= 128 and K % 128 == 0.
 * Group sizes: the GEMM takes G in {32, 64, 128, 256, 512, 1024} or G == K
 * (per-channel, K <= 65536: the kernels keep 256 times the row's integer sum,
 * up to 2^14 K in magnitude, in one int32); these are the granularities of
 * Sec. 3.2.2 and Sec. 4.1.  The quantizer takes any G with G % 32 == 0 and
 * K % G == 0.
 * Alignment: every pointer 16-byte aligned.
 * Device: the current device must be gfx950 (MI355X / MI350X).
 */
#ifndef APEX4_H
#define APEX4_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    APEX4_OK = 0,
    APEX4_ERR_NULL = -1,    /* a required pointer is NULL */
    APEX4_ERR_SHAPE = -2,   /* M, N, K or a row window out of range */
    APEX4_ERR_GROUP = -3,   /* unsupported group size G */
    APEX4_ERR_ALIGN = -4,   /* a pointer is not 16-byte aligned */
    APEX4_ERR_LAUNCH = -5,  /* the HIP launch failed */
    APEX4_ERR_DEVICE = -6,  /* no device, or the current device is not gfx950 */
    APEX4_ERR_WORKSPACE = -7 /* workspace NULL or smaller than the size query returns */
} apex4_status;

/*
 * Per-token, per-group activation quantizer (SymQuant with b = 4).
 * Sec. 3.2.1, Eq. (SymQuant): S_g = max|X_g| / 7, X_g^q = clamp(round(X_g/S_g), -8, 7);
 * applied online to activations (Sec. 4.4) and offline to weights (Alg. 1).
 *
 *   x    [M, K] binary16 input (device).
 *   A_q  [M, K/2] packed codes (device, output).
 *   s_a  [M, K/G] binary16 scales (device, output).
 *
 * Per (row, group): amax = max|x|; S = the binary16 nearest to amax/7 (ties to
 * even); codes = clamp(round-half-even(x / S), -8, 7), taken on the exact
 * quotient; a group whose S is zero gets zero codes.  Bit-exact and
 * deterministic.  The same call quantizes weights ([N, K] -> W_q, s_w).
 */
int apex4_quantize_act(const void* x, int64_t M, int64_t K, int64_t G,
                       uint8_t* A_q, void* s_a, void* stream);

/*
 * Pure W4A4 group-quantized GEMM.
 * Sec. 3.2.1, Eq. (group_decomposition): C = sum_g (A_g^q W_g^q) (.) (S_g^a S_g^w^T);
 * Sec. 4.2: immediate per-group dequantization (groups) and delayed
 * dequantization (per-channel, G == K).
 *
 *   A_q [M, K/2] codes, s_a [M, K/G] scales, W_q [N, K/2] codes, s_w [N, K/G]
 *   scales (all device, read-only);  Y [M, N] binary16 (device, output).
 *
 *   Y[m,n] = binary16( sum_g s_a[m,g] s_w[n,g] P[m,n,g] ),
 *   P[m,n,g] = sum_{k in g} A_q[m,k] W_q[n,k]  (exact 32-bit integer sums).
 * The scaled sum is accumulated in binary32; the result is rounded once to
 * binary16 (round to nearest even).
 */
int apex4_w4a4_gemm(const uint8_t* A_q, const void* s_a,
                    const uint8_t* W_q, const void* s_w,
                    int64_t M, int64_t N, int64_t K, int64_t G,
                    void* Y, void* stream);

/*
 * apex4_w4a4_gemm_ws without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same kernels and the same Y, bit for bit,
 * as apex4_w4a4_gemm_ws; where that call would split K (the partial planes)
 * or take the few-row kernel's stream-K form (its counters and parts), the
 * workspace is a static device array of APEX4_NOALLOC_SCRATCH_BYTES that the
 * library holds on each device it runs on until the process ends.  The call
 * itself allocates nothing (no hipMalloc / hipFree).
 *
 *   Arguments and errors as apex4_w4a4_gemm, plus APEX4_ERR_WORKSPACE when the
 *   shape's split would need more than APEX4_NOALLOC_SCRATCH_BYTES (the size
 *   query apex4_w4a4_gemm_workspace_size returns that need; on a 256-CU
 *   MI355X every split fits).
 *   All calls on one device share its array: calls that may overlap on one
 *   device (different streams, or host threads) race and must be ordered by
 *   the caller.  The caller clears nothing: the stream-K counters are set to
 *   zero by a fill kernel at the start of every call that uses them, and
 *   every other byte a call reads it has written first.
 */
#define APEX4_NOALLOC_SCRATCH_BYTES (32ll << 20)
int apex4_w4a4_gemm_noalloc(const uint8_t* A_q, const void* s_a,
                            const uint8_t* W_q, const void* s_w,
                            int64_t M, int64_t N, int64_t K, int64_t G,
                            void* Y, void* stream);

/*
 * Debug form of apex4_w4a4_gemm: the exact integer group sums of Eq.
 * (group_decomposition).  The whole M x N problem runs through the kernel
 * that apex4_w4a4_gemm picks for this shape (one-row, few-row or tile kernel),
 * in its dump form with the scales and Y left out; only the window's sums are
 * written.
 *
 *   P [mr, N, K/G] int32 (device, output): P[i, n, g] for rows m0 + i,
 *   0 <= m0, 0 <= mr, m0 + mr <= M; may be NULL when mr == 0.
 */
int apex4_w4a4_gemm_groupsums(const uint8_t* A_q, const uint8_t* W_q,
                              int64_t M, int64_t N, int64_t K, int64_t G,
                              int64_t m0, int64_t mr, int32_t* P, void* stream);

/* flags of apex4_w4a4_gemm_debug (and of apex4_w4a4_gemm_plan, apex4_w4a4_linear_debug,
   apex4_w4a4_linear_ws) */
#define APEX4_DEBUG_GENERAL_TILES 1 /* tile kernel only: no one-row, few-row or ping-pong (G = 128, 256) kernel */
#define APEX4_DEBUG_W_TILED 2       /* W_q is in the tiled layout of apex4_tile_weights */

/*
 * Debug form of apex4_w4a4_gemm / apex4_w4a4_gemm_ws (and, with
 * APEX4_DEBUG_W_TILED, apex4_w4a4_gemm_tiled) that returns, from the same
 * launches that compute Y, the exact int32 group sums of Eq.
 * (group_decomposition) for rows [m0, m0 + mr).
 *
 *   Operands and Y as apex4_w4a4_gemm.  workspace == NULL: the kernel choice
 *   of apex4_w4a4_gemm; otherwise that of apex4_w4a4_gemm_ws (workspace as
 *   there, including APEX4_ERR_WORKSPACE).
 *   P [mr, N, K/G] int32 (device, output), window as in
 *   apex4_w4a4_gemm_groupsums; mr == 0 writes no sums (P may be NULL).
 *   flags: 0 or a combination of APEX4_DEBUG_GENERAL_TILES and
 *   APEX4_DEBUG_W_TILED (other bits: APEX4_ERR_SHAPE).
 * Without APEX4_DEBUG_GENERAL_TILES, Y is bit for bit the Y of the production
 * entry point named above.  For tests and diagnostics; slower than the
 * production calls.
 */
int apex4_w4a4_gemm_debug(const uint8_t* A_q, const void* s_a,
                          const uint8_t* W_q, const void* s_w,
                          int64_t M, int64_t N, int64_t K, int64_t G,
                          void* Y, void* workspace, int64_t workspace_bytes,
                          int64_t m0, int64_t mr, int32_t* P, int flags, void* stream);

/* entry points and kernels of apex4_w4a4_gemm_plan */
#define APEX4_ENTRY_GEMM 0    /* apex4_w4a4_gemm (and _debug without workspace) */
#define APEX4_ENTRY_GEMM_WS 1 /* apex4_w4a4_gemm_ws (and _debug with workspace) */
#define APEX4_ENTRY_LINEAR 2  /* apex4_w4a4_linear (and _debug); its GEMM, after the quantizer */
#define APEX4_ENTRY_LINEAR_WS 3 /* apex4_w4a4_linear_ws; its GEMM, after the quantizer */
#define APEX4_KERNEL_GEMV 1       /* one row (two on tiled weights): v_dot8 on the packed codes */
#define APEX4_KERNEL_FUSED 2      /* one row: quantizer fused into the GEMV's prologue */
#define APEX4_KERNEL_DECODE 3     /* up to 32 rows: weights streamed once through the MFMA */
#define APEX4_KERNEL_TILE_64 4    /* 64 x 128 output tiles */
#define APEX4_KERNEL_TILE_128 5   /* 128 x 256 output tiles */
#define APEX4_KERNEL_PINGPONG 6   /* G = 128 or 256 on 128 x 256 tiles, MFMA and dequant waves alternating */
#define APEX4_KERNEL_DECODE_SPLIT 7 /* up to 32 rows, stream-K over the CUs (workspace entry points) */

/*
 * The GEMM kernel that `entry` runs for this shape on the current device, and
 * its split over K (*splits = S > 1 only for APEX4_ENTRY_GEMM_WS and
 * APEX4_ENTRY_LINEAR_WS, whose workspace size query then returns S M N 4 bytes).  flags as in
 * apex4_w4a4_gemm_debug (APEX4_DEBUG_W_TILED: the tiled entry points;
 * APEX4_ENTRY_LINEAR and APEX4_ENTRY_LINEAR_WS take no APEX4_DEBUG_GENERAL_TILES).  M == 0 gives kernel 0,
 * splits 0.  Shape and group rules as apex4_w4a4_gemm; unknown entry or flags:
 * APEX4_ERR_SHAPE.  Launches nothing.
 */
int apex4_w4a4_gemm_plan(int entry, int64_t M, int64_t N, int64_t K, int64_t G, int flags,
                         int* kernel, int* splits);

/*
 * Tiled weight layout: the offline packing step of the weights (Sec. 4.4
 * quantizes and packs W once, offline, into the vectors its kernel loads), laid
 * out for the CDNA4 MFMA fragments: 32-row tiles by 128-wide K stages, and in
 * each, the 32 packed bytes every lane of a 32-column fragment consumes stored
 * contiguously in lane order, so that a wave reads its fragment of a stage as
 * one 2 KB block:
 *   W_t[t][s][j][l][b] = W_q[32 t + l % 32][64 s + 32 (l / 32) + 16 j + b]
 *   (t < ceil(N/32), s < ceil(K/128), j < 2, l < 64, b < 16; zero past N and
 *   past K/2).
 * apex4_tiled_weights_size writes its size, ceil(N/32) ceil(K/128) 2048 bytes.
 * apex4_tile_weights writes it from packed codes W_q [N, K/2] (device,
 * read-only) into W_t (device, output, that size; must not alias W_q).
 * N >= 1, K >= 32 and K % 32 == 0; W_q and W_t under 4 GiB.
 */
int apex4_tiled_weights_size(int64_t N, int64_t K, int64_t* bytes);
int apex4_tile_weights(const uint8_t* W_q, int64_t N, int64_t K, uint8_t* W_t, void* stream);

/*
 * apex4_w4a4_gemm / apex4_w4a4_gemm_ws on tiled weights: the same Y, bit for
 * bit, with W_t from apex4_tile_weights in place of W_q (s_w unchanged).
 * workspace == NULL: the kernel choice of apex4_w4a4_gemm (no split over K);
 * otherwise that of apex4_w4a4_gemm_ws (workspace as there).
 * G in {128, 256, 512, 1024} or G == K >= 128 (APEX4_ERR_GROUP otherwise: the
 * layout serves kernels that take one group per stage or more); W_t under
 * 4 GiB; other rules as apex4_w4a4_gemm.
 * With one or two rows the result is within the tolerance of
 * apex4_w4a4_gemm (the dot-product kernel adds its fp32 partial sums in
 * another order) and otherwise the same bits.
 */
int apex4_w4a4_gemm_tiled(const uint8_t* A_q, const void* s_a,
                          const uint8_t* W_t, const void* s_w,
                          int64_t M, int64_t N, int64_t K, int64_t G,
                          void* Y, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Quantize-then-GEMM linear layer: the inference forward of one quantized
 * linear layer (Sec. 3.2.1: activations quantized dynamically, weights
 * offline).  Y and the work buffers end up exactly as after
 * apex4_quantize_act(x) into the work buffers followed by apex4_w4a4_gemm on
 * the same stream.  For one row (M = 1) and G in {32, 64, 128, 256, 512}
 * (G < K) this is one fused kernel that quantizes x in its prologue;
 * otherwise the two kernels are enqueued in that order.
 *
 *   x [M, K] binary16, W_q [N, K/2], s_w [N, K/G]  (device, read-only);
 *   Y [M, N] binary16 (device, output);
 *   A_q_work [M, K/2] and s_a_work [M, K/G] (device, caller-owned scratch,
 *   overwritten with the quantized activations).
 */
int apex4_w4a4_linear(const void* x, const uint8_t* W_q, const void* s_w,
                      int64_t M, int64_t N, int64_t K, int64_t G,
                      void* Y, uint8_t* A_q_work, void* s_a_work, void* stream);

/*
 * apex4_w4a4_linear on tiled weights (apex4_tile_weights): the same kernels'
 * tiled forms, G and W_t rules as apex4_w4a4_gemm_tiled.
 */
int apex4_w4a4_linear_tiled(const void* x, const uint8_t* W_t, const void* s_w,
                            int64_t M, int64_t N, int64_t K, int64_t G,
                            void* Y, uint8_t* A_q_work, void* s_a_work, void* stream);

/*
 * Workspace form of apex4_w4a4_linear (flags 0: W row-major, W_q) and of
 * apex4_w4a4_linear_tiled (flags APEX4_DEBUG_W_TILED: W in the tiled layout,
 * W_t): the quantizer into the work buffers, then the GEMM with the kernel
 * choice of apex4_w4a4_gemm_ws (tiled: apex4_w4a4_gemm_tiled given a
 * workspace), i.e. split over K, or the few-row kernel's stream-K form, where
 * those apply (Eq. (group_decomposition) split over K across workgroups).
 * For one row where apex4_w4a4_linear fuses the quantizer into the GEMM, that
 * fused kernel runs and takes no workspace.  Y and the work buffers end up
 * exactly as after apex4_quantize_act followed by that GEMM entry point on the
 * same stream.
 *
 *   x, W, s_w, Y, A_q_work, s_a_work: as apex4_w4a4_linear;
 *   workspace: as apex4_w4a4_gemm_ws, at least apex4_w4a4_gemm_workspace_size
 *   bytes for this shape (the same size for both weight layouts); may be NULL
 *   where that size is 0.
 * flags other than 0 and APEX4_DEBUG_W_TILED: APEX4_ERR_SHAPE.  Errors as
 * apex4_w4a4_linear, plus APEX4_ERR_WORKSPACE when the workspace is needed and
 * NULL or short; that check comes before any launch, so nothing is written.
 */
int apex4_w4a4_linear_ws(const void* x, const uint8_t* W, const void* s_w,
                         int64_t M, int64_t N, int64_t K, int64_t G,
                         void* Y, uint8_t* A_q_work, void* s_a_work,
                         void* workspace, int64_t workspace_bytes, int flags, void* stream);

/*
 * Debug form of apex4_w4a4_linear (flags 0) or apex4_w4a4_linear_tiled (flags
 * APEX4_DEBUG_W_TILED): the same kernels (fused or quantize + GEMM), Y and
 * work buffers bit for bit, plus the exact int32 group sums of rows
 * [m0, m0 + mr) into P [mr, N, K/G] as in apex4_w4a4_gemm_debug.
 */
int apex4_w4a4_linear_debug(const void* x, const uint8_t* W_q, const void* s_w,
                            int64_t M, int64_t N, int64_t K, int64_t G,
                            void* Y, uint8_t* A_q_work, void* s_a_work,
                            int64_t m0, int64_t mr, int32_t* P, int flags, void* stream);

/*
 * Workspace form of apex4_w4a4_gemm for shapes that leave compute units idle
 * (Eq. (group_decomposition) split over K; the striped work decomposition of
 * Sec. 4.2 across workgroups).  When the GEMM's tiles number too few for the
 * compute units (M > 32), K is split into S in {2, 4, 8} ranges of whole
 * groups; each workgroup writes a partial tile into the workspace (fp32, or
 * the exact int32 sums for G == K), and a second kernel sums the S partials in
 * range order and rounds once to binary16.  With M <= 32 rows, where the
 * 32-column tiles leave more than a tenth of the compute units idle in the last
 * round and the tiles are long (below one tile per compute unit, at least 128
 * stage-groups, i.e. K/128 stages times 128/G groups per stage, and K >= 24576
 * once half the compute units or more have a tile; K >= 24576 above), the
 * few-row kernel runs in a stream-K form: the full rounds stay
 * whole tiles, the remaining tiles' 128-wide K stages are spread evenly over
 * the workgroups, and a tile cut between workgroups has its fp32 parts added in
 * segment order by the workgroup that finishes last (counters cleared by a
 * kernel on every call, so a captured call replays).  Y is then within the
 * tolerance of apex4_w4a4_gemm (the fp32 summation order differs; for G == K
 * the tile kernels' split gives the same bits), deterministic for a given shape
 * and device.
 *
 * apex4_w4a4_gemm_workspace_size writes to *bytes the workspace this shape
 * needs on the current device: S * M * N * 4 for the split over K, counters
 * and fp32 parts for the stream-K form, or 0 where neither applies (then
 * apex4_w4a4_gemm_ws is apex4_w4a4_gemm and workspace may be NULL).
 *
 *   workspace: caller-owned device memory, 16-byte aligned, at least *bytes
 *   long; overwritten; must not alias the operands.  Calls that share a
 *   workspace must be ordered on one stream.
 * Errors as apex4_w4a4_gemm, plus APEX4_ERR_WORKSPACE when the workspace is
 * needed and NULL or shorter than the size query returns (checked last, after
 * the device, since the split depends on the device's compute-unit count).
 */
int apex4_w4a4_gemm_workspace_size(int64_t M, int64_t N, int64_t K, int64_t G, int64_t* bytes);
int apex4_w4a4_gemm_ws(const uint8_t* A_q, const void* s_a,
                       const uint8_t* W_q, const void* s_w,
                       int64_t M, int64_t N, int64_t K, int64_t G,
                       void* Y, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Re-encode packed 4-bit codes as FP6 e3m2 codes for apex4_w4a4_gemm_fp6.
 * Every code q in [-8, 7] is exact in FP6 e3m2 (1 sign, 3 exponent with bias 3,
 * 2 mantissa bits); this is a change of container for the codes of Sec. 3.2.1,
 * not of their values, made once per weight matrix (Alg. 1 quantizes weights
 * offline) and per activation batch.
 *
 *   q4 [rows, K/2] packed codes as above (device, read-only);
 *   q6 [rows, 3K/4] (device, output): code k of a row in bits [6k, 6k + 6) of
 *   the row's bytes read as a little-endian bit string.
 * rows >= 0; K >= 128, K % 128 == 0; rows == 0 is a no-op.
 */
int apex4_pack_fp6(const uint8_t* q4, int64_t rows, int64_t K, uint8_t* q6, void* stream);

/*
 * apex4_w4a4_gemm on FP6 containers: the same Y, bit for bit, from the codes
 * re-encoded by apex4_pack_fp6 (Eq. (group_decomposition); the group sums are
 * exact on the FP6 matrix cores, whose products and fp32 sums of at most 128
 * products of codes are integers below 2^24).
 *
 *   A_6 [M, 3K/4], W_6 [N, 3K/4] FP6 codes; s_a [M, K/G], s_w [N, K/G] binary16
 *   scales (device, read-only); Y [M, N] binary16 (device, output).
 * G == 128 only (APEX4_ERR_GROUP otherwise); each FP6 operand under 4 GiB
 * (M 3K/4 and N 3K/4 below 2^32 bytes); other rules as apex4_w4a4_gemm.
 */
int apex4_w4a4_gemm_fp6(const uint8_t* A_6, const void* s_a,
                        const uint8_t* W_6, const void* s_w,
                        int64_t M, int64_t N, int64_t K, int64_t G,
                        void* Y, void* stream);

/*
 * MX numerics variant (CDNA4 only).  NOT the paper's scales: SymQuant's 4-bit
 * symmetric codes (Sec. 3.2.1) with each group scale restricted to a power of
 * two, 2^E with E = min{e integer : max|X_g| <= 7 * 2^e} (E = 0 for an all-zero
 * group), so that the block-scaled FP6 MFMA applies it and no per-group
 * dequantization is left (Sec. 2.2 makes this point for block-scaled FP4).
 *
 * apex4_quantize_mx: x [M, K] binary16 -> Q6 [M, 3K/4] FP6 e3m2 codes (layout
 *   of apex4_pack_fp6), codes clamp(round-half-even(x / 2^E), -8, 7); e [M, K/G]
 *   E8M0 bytes E + 127.  Bit-exact and deterministic.
 * apex4_w4a4_gemm_mx: Y[m,n] = binary16( sum_g 2^(Ea[m,g] + Ew[n,g] - 254) P[m,n,g] )
 *   with P the exact group sums of Eq. (group_decomposition); accumulated in
 *   binary32 by the MFMA across all of K, rounded once to binary16.
 *   A_6 [M, 3K/4], e_a [M, K/G], W_6 [N, 3K/4], e_w [N, K/G] (device,
 *   read-only); Y [M, N] binary16 (device, output).
 * G in {32, 64, 128, 256, 512, 1024} with G <= K (APEX4_ERR_GROUP otherwise);
 * K % 128 == 0, K % G == 0; FP6 operands under 4 GiB; 16-byte aligned pointers.
 */
int apex4_quantize_mx(const void* x, int64_t M, int64_t K, int64_t G,
                      uint8_t* Q6, uint8_t* e, void* stream);
int apex4_w4a4_gemm_mx(const uint8_t* A_6, const uint8_t* e_a,
                       const uint8_t* W_6, const uint8_t* e_w,
                       int64_t M, int64_t N, int64_t K, int64_t G,
                       void* Y, void* stream);

/*
 * Workspace form of apex4_w4a4_gemm_mx, as apex4_w4a4_gemm_ws is of
 * apex4_w4a4_gemm: when the MX GEMM's tiles leave compute units idle, K is
 * split into S in {2, 4, 8} ranges; fp32 partial tiles go to the caller's
 * workspace (S * M * N * 4 bytes, from the size query; 0 = no split, then this
 * is apex4_w4a4_gemm_mx and workspace may be NULL) and are summed in range
 * order, then rounded once to binary16.  Deterministic, within the tolerance
 * of the unsplit result.  Errors as apex4_w4a4_gemm_mx, plus
 * APEX4_ERR_WORKSPACE (checked last, after the device).
 */
int apex4_w4a4_gemm_mx_workspace_size(int64_t M, int64_t N, int64_t K, int64_t G, int64_t* bytes);
int apex4_w4a4_gemm_mx_ws(const uint8_t* A_6, const uint8_t* e_a,
                          const uint8_t* W_6, const uint8_t* e_w,
                          int64_t M, int64_t N, int64_t K, int64_t G,
                          void* Y, void* workspace, int64_t workspace_bytes, void* stream);

/* Static description of a status code (never NULL). */
const char* apex4_status_string(int status);

/* Library version: major * 10000 + minor * 100 + patch. */
int apex4_version(void);

#ifdef __cplusplus
}
#endif

#endif /* APEX4_H */
