/*
 * apex4_oracle.h -- CPU oracle for the W4A4 group-quantized GEMM path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  The product path
 * (the HIP library) never calls it and shares no code, header or table with it.
 *
 * Paper: "APEX4: Efficient Pure W4A4 LLM Inference via Intra-SM Compute
 * Rebalancing" (arXiv 2606.08761).
 *   - Quantizer: Sec. 3.2.1, Eq. (SymQuant) and Alg. 1 (SymQuant helper):
 *       S_g = max|X_g| / (2^(b-1) - 1),  X_g^q = clamp(round(X_g / S_g), -2^(b-1), 2^(b-1) - 1), b = 4.
 *   - GEMM: Sec. 3.2.1, Eq. (group_decomposition):
 *       C = sum_g (A_g^q W_g^q) (.) (S_g^a S_g^w^T)
 *     computed here as exact int64 group sums followed by an fp64 scaled sum.
 *
 * Conventions (readings where the paper is silent; each is listed in the
 * design notes with its justification):
 *   - round() is round-half-to-even on the exact quotient;
 *   - the scale is the binary16 value nearest to amax/7 (ties to even), and the
 *     integer codes use that binary16 scale;
 *   - a group whose binary16 scale is zero gets all-zero codes and scale 0;
 *   - codes are packed two per byte along K, low nibble = even k;
 *   - A_q is [M, K/2] bytes, W_q is [N, K/2] bytes, scales are [rows, K/G]
 *     binary16 bit patterns, Y = A W^T is [M, N].
 *
 * Parity pins: every function here is checked, on the CPU, against values the
 * paper or mathematics fix (hand-computed examples, exhaustive comparisons with
 * numpy's IEEE conversions, exact rational arithmetic, closed forms and
 * invariants of the group decomposition).
 */
#ifndef APEX4_ORACLE_H
#define APEX4_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* IEEE 754 binary16 -> binary64, exact. */
double apex4o_f16_to_f64(uint16_t h);
/* binary64 -> binary16, round to nearest, ties to even; overflow -> +-inf. */
uint16_t apex4o_f64_to_f16(double x);
/* Vectorised forms of the two converters above. */
void apex4o_f16_to_f64_n(const uint16_t* h, int64_t n, double* out);
void apex4o_f64_to_f16_n(const double* x, int64_t n, uint16_t* out);

/* SymQuant of one row-major [R, K] binary16 matrix, groups of G along K.
 * q_packed: [R, K/2] bytes; scales: [R, K/G] binary16.  Requires K % G == 0,
 * G even.  Returns 0, or -1 on a shape error. */
int apex4o_quantize(const uint16_t* x, int64_t R, int64_t K, int64_t G,
                    uint8_t* q_packed, uint16_t* scales);

/* Exact group partial sums P[i, n, g] = sum_{k in g} A_q[m0+i, k] * W_q[n, k]
 * for rows m0 <= m < m0+mr.  P is [mr, N, K/G] int64. */
int apex4o_groupsums(const uint8_t* Aq, const uint8_t* Wq, int64_t M, int64_t N,
                     int64_t K, int64_t G, int64_t m0, int64_t mr, int64_t* P);

/* y[i, n] = sum_g s_a[rows[i], g] * s_w[n, g] * P[rows[i], n, g] in binary64,
 * g ascending, for the listed rows (any order, repeats allowed).
 * y is [nrows, N]. */
int apex4o_gemm_rows(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                     const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G,
                     const int64_t* rows, int64_t nrows, double* y);

/* Number of OpenMP threads the oracle's parallel loops use. */
int apex4o_num_threads(void);
/* Threads used by the following oracle calls (OpenMP; n > 0).  Timing only. */
void apex4o_set_num_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
