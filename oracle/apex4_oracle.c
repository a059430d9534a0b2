/*
 * apex4_oracle.c -- plain, slow, obviously correct CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * CPU-baseline leg of the benchmark, never by the product library.
 *
 * Every function restates a definition from the APEX4 paper (arXiv 2606.08761)
 * in the most direct form: integer sums are exact (int64), the scaled sum is
 * taken in binary64, and every rounding is written out from the IEEE 754
 * definition rather than delegated to hardware conversions.
 * No blocking, no fusion, no reordering beyond what the definitions state.
 */
#include "apex4_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* binary16 <-> binary64 (IEEE 754-2008, Sec. 3.4 binary interchange format)  */
/* ------------------------------------------------------------------------ */

double apex4o_f16_to_f64(uint16_t h)
{
    const int sign = (h >> 15) & 1;
    const int e = (h >> 10) & 0x1f;      /* biased exponent, bias 15 */
    const int f = h & 0x3ff;             /* 10 fraction bits */
    double v;
    if (e == 0) {
        v = ldexp((double)f, -24);       /* subnormal: 0.f * 2^-14 = f * 2^-24 */
    } else if (e == 31) {
        v = f ? NAN : INFINITY;
    } else {
        v = ldexp((double)(1024 + f), e - 25); /* 1.f * 2^(e-15) */
    }
    return sign ? -v : v;
}

/* Encode a non-negative value that is an exact binary16 number n * 2^(ex-10)
 * with 0 <= n <= 2048 and ex >= -14 (the caller guarantees it). */
static uint16_t encode_f16(double n, int ex)
{
    if (n == 2048.0) { n = 1024.0; ex += 1; }      /* carried into next binade */
    if (n < 1024.0) {                              /* only possible at ex == -14 */
        return (uint16_t)n;                        /* subnormal (or zero) */
    }
    if (ex > 15) return 0x7c00;                    /* overflow to infinity */
    return (uint16_t)(((ex + 15) << 10) | ((int)n - 1024));
}

uint16_t apex4o_f64_to_f16(double x)
{
    const uint16_t sign = signbit(x) ? 0x8000 : 0;
    if (isnan(x)) return 0x7e00;
    double a = fabs(x);
    if (isinf(a)) return sign | 0x7c00;
    if (a == 0.0) return sign;
    /* a lies in [2^ex, 2^(ex+1)); below 2^-14 the grid spacing stays 2^-24. */
    int e2;
    (void)frexp(a, &e2);
    int ex = e2 - 1;
    if (ex < -14) ex = -14;
    /* Grid spacing in this binade is 2^(ex-10); count grid steps exactly. */
    double steps = ldexp(a, 10 - ex);   /* exact: scaling by a power of two */
    double n = floor(steps);
    double rem = steps - n;             /* exact */
    if (rem > 0.5 || (rem == 0.5 && fmod(n, 2.0) != 0.0)) n += 1.0; /* RNE */
    if (ex > 15) return sign | 0x7c00;
    return sign | encode_f16(n, ex);
}

void apex4o_f16_to_f64_n(const uint16_t* h, int64_t n, double* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = apex4o_f16_to_f64(h[i]);
}

void apex4o_f64_to_f16_n(const double* x, int64_t n, uint16_t* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = apex4o_f64_to_f16(x[i]);
}

/* ------------------------------------------------------------------------ */
/* SymQuant (Sec. 3.2.1, Eq. SymQuant; Alg. 1 SymQuant helper), b = 4         */
/* ------------------------------------------------------------------------ */

/* Next binary16 bit pattern above / below a non-negative finite pattern. */
static uint16_t f16_up(uint16_t h) { return (uint16_t)(h + 1); }
static uint16_t f16_down(uint16_t h) { return h ? (uint16_t)(h - 1) : 0; }

/* Scale S = amax / (2^(b-1) - 1) = amax / 7, delivered as the binary16 value
 * nearest to the exact quotient (ties to the even bit pattern).
 * Candidates: the binary16 rounding of the binary64 quotient and its two
 * neighbours; the winner minimises |7 v - amax|, which is computed exactly
 * (7 v and amax are short binary numbers of nearby magnitude). */
static uint16_t scale_of_amax(double amax)
{
    uint16_t c = apex4o_f64_to_f16(amax / 7.0);
    uint16_t cand[3] = { f16_down(c), c, f16_up(c) };
    uint16_t best = cand[1];
    double best_err = fabs(7.0 * apex4o_f16_to_f64(best) - amax);
    for (int i = 0; i < 3; i += 2) {
        double v = apex4o_f16_to_f64(cand[i]);
        if (isinf(v)) continue;
        double err = fabs(7.0 * v - amax);
        if (err < best_err || (err == best_err && (cand[i] & 1) == 0 && (best & 1) == 1)) {
            best = cand[i];
            best_err = err;
        }
    }
    return best;
}

/* Nearest integer to the exact quotient x / s (ties to even), s > 0.
 * The binary64 quotient gives a candidate; the exact residual x - n s decides. */
static double round_quotient(double x, double s)
{
    double n = nearbyint(x / s);
    for (int it = 0; it < 2; ++it) {
        double r = x - n * s;             /* exact: short operands */
        double h = 0.5 * s;
        if (r > h) n += 1.0;
        else if (r < -h) n -= 1.0;
        else if (r == h && fmod(n, 2.0) != 0.0) n += 1.0;
        else if (r == -h && fmod(n, 2.0) != 0.0) n -= 1.0;
        else break;
    }
    return n;
}

int apex4o_quantize(const uint16_t* x, int64_t R, int64_t K, int64_t G,
                    uint8_t* q_packed, uint16_t* scales)
{
    if (R < 0 || K <= 0 || G <= 0 || (K % G) != 0 || (G % 2) != 0) return -1;
    const int64_t ng = K / G;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < R; ++r) {
        const uint16_t* xr = x + r * K;
        for (int64_t g = 0; g < ng; ++g) {
            /* amax = max_{k in g} |x| (exact) */
            double amax = 0.0;
            for (int64_t k = g * G; k < (g + 1) * G; ++k) {
                double v = fabs(apex4o_f16_to_f64(xr[k]));
                if (v > amax) amax = v;
            }
            uint16_t s16 = scale_of_amax(amax);
            double s = apex4o_f16_to_f64(s16);
            scales[r * ng + g] = s16;
            for (int64_t k = g * G; k < (g + 1) * G; k += 2) {
                int q2[2];
                for (int j = 0; j < 2; ++j) {
                    double q = 0.0;
                    if (s != 0.0) {
                        q = round_quotient(apex4o_f16_to_f64(xr[k + j]), s);
                        if (q < -8.0) q = -8.0;      /* clamp to [-2^(b-1), 2^(b-1)-1] */
                        if (q > 7.0) q = 7.0;
                    }
                    q2[j] = (int)q;
                }
                /* two codes per byte, low nibble = even k */
                q_packed[r * (K / 2) + k / 2] = (uint8_t)((q2[0] & 0xF) | ((q2[1] & 0xF) << 4));
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Group-decomposed GEMM (Sec. 3.2.1, Eq. group_decomposition)                */
/* ------------------------------------------------------------------------ */

/* Signed 4-bit code k of a packed row (low nibble = even k). */
static int code_at(const uint8_t* row, int64_t k)
{
    int nib = (k & 1) ? (row[k >> 1] >> 4) : (row[k >> 1] & 0xF);
    return nib >= 8 ? nib - 16 : nib;
}

static void unpack_row(const uint8_t* row, int64_t K, int8_t* out)
{
    for (int64_t k = 0; k < K; ++k) out[k] = (int8_t)code_at(row, k);
}

static int check_gemm_shape(int64_t M, int64_t N, int64_t K, int64_t G)
{
    if (M < 0 || N < 0 || K <= 0 || G <= 0 || (K % G) != 0 || (K % 2) != 0) return -1;
    return 0;
}

int apex4o_groupsums(const uint8_t* Aq, const uint8_t* Wq, int64_t M, int64_t N,
                     int64_t K, int64_t G, int64_t m0, int64_t mr, int64_t* P)
{
    if (check_gemm_shape(M, N, K, G) || m0 < 0 || mr < 0 || m0 + mr > M) return -1;
    const int64_t ng = K / G;
    int8_t* W8 = (int8_t*)malloc((size_t)(N > 0 ? N : 1) * (size_t)K);
    if (!W8) return -2;
    for (int64_t n = 0; n < N; ++n) unpack_row(Wq + n * (K / 2), K, W8 + n * K);
#pragma omp parallel
    {
        int8_t* a8 = (int8_t*)malloc((size_t)K);
#pragma omp for schedule(static)
        for (int64_t i = 0; i < mr; ++i) {
            unpack_row(Aq + (m0 + i) * (K / 2), K, a8);
            for (int64_t n = 0; n < N; ++n) {
                const int8_t* w8 = W8 + n * K;
                for (int64_t g = 0; g < ng; ++g) {
                    int64_t acc = 0;
                    for (int64_t k = g * G; k < (g + 1) * G; ++k) acc += (int64_t)a8[k] * (int64_t)w8[k];
                    P[(i * N + n) * ng + g] = acc;
                }
            }
        }
        free(a8);
    }
    free(W8);
    return 0;
}

int apex4o_gemm_rows(const uint8_t* Aq, const uint16_t* sa, const uint8_t* Wq,
                     const uint16_t* sw, int64_t M, int64_t N, int64_t K, int64_t G,
                     const int64_t* rows, int64_t nrows, double* y)
{
    if (check_gemm_shape(M, N, K, G) || nrows < 0) return -1;
    for (int64_t i = 0; i < nrows; ++i)
        if (rows[i] < 0 || rows[i] >= M) return -1;
    const int64_t ng = K / G;
    int8_t* W8 = (int8_t*)malloc((size_t)(N > 0 ? N : 1) * (size_t)K);
    double* swd = (double*)malloc((size_t)(N > 0 ? N : 1) * (size_t)ng * sizeof(double));
    if (!W8 || !swd) { free(W8); free(swd); return -2; }
    for (int64_t n = 0; n < N; ++n) unpack_row(Wq + n * (K / 2), K, W8 + n * K);
    for (int64_t t = 0; t < N * ng; ++t) swd[t] = apex4o_f16_to_f64(sw[t]);
#pragma omp parallel
    {
        int8_t* a8 = (int8_t*)malloc((size_t)K);
        double* sad = (double*)malloc((size_t)ng * sizeof(double));
#pragma omp for schedule(static)
        for (int64_t i = 0; i < nrows; ++i) {
            const int64_t m = rows[i];
            unpack_row(Aq + m * (K / 2), K, a8);
            for (int64_t g = 0; g < ng; ++g) sad[g] = apex4o_f16_to_f64(sa[m * ng + g]);
            for (int64_t n = 0; n < N; ++n) {
                const int8_t* w8 = W8 + n * K;
                double acc = 0.0;
                for (int64_t g = 0; g < ng; ++g) {
                    int64_t p = 0;      /* exact integer partial sum of group g */
                    for (int64_t k = g * G; k < (g + 1) * G; ++k) p += (int64_t)a8[k] * (int64_t)w8[k];
                    /* s_a * s_w * p is exact in binary64 (11 + 11 + <=22 significant bits) */
                    acc += (sad[g] * swd[n * ng + g]) * (double)p;
                }
                y[i * N + n] = acc;
            }
        }
        free(a8);
        free(sad);
    }
    free(W8);
    free(swd);
    return 0;
}

int apex4o_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void apex4o_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
