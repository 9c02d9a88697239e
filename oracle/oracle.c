/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY. Plain, slow, obviously correct CPU
 * reference for the sparse-times-dense product of the paper. Only the tests,
 * the smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product path never does.
 *
 * What is computed (Section 5.1, "M/K/N" notation): the weight matrix W is
 * M x K and sparse, the input X is K x N and dense, the output Y is M x N.
 * The storage format of Section 3.2 (any format, ours included) is a lossless
 * re-encoding of W restricted to its kept entries, and the kernel of
 * Section 4 reduces all parts of the format into one result (Section 4.4,
 * the final reduction), so the exact result is the masked dense product
 *
 *     Y[m][n] = sum over k with mask[m][k] != 0 of W[m][k] * X[k][n]
 *
 * evaluated here in float64. Every fp16 x fp16 product is exact in float64
 * (11-bit significands), so the only rounding is the float64 summation.
 * Alongside Y the oracle returns A[m][n] = sum |W[m][k]| * |X[k][n]| over the
 * same k, the scale of the elementwise tolerance.
 *
 * Layouts (plain pointers, element strides):
 *   W    row-major M x K fp16 bit patterns, row m at W + m*ldw
 *   mask row-major M x K bytes, row m at mask + m*ldm, nonzero = kept
 *   X    token-major: column n of the logical K x N matrix at X + n*ldx
 *   Y, A token-major N x R float64 (R = number of output rows), Y[n*R + i]
 *
 * Compile-time option ORACLE_MUTANT=<id> plants one deliberate mistake; the
 * test suite builds those variants to show that its pins catch each of them.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#ifndef ORACLE_MUTANT
#define ORACLE_MUTANT 0
#endif

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * exponent 0: zero or subnormal, value = fraction * 2^-24;
 * exponent 31: infinity (fraction 0) or NaN;
 * otherwise (1024 + fraction) * 2^(exponent - 25). */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int f = h & 0x3FF;
    double v;
    if (e == 0) {
#if ORACLE_MUTANT == 4
        v = 0.0; /* planted: subnormals flushed */
#else
        v = ldexp((double)f, -24);
#endif
    } else if (e == 31) {
        v = f ? NAN : INFINITY;
    } else {
#if ORACLE_MUTANT == 3
        v = ldexp((double)(1024 + f), e - 24); /* planted: wrong exponent bias */
#else
        v = ldexp((double)(1024 + f), e - 25);
#endif
    }
#if ORACLE_MUTANT == 6
    (void)sign;
    return v; /* planted: sign dropped */
#else
    return sign ? -v : v;
#endif
}

void oracle_f16_to_f64_array(const uint16_t *h, int64_t n, double *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_f16_to_f64(h[i]);
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Masked product for the output rows listed in rows[0..R-1] (rows == NULL
 * means all M rows in order, R == M). Returns 0, or -1 on bad arguments. */
int oracle_masked_gemm_rows(const uint16_t *W, int64_t ldw,
                            const uint8_t *mask, int64_t ldm,
                            const uint16_t *X, int64_t ldx,
                            int64_t M, int64_t K, int64_t N,
                            const int64_t *rows, int64_t R,
                            double *Y, double *A)
{
    if (M < 0 || K < 0 || N < 0 || R < 0 || ldw < K || ldm < K || ldx < K) return -1;
    if (rows == NULL && R != M) return -1;
    /* X decoded once: Xd[n][k] */
    double *Xd = (double *)malloc(sizeof(double) * (size_t)(N * K > 0 ? N * K : 1));
    if (!Xd) return -1;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k) Xd[n * K + k] = oracle_f16_to_f64(X[n * ldx + k]);

    int bad = 0;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t i = 0; i < R; ++i) {
        int64_t m = rows ? rows[i] : i;
        if (m < 0 || m >= M) { bad = 1; continue; }
        for (int64_t n = 0; n < N; ++n) {
            double s = 0.0, a = 0.0;
#if ORACLE_MUTANT == 5
            for (int64_t k = 0; k + 1 < K; ++k) { /* planted: last column dropped */
#else
            for (int64_t k = 0; k < K; ++k) {
#endif
#if ORACLE_MUTANT == 1
                /* planted: mask ignored */
#else
                if (!mask[m * ldm + k]) continue;
#endif
                double w = oracle_f16_to_f64(W[m * ldw + k]);
#if ORACLE_MUTANT == 2
                double x = (k < N && n < K) ? Xd[k * K + n] : 0.0; /* planted: X transposed */
#else
                double x = Xd[n * K + k];
#endif
                s += w * x;
                a += fabs(w) * fabs(x);
            }
            Y[n * R + i] = s;
            A[n * R + i] = a;
        }
    }
    free(Xd);
    return bad ? -1 : 0;
}

/* The fp16 bit patterns of W restricted to its kept entries: kept entries keep
 * their bits (including -0, subnormals, NaN payloads), the rest become +0. */
void oracle_masked_bits(const uint16_t *W, int64_t ldw, const uint8_t *mask, int64_t ldm,
                        int64_t M, int64_t K, uint16_t *out)
{
    for (int64_t m = 0; m < M; ++m)
        for (int64_t k = 0; k < K; ++k)
            out[m * K + k] = mask[m * ldm + k] ? W[m * ldw + k] : (uint16_t)0;
}
