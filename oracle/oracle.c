/*
 * CPU oracle for C = A . B  (TEST INFRASTRUCTURE ONLY).
 *
 * Only tests, the smoke check and the bench's CPU-baseline leg may load this
 * library; the product path never does.  It shares no code with the HIP
 * library.
 *
 * What it computes.  The paper's kernels (MatMul and BatchMatMul, written as
 * [M,K,N] in its kernel table, Table 3) are schedules of one loop nest: a
 * candidate is a sequence of primitives (tiling, reorder, unroll, ...) applied
 * to the same computation (Sec. 2, "kernel generation pipeline"; Fig. 10 tiles
 * only re-block it).  Every candidate therefore reaches, up to rounding order,
 * the plain product
 *
 *     R[b][i][j] = sum_{k=0}^{K-1} A[b][i][k] * B[b][k][j]
 *
 * and that definition is what this file evaluates: every product and every
 * partial sum in fp64, k ascending, starting from 0.  fp32 and fp16 inputs
 * convert to fp64 exactly, and the product of two such values is exact in fp64
 * (at most 48 significand bits), so the only rounding is in the additions.
 *
 * Layout: row-major with leading dimensions (lda >= K, ldb >= N, ldr >= N) and
 * batch strides in elements.  R is fp64.
 *
 * Loop order: the operands are converted to fp64 once per call (exactly; a
 * plain loop over every element), then each output row i is accumulated in
 * place, k outer, j inner.  For every single element this is the same
 * k-ascending sum as the i-j-k triple loop, so the result is bit-identical to
 * it and does not depend on the number of OpenMP threads (work is split over
 * (b, i, column block) only).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* IEEE 754 binary16 -> binary64, exact: 1 sign bit, 5 exponent bits (bias
 * 15), 10 fraction bits; exponent 0 encodes zero/subnormals (no implicit 1,
 * scale 2^-14), exponent 31 encodes inf/NaN. */
double oracle_f16_to_f64(uint16_t h)
{
    const int sign = (h >> 15) & 1;
    const int e = (h >> 10) & 0x1f;
    const int f = h & 0x3ff;
    double v;
    if (e == 0) {
        v = (double)f / 1024.0 / 16384.0; /* f * 2^-10 * 2^-14 */
    } else if (e == 31) {
        if (f == 0) {
            v = 1.0 / 0.0;
        } else {
            uint64_t nan_bits = 0x7ff8000000000000ull;
            memcpy(&v, &nan_bits, sizeof v);
        }
    } else {
        v = 1.0 + (double)f / 1024.0;
        int p = e - 15;
        while (p > 0) { v *= 2.0; --p; }
        while (p < 0) { v *= 0.5; ++p; }
    }
    return sign ? -v : v;
}

enum { ORACLE_F32 = 0, ORACLE_F16 = 1 };
enum { COLS_PER_TASK = 512 };

/* Elements an operand occupies: slices at stride `stride`, `rows` rows of
 * `ld` elements, `cols` used per row (0 when the operand is empty). */
static int64_t span_of(int64_t batch, int64_t stride, int64_t rows, int64_t ld, int64_t cols)
{
    if (batch == 0 || rows == 0 || cols == 0)
        return 0;
    return (batch - 1) * stride + (rows - 1) * ld + cols;
}

/* Every element of an operand's span, converted exactly to fp64, once.  The
 * span includes padding between rows and slices; those values are converted
 * but never used. */
static double *to_f64(const void *p, int64_t n, int dtype)
{
    double *out = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    if (!out)
        return NULL;
    if (dtype == ORACLE_F32) {
        const float *f = (const float *)p;
        for (int64_t t = 0; t < n; ++t)
            out[t] = (double)f[t];
    } else {
        const uint16_t *h = (const uint16_t *)p;
        for (int64_t t = 0; t < n; ++t)
            out[t] = oracle_f16_to_f64(h[t]);
    }
    return out;
}

/* Batched product in fp64; see the file comment for the definition.  The
 * operands are first converted to fp64 (exactly), then the sums run. */
int oracle_matmul(int64_t batch, int64_t M, int64_t N, int64_t K,
                  const void *A, int64_t lda, int64_t strideA,
                  const void *B, int64_t ldb, int64_t strideB,
                  double *R, int64_t ldr, int64_t strideR,
                  int dtype, int nthreads)
{
    if (batch < 0 || M < 0 || N < 0 || K < 0)
        return -1;
    if (dtype != ORACLE_F32 && dtype != ORACLE_F16)
        return -2;
    if (batch == 0 || M == 0 || N == 0)
        return 0;
    if (lda < K || ldb < N || ldr < N)
        return -1;

    double *Ad = to_f64(A, span_of(batch, strideA, M, lda, K), dtype);
    double *Bd = to_f64(B, span_of(batch, strideB, K, ldb, N), dtype);
    if (!Ad || !Bd) {
        free(Ad);
        free(Bd);
        return -3;
    }

    const int64_t col_tasks = (N + COLS_PER_TASK - 1) / COLS_PER_TASK;
    const int64_t ntasks = batch * M * col_tasks;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
#endif
    for (int64_t t = 0; t < ntasks; ++t) {
        const int64_t b = t / (M * col_tasks);
        const int64_t i = (t / col_tasks) % M;
        const int64_t j0 = (t % col_tasks) * COLS_PER_TASK;
        const int64_t j1 = (j0 + COLS_PER_TASK < N) ? j0 + COLS_PER_TASK : N;
        double *r = R + b * strideR + i * ldr;
        for (int64_t j = j0; j < j1; ++j)
            r[j] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double a = Ad[b * strideA + i * lda + k];
            const double *brow = Bd + b * strideB + k * ldb;
            for (int64_t j = j0; j < j1; ++j)
                r[j] += a * brow[j];
        }
    }
    free(Ad);
    free(Bd);
    (void)nthreads;
    return 0;
}

/* Weight-only 4-bit GEMV (the paper runs Llama-2 decode with 4-bit weights,
 * Sec. 7, without giving the format; this is the format the library reads,
 * the layout of a linear layer's weight: one row per output feature n,
 * quantised along the input features k in groups of G):
 *
 *     y[n] = sum_{k=0}^{K-1} x[k] * W[k][n],   W[k][n] = (q[n][k] - 8) * s[n][k / G]
 *
 * q[n][k] is an unsigned 4-bit code, eight per 32-bit word along k: input k
 * of output n is bits 4 (k % 8) .. 4 (k % 8) + 3 of word k / 8 of row n (ldq
 * words per row); s is a binary16 scale per output and group of G
 * consecutive inputs (lds halves per row); x is binary16.  Every weight and
 * every product x[k] W[k][n] is exact in fp64 (at most 11 + 15 significand
 * bits), so, as in oracle_matmul, only the k-ascending additions round. */
int oracle_gemv_q4(int64_t K, int64_t N, const uint16_t *x, const uint32_t *Wq, int64_t ldq,
                   const uint16_t *S, int64_t lds, int64_t G, double *y, int nthreads)
{
    if (K < 0 || N < 0 || G < 1)
        return -1;
    if (ldq < (K + 7) / 8 || lds < (K + G - 1) / G)
        return -1;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads)
#endif
    for (int64_t n = 0; n < N; ++n) {
        const uint32_t *row = Wq + n * ldq;
        const uint16_t *srow = S + n * lds;
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const int q = (int)((row[k / 8] >> (4 * (k % 8))) & 15u);
            const double w = ((double)q - 8.0) * oracle_f16_to_f64(srow[k / G]);
            acc += oracle_f16_to_f64(x[k]) * w;
        }
        y[n] = acc;
    }
    (void)nthreads;
    return 0;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
