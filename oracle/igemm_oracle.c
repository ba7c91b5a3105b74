/*
 * CPU oracle for integer GEMM  C += A * B  -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library. The GPU library never links, includes or calls it, and
 * this file includes nothing of the GPU library.
 *
 * What it computes (plain definition, no blocking, no reordering beyond the
 * order of the three loops, which integer arithmetic makes irrelevant):
 *
 *   Sec. 4.1 (GEMM in conventional processor architectures) defines the
 *   operation C += A B with A m x k, B k x n and C m x n. Fig. "baseline
 *   GEMM" (micro-kernel, loop L6) writes the same update as a sequence of
 *   rank-1 updates C += A(:,p) B(p,:) over p.
 *
 *   Sec. 6.2 (evaluation of the micro-kernel) motivates wide accumulators so
 *   that int16 products accumulate without overflow. Here every product and
 *   every partial sum is formed exactly in int64: |sum| <= k * 2^30 + 2^31,
 *   which is below 2^63 for any k < 2^32.
 *
 *   The output is int32 with two's-complement wraparound: the exact int64
 *   result is reduced modulo 2^32 once, at the end. (The paper's micro-kernel
 *   instead narrows its accumulators to int16 C through a shift-round-
 *   saturate step whose rounding it does not specify; this library's C is
 *   int32, so the modular reading is the one taken.)
 *
 * Storage: row-major with leading dimensions in elements:
 *   A[i,p] = A[i*lda + p], B[p,j] = B[p*ldb + j], C[i,j] = C[i*ldc + j].
 * Elements outside the logical m x k / k x n / m x n windows are never read
 * or written.
 *
 * Parallelism: OpenMP over rows i only; each row is computed by one thread in
 * the same order, so the result does not depend on the thread count.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Reduce an exact int64 sum modulo 2^32 to the int32 with the same low 32
 * bits. Written without any implementation-defined signed conversion. */
static int32_t wrap_to_i32(int64_t v)
{
    uint32_t u = (uint32_t)((uint64_t)v & 0xFFFFFFFFu);
    if (u <= 0x7FFFFFFFu)
        return (int32_t)u;
    return (int32_t)(u - 0x80000000u) - (int32_t)0x7FFFFFFF - 1;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Returns 0 on success, -1 on invalid arguments, -2 if a row buffer could not
 * be allocated. */
int oracle_igemm_i16(int64_t m, int64_t n, int64_t k,
                     const int16_t *A, int64_t lda,
                     const int16_t *B, int64_t ldb,
                     int32_t *C, int64_t ldc)
{
    if (m < 0 || n < 0 || k < 0)
        return -1;
    if (m == 0 || n == 0)
        return 0;
    if (ldc < n || (k > 0 && (lda < k || ldb < n)))
        return -1;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < m; ++i) {
        int64_t *acc = (int64_t *)malloc((size_t)n * sizeof(int64_t));
        if (!acc) {
#pragma omp atomic write
            err = -2;
            continue;
        }
        for (int64_t j = 0; j < n; ++j)
            acc[j] = (int64_t)C[i * ldc + j];
        for (int64_t p = 0; p < k; ++p) {
            const int64_t a = (int64_t)A[i * lda + p];
            const int16_t *brow = B + p * ldb;
            for (int64_t j = 0; j < n; ++j)
                acc[j] += a * (int64_t)brow[j];
        }
        for (int64_t j = 0; j < n; ++j)
            C[i * ldc + j] = wrap_to_i32(acc[j]);
        free(acc);
    }
    return err;
}

int oracle_igemm_i8(int64_t m, int64_t n, int64_t k,
                    const int8_t *A, int64_t lda,
                    const int8_t *B, int64_t ldb,
                    int32_t *C, int64_t ldc)
{
    if (m < 0 || n < 0 || k < 0)
        return -1;
    if (m == 0 || n == 0)
        return 0;
    if (ldc < n || (k > 0 && (lda < k || ldb < n)))
        return -1;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < m; ++i) {
        int64_t *acc = (int64_t *)malloc((size_t)n * sizeof(int64_t));
        if (!acc) {
#pragma omp atomic write
            err = -2;
            continue;
        }
        for (int64_t j = 0; j < n; ++j)
            acc[j] = (int64_t)C[i * ldc + j];
        for (int64_t p = 0; p < k; ++p) {
            const int64_t a = (int64_t)A[i * lda + p];
            const int8_t *brow = B + p * ldb;
            for (int64_t j = 0; j < n; ++j)
                acc[j] += a * (int64_t)brow[j];
        }
        for (int64_t j = 0; j < n; ++j)
            C[i * ldc + j] = wrap_to_i32(acc[j]);
        free(acc);
    }
    return err;
}
