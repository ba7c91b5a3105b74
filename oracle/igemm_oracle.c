/*
 * CPU oracle for integer GEMM  C += A * B, for the convolution that the
 * paper lowers to it, and for the int16-output variant with the paper's
 * shift-round-saturate conversion (both further down) -- TEST
 * INFRASTRUCTURE ONLY.
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

/*
 * Convolution  Y += conv(X, W)  -- the operation that the lowering of Sec. 4.2
 * (GEMM and DL inference) turns into one GEMM: IM2ROW rewrites the input
 * activations as a matrix with one row per output pixel and one column per
 * (filter row, filter column, input channel), and the filters as a matrix with
 * one row per such triple and one column per output channel. The oracle does
 * not build that matrix: it is the direct definition, summing over the filter
 * window and the input channels for every output pixel and channel.
 *
 * Layouts (all dense, row-major in the order given):
 *   X  n x h x w x c           input activations (NHWC)
 *   W  r x s x c x k           filters (filter row, filter column, input
 *                              channel, output channel)
 *   Y  n x oh x ow x k         output activations, updated in place
 * with oh = (h + 2 pad_h - dil_h (r - 1) - 1) / stride_h + 1 (floor; 0 when the
 * numerator is negative) and likewise ow. Output pixel (oy, ox) reads input
 * row oy * stride_h - pad_h + fy * dil_h and column ox * stride_w - pad_w +
 * fx * dil_w for filter position (fy, fx); positions outside the input are
 * zero (zero padding). Exact int64 sums, reduced modulo 2^32 once at the end.
 */
int64_t oracle_conv2d_out_dim(int64_t in, int64_t f, int64_t stride, int64_t pad, int64_t dil)
{
    if (in < 0 || f < 1 || stride < 1 || pad < 0 || dil < 1)
        return -1;
    const int64_t span = in + 2 * pad - dil * (f - 1) - 1;
    return span < 0 ? 0 : span / stride + 1;
}

#define ORACLE_CONV2D(NAME, T)                                                               \
    int NAME(int64_t n, int64_t h, int64_t w, int64_t c, int64_t k, int64_t r, int64_t s,  \
             int64_t stride_h, int64_t stride_w, int64_t pad_h, int64_t pad_w,             \
             int64_t dil_h, int64_t dil_w, const T *X, const T *W, int32_t *Y)             \
    {                                                                                        \
        if (n < 0 || c < 0 || k < 0)                                                         \
            return -1;                                                                       \
        const int64_t oh = oracle_conv2d_out_dim(h, r, stride_h, pad_h, dil_h);              \
        const int64_t ow = oracle_conv2d_out_dim(w, s, stride_w, pad_w, dil_w);              \
        if (oh < 0 || ow < 0)                                                                \
            return -1;                                                                       \
        int err = 0;                                                                         \
        _Pragma("omp parallel for collapse(2) schedule(dynamic, 1)")                         \
        for (int64_t b = 0; b < n; ++b)                                                      \
            for (int64_t oy = 0; oy < oh; ++oy) {                                            \
                int64_t *acc = (int64_t *)malloc((size_t)(k > 0 ? k : 1) * sizeof(int64_t)); \
                if (!acc) {                                                                  \
                    _Pragma("omp atomic write") err = -2;                                    \
                    continue;                                                                \
                }                                                                            \
                for (int64_t ox = 0; ox < ow; ++ox) {                                        \
                    int32_t *y = Y + ((b * oh + oy) * ow + ox) * k;                          \
                    for (int64_t co = 0; co < k; ++co)                                       \
                        acc[co] = (int64_t)y[co];                                            \
                    for (int64_t fy = 0; fy < r; ++fy) {                                     \
                        const int64_t iy = oy * stride_h - pad_h + fy * dil_h;               \
                        if (iy < 0 || iy >= h)                                               \
                            continue;                                                        \
                        for (int64_t fx = 0; fx < s; ++fx) {                                 \
                            const int64_t ix = ox * stride_w - pad_w + fx * dil_w;           \
                            if (ix < 0 || ix >= w)                                           \
                                continue;                                                    \
                            const T *xp = X + ((b * h + iy) * w + ix) * c;                   \
                            const T *wp = W + (fy * s + fx) * c * k;                         \
                            for (int64_t ci = 0; ci < c; ++ci) {                             \
                                const int64_t xv = (int64_t)xp[ci];                          \
                                const T *wrow = wp + ci * k;                                 \
                                for (int64_t co = 0; co < k; ++co)                           \
                                    acc[co] += xv * (int64_t)wrow[co];                       \
                            }                                                                \
                        }                                                                    \
                    }                                                                        \
                    for (int64_t co = 0; co < k; ++co)                                       \
                        y[co] = wrap_to_i32(acc[co]);                                        \
                }                                                                            \
                free(acc);                                                                   \
            }                                                                                \
        return err;                                                                          \
    }

ORACLE_CONV2D(oracle_conv2d_i16, int16_t)
ORACLE_CONV2D(oracle_conv2d_i8, int8_t)

/*
 * int16-output GEMM with the conversion of the paper's micro-kernel -- the
 * epilogue of the listing of Sec. 5.2 (Fig. "simplified version of the
 * micro-kernel"): after the k_c loop, each accumulator is converted to int16
 * with a shift-round-saturate step and the converted micro-tile is added to
 * the int16 micro-tile C_r. In the blocked algorithm (Fig. "baseline GEMM")
 * the micro-kernel runs once per k_c block of loop L2, so the conversion is
 * applied to each block's partial product separately.
 *
 * The paper does not define the conversion beyond its name and shift (0 in
 * the listing), nor the addition's overflow rule; the readings taken:
 *   for each block q of kc consecutive k indices (ascending; the last block
 *   may be shorter; kc = 0 means one block holding all of k):
 *     acc   = sum over p in block q of A[i,p] * B[p,j]     (exact, int64)
 *     t     = floor((acc + r) / 2^shift), r = 2^(shift-1) if round_half_up
 *             and shift > 0, else 0  (floor: the rounding of an arithmetic
 *             shift)
 *     t     = min(max(t, -32768), 32767)                   (saturation)
 *     C[i,j] = (C[i,j] + t) modulo 2^16, as int16          (wraparound)
 * Storage as for the GEMM oracle above, C being int16.
 *
 * Returns 0, or -1 for invalid arguments (negative sizes, kc < 0, shift
 * outside [0, 47], leading dimensions too small).
 */
static int64_t floor_div_pow2(int64_t v, int shift)
{
    const int64_t d = (int64_t)1 << shift;
    int64_t q = v / d; /* truncates toward zero */
    if (v % d != 0 && v < 0)
        q -= 1;
    return q;
}

static int16_t wrap_to_i16(int64_t v)
{
    uint16_t u = (uint16_t)((uint64_t)v & 0xFFFFu);
    if (u <= 0x7FFFu)
        return (int16_t)u;
    return (int16_t)((int32_t)u - 65536);
}

#define ORACLE_SRS(NAME, T)                                                                   \
    int NAME(int64_t m, int64_t n, int64_t k, const T *A, int64_t lda, const T *B, int64_t ldb, \
             int16_t *C, int64_t ldc, int64_t kc, int shift, int round_half_up)              \
    {                                                                                         \
        if (m < 0 || n < 0 || k < 0 || kc < 0 || shift < 0 || shift > 47)                     \
            return -1;                                                                        \
        if (m == 0 || n == 0)                                                                 \
            return 0;                                                                         \
        if (ldc < n || (k > 0 && (lda < k || ldb < n)))                                       \
            return -1;                                                                        \
        const int64_t blk = kc == 0 ? k : kc;                                                 \
        const int64_t half = (round_half_up && shift > 0) ? ((int64_t)1 << (shift - 1)) : 0;  \
        _Pragma("omp parallel for schedule(dynamic, 1)")                                      \
        for (int64_t i = 0; i < m; ++i) {                                                     \
            for (int64_t j = 0; j < n; ++j) {                                                 \
                int64_t c = (int64_t)C[i * ldc + j];                                          \
                for (int64_t p0 = 0; p0 < k; p0 += blk) {                                     \
                    const int64_t p1 = p0 + blk < k ? p0 + blk : k;                           \
                    int64_t acc = 0;                                                          \
                    for (int64_t p = p0; p < p1; ++p)                                         \
                        acc += (int64_t)A[i * lda + p] * (int64_t)B[p * ldb + j];             \
                    int64_t t = floor_div_pow2(acc + half, shift);                            \
                    if (t > 32767)                                                            \
                        t = 32767;                                                            \
                    if (t < -32768)                                                           \
                        t = -32768;                                                           \
                    c = (int64_t)wrap_to_i16(c + t);                                          \
                }                                                                             \
                C[i * ldc + j] = (int16_t)c;                                                  \
            }                                                                                 \
        }                                                                                     \
        return 0;                                                                             \
    }

ORACLE_SRS(oracle_igemm_srs_i16, int16_t)
ORACLE_SRS(oracle_igemm_srs_i8, int8_t)
