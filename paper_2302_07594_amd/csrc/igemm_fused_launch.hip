// Launches of the fused kernels (igemm_tiled.h) for GEMM plans and for
// convolutions lowered by IM2ROW.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm.h"
#include "igemm_internal.h"

namespace igemm {
namespace {

const void *gemm_kernel_fn(int id, bool va, bool vb, bool split) {
    switch (id) {
        case K_I8_256x256:
        case K_I8_128x128: return fused_i8_wide(id, va, vb, split);
        case K_I8_32x256:
        case K_I8_16x256: return fused_i8_rows(id, va, vb, split);
        case K_I16_128x128:
        case K_I16_64x64: return fused_i16_wide(id, va, vb, split);
        case K_I16_32x128:
        case K_I16_16x128: return fused_i16_rows(id, va, vb, split);
        default: return nullptr;
    }
}

const void *conv_kernel_fn(int id, int gather, bool vb, bool split) {
    switch (id) {
        case K_I8_32x256:
        case K_I8_16x256: return fused_conv_i8(id, gather, vb, split);
        case K_I16_128x128:
        case K_I16_64x64:
        case K_I16_32x128:
        case K_I16_16x128: return fused_conv_i16(id, gather, vb, split);
        default: return nullptr;
    }
}

}  // namespace
int launch_tiled(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                 int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                 void *stream) {
    (void)es;
    const void *fn = gemm_kernel_fn(p.kernel, p.vec_a != 0, p.vec_b != 0, p.split > 1);
    if (fn == nullptr) return IGEMM_EINVAL;
    int mi = (int)m, ni = (int)n, ki = (int)k, kc = (int)p.k_chunk;
    int tm = (int)((m + p.bm - 1) / p.bm), tn = (int)((n + p.bn - 1) / p.bn);
    ConvGeom g = {};
    int epi = 0;
    void *args[] = {(void *)&A, (void *)&lda, (void *)&B, (void *)&ldb, (void *)&C,
                    (void *)&ldc, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&kc,
                    (void *)&tm, (void *)&tn, (void *)&g, (void *)&epi};
    hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3(kThreads), args, 0,
                                   (hipStream_t)stream);
    return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

int launch_conv(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const ConvGeom &g,
                int gather, const void *X, const void *W, int32_t *Y, int64_t ldy,
                void *stream) {
    (void)es;
    if (p.kernel == K_I16_SMALL_64x64)
        return launch_small_conv(p, m, n, k, g, gather, X, W, Y, ldy, stream);
    const void *fn = conv_kernel_fn(p.kernel, gather, p.vec_b != 0, p.split > 1);
    if (fn == nullptr) return IGEMM_EINVAL;
    int mi = (int)m, ni = (int)n, ki = (int)k, kc = (int)p.k_chunk;
    int tm = (int)((m + p.bm - 1) / p.bm), tn = (int)((n + p.bn - 1) / p.bn);
    int64_t lda = k, ldb = n;
    ConvGeom gg = g;
    int epi = 0;
    void *args[] = {(void *)&X, (void *)&lda, (void *)&W, (void *)&ldb, (void *)&Y,
                    (void *)&ldy, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&kc,
                    (void *)&tm, (void *)&tn, (void *)&gg, (void *)&epi};
    hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3(kThreads), args, 0,
                                   (hipStream_t)stream);
    return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

int launch_srs(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
               int64_t lda, const void *B, int64_t ldb, int16_t *C, int64_t ldc, int shift,
               int round_half_up, void *stream) {
    (void)es;
    if (p.split != 1) return IGEMM_EINVAL;
    const void *fn = fused_srs(p.kernel, p.vec_a != 0, p.vec_b != 0);
    if (fn == nullptr) return IGEMM_EINVAL;
    int mi = (int)m, ni = (int)n, ki = (int)k, kc = (int)p.k_chunk;
    int tm = (int)((m + p.bm - 1) / p.bm), tn = (int)((n + p.bn - 1) / p.bn);
    ConvGeom g = {};
    int epi = (shift & 0xff) | (round_half_up ? 0x100 : 0);
    int32_t *Cp = (int32_t *)C;  // the kernel reads it as int16 for this variant
    void *args[] = {(void *)&A, (void *)&lda, (void *)&B, (void *)&ldb, (void *)&Cp,
                    (void *)&ldc, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&kc,
                    (void *)&tm, (void *)&tn, (void *)&g, (void *)&epi};
    hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3(kThreads), args, 0,
                                   (hipStream_t)stream);
    return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

}  // namespace igemm
