// The C entry points: validation, planning and dispatch to the fused tiled
// kernels, the streaming kernel or (on a caller's workspace) the
// pack-then-multiply path. The library allocates no device memory.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "igemm.h"
#include "igemm_internal.h"

namespace igemm {
namespace {

constexpr int kMaxDevices = 64;

// Compute units per device, looked up once per device. Relaxed atomics: a
// racing first call may query twice, and both store the same value.
std::atomic<int> g_num_cu[kMaxDevices];

int num_cu_of_current_device() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    const bool cacheable = dev >= 0 && dev < kMaxDevices;
    if (cacheable) {
        const int c = g_num_cu[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cu <= 0)
        cu = 256;
    if (cacheable) g_num_cu[dev].store(cu, std::memory_order_relaxed);
    return cu;
}

// Scratch of igemm_i16_noalloc: one array per device, loaded with the code
// object and kept until the process ends. In host code `scratch` names a
// host-side stand-in, not device memory: host code uses only the device
// address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[IGEMM_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;                       // guards first look-ups only
std::atomic<void *> g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array (looked up once per
// device, with that device current), or nullptr on failure.
void *scratch_of_current_device() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p != nullptr) return p;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    return p;
}

// The one-call workspace holds the A part, then the B part.
int pack_both(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
              int64_t lda, const void *B, int64_t ldb, void *ws, void *stream) {
    char *wb = (char *)ws + p.packed_a_bytes;
    // int16 always packs A, and that kernel clears B's column corrections
    // before pack_b adds into them; int8 has no corrections.
    int st = launch_pack_a(es, p, m, n, k, A, lda, ws, wb, stream);
    if (st != IGEMM_OK) return st;
    return launch_pack_b(es, p, m, n, k, A, lda, B, ldb, wb, false, stream);
}
int multiply_both(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, int32_t *C, int64_t ldc, const void *ws, void *stream) {
    return launch_multiply(es, p, m, n, k, A, lda, C, ldc, ws,
                           (const char *)ws + p.packed_a_bytes, stream);
}

int run(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
        int64_t ldb, int32_t *C, int64_t ldc, void *stream, int kernel, int split,
        void *workspace, int64_t workspace_bytes) {
    int st = validate(es, m, n, k, A, lda, B, ldb, C, ldc);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    if (kernel < -1 || kernel >= K_COUNT || split < -1 || split == 0) return IGEMM_EINVAL;
    if (kernel >= 0 && kKernels[kernel].es != es) return IGEMM_EINVAL;
    if (workspace != nullptr && ((uintptr_t)workspace % 256 != 0 || workspace_bytes < 0))
        return IGEMM_EINVAL;
    // The library allocates nothing: the packed path runs only on a
    // caller's workspace; without one, automatic choice keeps to the kernels
    // that read the operands in place, and an explicit packed kernel is
    // refused.
    const bool have_ws = workspace != nullptr;
    if (kernel >= 0 && kKernels[kernel].packed && !have_ws) return IGEMM_EINVAL;
    igemm_plan p;
    st = make_plan(es, m, n, k, A, lda, B, ldb, ldc, num_cu_of_current_device(), kernel, split,
                   have_ws, &p);
    if (st != IGEMM_OK) return st;
    if (p.kernel == K_I8_STREAM || p.kernel == K_I16_STREAM)
        return launch_stream(p, m, n, k, A, lda, B, ldb, C, ldc, stream);
    if (p.kernel == K_I16_DIRECT_128x128 || p.kernel == K_I8_DIRECT_256x256)
        return launch_direct(es, p, m, n, k, A, lda, B, ldb, C, ldc, stream);
    if (p.kernel == K_I16_SMALL_64x64)
        return launch_small(p, m, n, k, A, lda, B, ldb, C, ldc, stream);
    if (!p.packed) return launch_tiled(es, p, m, n, k, A, lda, B, ldb, C, ldc, stream);
    if (workspace_bytes < p.workspace_bytes) return IGEMM_ENOMEM;
    st = pack_both(es, p, m, n, k, A, lda, B, ldb, workspace, stream);
    if (st != IGEMM_OK) return st;
    return multiply_both(es, p, m, n, k, A, lda, C, ldc, workspace, stream);
}

// Plan of a pack-once call: the packed kernel of the operand type (kernel -1)
// or the given packed kernel; the B and C arguments only need to pass the
// argument checks.
int packed_plan(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                const void *B, int64_t ldb, int64_t ldc, int kernel, const void *workspace,
                int64_t workspace_bytes, igemm_plan *p) {
    if (kernel < -1 || kernel >= K_COUNT) return IGEMM_EINVAL;
    if (kernel == -1) kernel = es == 2 ? K_I16_PACKED_128x128 : K_I8_PACKED_256x256;
    if (kKernels[kernel].es != es || !kKernels[kernel].packed) return IGEMM_EINVAL;
    if (workspace == nullptr || (uintptr_t)workspace % 256 != 0 || workspace_bytes < 0)
        return IGEMM_EINVAL;
    int st = make_plan(es, m, n, k, A, lda, B, ldb, ldc, 256, kernel, -1, true, p);
    if (st != IGEMM_OK) return st;
    return workspace_bytes < p->workspace_bytes ? IGEMM_ENOMEM : IGEMM_OK;
}

int run_pack(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
             int64_t ldb, int kernel, void *workspace, int64_t workspace_bytes, void *stream) {
    // C is not touched by packing: a placeholder passes the checks.
    const void *fake_c = (const void *)(uintptr_t)4096;
    int st = validate(es, m, n, k, A, lda, B, ldb, fake_c, n > 0 ? n : 1);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    igemm_plan p;
    st = packed_plan(es, m, n, k, A, lda, B, ldb, n, kernel, workspace, workspace_bytes, &p);
    if (st != IGEMM_OK) return st;
    return pack_both(es, p, m, n, k, A, lda, B, ldb, workspace, stream);
}

int run_prepacked(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                  int32_t *C, int64_t ldc, int kernel, const void *workspace,
                  int64_t workspace_bytes, void *stream) {
    // B was consumed by the pack call: a placeholder passes the checks.
    const void *fake_b = (const void *)(uintptr_t)4096;
    int st = validate(es, m, n, k, A, lda, fake_b, n > 0 ? n : 1, C, ldc);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    igemm_plan p;
    st = packed_plan(es, m, n, k, A, lda, fake_b, n, ldc, kernel, workspace, workspace_bytes, &p);
    if (st != IGEMM_OK) return st;
    return multiply_both(es, p, m, n, k, A, lda, C, ldc, workspace, stream);
}

// Pack B alone (the fixed operand); its layout depends on n, k and the kernel
// only.
int run_pack_b(int es, int64_t n, int64_t k, const void *B, int64_t ldb, int kernel,
               void *packed_b, int64_t packed_b_bytes, void *stream) {
    const void *fake = (const void *)(uintptr_t)4096;
    int st = validate(es, 1, n, k, fake, k > 0 ? k : 1, B, ldb, fake, n > 0 ? n : 1);
    if (st != IGEMM_OK) return st;
    if (n == 0 || k == 0) return IGEMM_OK;
    igemm_plan p;
    st = packed_plan(es, 1, n, k, fake, k, B, ldb, n, kernel, packed_b, 0, &p);
    if (st != IGEMM_OK && st != IGEMM_ENOMEM) return st;
    if (packed_b_bytes < p.packed_b_bytes) return IGEMM_ENOMEM;
    return launch_pack_b(es, p, 1, n, k, fake, k, B, ldb, packed_b, true, stream);
}

// C += A B with B packed by run_pack_b: pack A into the caller's workspace
// (none is needed for int8 A that the multiply reads in place), then
// multiply.
int run_packed_b(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                 const void *packed_b, int64_t packed_b_bytes, int32_t *C, int64_t ldc,
                 int kernel, void *workspace, int64_t workspace_bytes, void *stream) {
    const void *fake = (const void *)(uintptr_t)4096;
    int st = validate(es, m, n, k, A, lda, fake, n > 0 ? n : 1, C, ldc);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    if (workspace != nullptr && ((uintptr_t)workspace % 256 != 0 || workspace_bytes < 0))
        return IGEMM_EINVAL;
    igemm_plan p;
    st = packed_plan(es, m, n, k, A, lda, fake, n, ldc, kernel, packed_b, 0, &p);
    if (st != IGEMM_OK && st != IGEMM_ENOMEM) return st;
    if (packed_b_bytes < p.packed_b_bytes) return IGEMM_ENOMEM;
    if (p.packed_a_bytes > 0 && workspace == nullptr) return IGEMM_EINVAL;
    if (workspace_bytes < p.packed_a_bytes) return IGEMM_ENOMEM;
    st = launch_pack_a(es, p, m, n, k, A, lda, workspace, nullptr, stream);
    if (st != IGEMM_OK) return st;
    return launch_multiply(es, p, m, n, k, A, lda, C, ldc, workspace, packed_b, stream);
}

// Y += conv(X, W) through the fused kernels with IM2ROW gathering of A.
int run_conv(int es, const igemm_conv2d_desc *d, const void *X, const void *W, int32_t *Y,
             void *stream, int kernel, int split) {
    igemm_plan p;
    ConvGeom g;
    int gather = 0;
    // Validate without touching the device, then plan for its CU count.
    int st = make_conv_plan(es, d, X, W, Y, 0, kernel, split, &p, &g, &gather);
    if (st != IGEMM_OK || p.kernel < 0) return st;
    st = make_conv_plan(es, d, X, W, Y, num_cu_of_current_device(), kernel, split, &p, &g,
                        &gather);
    if (st != IGEMM_OK) return st;
    const int64_t oh = conv_out_dim(d->h, d->r, d->stride_h, d->pad_h, d->dil_h);
    const int64_t ow = conv_out_dim(d->w, d->s, d->stride_w, d->pad_w, d->dil_w);
    return launch_conv(es, p, d->n * oh * ow, d->k, d->r * d->s * d->c, g, gather, X, W, Y, d->k,
                       stream);
}

// int16-output update: the packed path for large int16 products whose blocks
// fall on the packed k-tiles (one block, or blocks of a multiple of 256, at
// most 64), else one fused launch per k block of kc elements, in order. All
// blocks are planned before the first launch, so an error enqueues nothing.
int srs_check(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
              int64_t ldb, const void *C, int64_t ldc, int64_t kc, int shift, int round_half_up,
              int kernel) {
    int st = validate(es, m, n, k, A, lda, B, ldb, C, ldc);
    if (st != IGEMM_OK) return st;
    if (kc < 0 || shift < 0 || shift > 47 || (round_half_up != 0 && round_half_up != 1) ||
        kernel < -1 || kernel >= K_COUNT)
        return IGEMM_EINVAL;
    return IGEMM_OK;
}
bool srs_packed_ok(int es, int64_t k, int64_t kc, int64_t *blk, int64_t *nblocks) {
    *blk = (kc == 0 || kc > k) ? k : kc;
    *nblocks = (k + *blk - 1) / *blk;
    return es == 2 && *nblocks <= 64 && (*nblocks == 1 || *blk % 256 == 0);
}
// Plans the packed path (pp->packed false when the fused path is taken) and
// returns the workspace it needs in *need.
int srs_packed_plan(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                    const void *B, int64_t ldb, int64_t ldc, int64_t kc, int num_cu, int kernel,
                    bool can_pack, igemm_plan *pp, int64_t *need) {
    *need = 0;
    pp->packed = 0;
    int64_t blk, nblocks;
    const bool packed_ok = srs_packed_ok(es, k, kc, &blk, &nblocks);
    if (kernel == K_I16_PACKED_128x128 && (!packed_ok || !can_pack)) return IGEMM_EINVAL;
    if (blk > kMaxKChunk) return IGEMM_ENOTSUP;
    if (kernel != K_I16_PACKED_128x128 && !(kernel < 0 && packed_ok)) return IGEMM_OK;
    int st = make_plan(es, m, n, k, A, lda, B, ldb, ldc, num_cu, kernel < 0 ? -1 : kernel, -1,
                       can_pack, pp);
    // A large product the GEMM plan gives to the direct kernel (short k)
    // still takes the packed path here: only the packed kernel has the
    // in-kernel int16-output conversion.
    if (st == IGEMM_OK && kernel < 0 && can_pack && pp->kernel == K_I16_DIRECT_128x128)
        st = make_plan(es, m, n, k, A, lda, B, ldb, ldc, num_cu, K_I16_PACKED_128x128, -1, true,
                       pp);
    if (st != IGEMM_OK) return st;
    if (pp->packed) *need = pp->workspace_bytes + srs_sums_bytes(*pp, m, n, k, nblocks, A, lda);
    return IGEMM_OK;
}
int run_srs(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
            int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift, int round_half_up,
            void *stream, int kernel, void *workspace = nullptr, int64_t workspace_bytes = 0) {
    int st = srs_check(es, m, n, k, A, lda, B, ldb, C, ldc, kc, shift, round_half_up, kernel);
    if (st != IGEMM_OK) return st;
    if (workspace != nullptr && ((uintptr_t)workspace % 256 != 0 || workspace_bytes < 0))
        return IGEMM_EINVAL;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    int64_t blk, nblocks;
    const bool packed_ok = srs_packed_ok(es, k, kc, &blk, &nblocks);
    if (blk > kMaxKChunk) return IGEMM_ENOTSUP;
    if (kernel == K_I16_PACKED_128x128 && !packed_ok) return IGEMM_EINVAL;
    if (kernel == K_I16_PACKED_128x128 || (kernel < 0 && packed_ok)) {
        // The packed path needs the caller's workspace.
        const bool can_pack = workspace != nullptr;
        igemm_plan pp;
        int64_t need = 0;
        st = srs_packed_plan(es, m, n, k, A, lda, B, ldb, ldc, kc, num_cu_of_current_device(),
                             kernel, can_pack, &pp, &need);
        if (st != IGEMM_OK) return st;
        if (pp.packed) {
            if (workspace_bytes < need) return IGEMM_ENOMEM;
            // the pack kernels also take the per-block limb sums
            char *wb = (char *)workspace + pp.packed_a_bytes;
            uint32_t *sums = (uint32_t *)((char *)workspace + pp.workspace_bytes);
            st = launch_pack_a(es, pp, m, n, k, A, lda, workspace, wb, stream, sums, blk,
                               nblocks);
            if (st != IGEMM_OK) return st;
            st = launch_pack_b(es, pp, m, n, k, A, lda, B, ldb, wb, false, stream, sums, blk,
                               nblocks);
            if (st != IGEMM_OK) return st;
            return launch_srs_packed(pp, m, n, k, blk, nblocks, A, lda, C, ldc, workspace, wb,
                                     sums, shift, round_half_up, stream);
        }
    }
    for (int pass = 0; pass < 2; ++pass) {
        const int num_cu = pass == 0 ? 0 : num_cu_of_current_device();
        for (int64_t q = 0; q < nblocks; ++q) {
            const int64_t p0 = q * blk;
            const int64_t kb = p0 + blk < k ? blk : k - p0;
            const char *Aq = (const char *)A + p0 * es;
            const char *Bq = (const char *)B + p0 * ldb * es;
            igemm_plan p;
            st = make_srs_plan(es, m, n, kb, Aq, lda, Bq, ldb, ldc, num_cu, kernel, &p);
            if (st != IGEMM_OK) return st;
            if (pass == 1) {
                st = launch_srs(es, p, m, n, kb, Aq, lda, Bq, ldb, C, ldc, shift, round_half_up,
                                stream);
                if (st != IGEMM_OK) return st;
            }
        }
    }
    return IGEMM_OK;
}

}  // namespace
}  // namespace igemm

extern "C" {

int igemm_i16_srs(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                  const int16_t *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                  int round_half_up, void *stream) {
    return igemm::run_srs(2, m, n, k, A, lda, B, ldb, C, ldc, kc, shift, round_half_up, stream,
                          -1);
}

int igemm_i8_srs(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                 const int8_t *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                 int round_half_up, void *stream) {
    return igemm::run_srs(1, m, n, k, A, lda, B, ldb, C, ldc, kc, shift, round_half_up, stream,
                          -1);
}

int igemm_srs_ex(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                 const void *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                 int round_half_up, void *stream, int kernel) {
    if (elem_bytes != 1 && elem_bytes != 2) return IGEMM_EINVAL;
    return igemm::run_srs(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc, shift, round_half_up,
                          stream, kernel);
}

int igemm_srs_query(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A,
                    int64_t lda, const void *B, int64_t ldb, const void *C, int64_t ldc,
                    int64_t kc, int num_cu, int kernel, int64_t *workspace_bytes) {
    if (workspace_bytes == nullptr || (elem_bytes != 1 && elem_bytes != 2) || num_cu < 0)
        return IGEMM_EINVAL;
    *workspace_bytes = 0;
    int st = igemm::srs_check(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc, 0, 0, kernel);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    igemm_plan pp;
    return igemm::srs_packed_plan(elem_bytes, m, n, k, A, lda, B, ldb, ldc, kc, num_cu, kernel,
                                  true, &pp, workspace_bytes);
}

int igemm_srs_ws(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                 const void *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                 int round_half_up, void *stream, int kernel, void *workspace,
                 int64_t workspace_bytes) {
    if (elem_bytes != 1 && elem_bytes != 2) return IGEMM_EINVAL;
    return igemm::run_srs(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc, shift, round_half_up,
                          stream, kernel, workspace, workspace_bytes);
}

int igemm_conv2d_i16(const igemm_conv2d_desc *desc, const int16_t *X, const int16_t *W,
                     int32_t *Y, void *stream) {
    return igemm::run_conv(2, desc, X, W, Y, stream, -1, -1);
}

int igemm_conv2d_i8(const igemm_conv2d_desc *desc, const int8_t *X, const int8_t *W, int32_t *Y,
                    void *stream) {
    return igemm::run_conv(1, desc, X, W, Y, stream, -1, -1);
}

int igemm_conv2d_ex(int elem_bytes, const igemm_conv2d_desc *desc, const void *X, const void *W,
                    int32_t *Y, void *stream, int kernel, int split) {
    return igemm::run_conv(elem_bytes, desc, X, W, Y, stream, kernel, split);
}

int igemm_i16(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
              const int16_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream) {
    return igemm::run(2, m, n, k, A, lda, B, ldb, C, ldc, stream, -1, -1, nullptr, 0);
}

int igemm_i8(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda, const int8_t *B,
             int64_t ldb, int32_t *C, int64_t ldc, void *stream) {
    return igemm::run(1, m, n, k, A, lda, B, ldb, C, ldc, stream, -1, -1, nullptr, 0);
}

int igemm_i16_ex(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                 const int16_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                 int kernel, int split) {
    return igemm::run(2, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split, nullptr, 0);
}

int igemm_i8_ex(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                int kernel, int split) {
    return igemm::run(1, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split, nullptr, 0);
}

int igemm_i16_ws(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                 const int16_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                 int kernel, int split, void *workspace, int64_t workspace_bytes) {
    return igemm::run(2, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split, workspace,
                      workspace_bytes);
}

int igemm_i16_noalloc(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                      const int16_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                      int kernel, int split) {
    // Argument errors first, before any HIP call (as igemm_i16_ws).
    int st = igemm::validate(2, m, n, k, A, lda, B, ldb, C, ldc);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    if (kernel < -1 || kernel >= igemm::K_COUNT || split < -1 || split == 0) return IGEMM_EINVAL;
    if (kernel >= 0 && igemm::kKernels[kernel].es != 2) return IGEMM_EINVAL;
    igemm_plan p;
    st = igemm::make_plan(2, m, n, k, A, lda, B, ldb, ldc, igemm::num_cu_of_current_device(),
                          kernel, split, true, &p);
    if (st != IGEMM_OK) return st;
    if (p.workspace_bytes > IGEMM_NOALLOC_SCRATCH_BYTES) return IGEMM_ESCRATCH;
    void *ws = igemm::scratch_of_current_device();
    if (ws == nullptr) return IGEMM_EHIP;
    // The same plan as above, with the scratch array as its workspace.
    return igemm::run(2, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split, ws,
                      IGEMM_NOALLOC_SCRATCH_BYTES);
}

int igemm_i8_ws(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                int kernel, int split, void *workspace, int64_t workspace_bytes) {
    return igemm::run(1, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split, workspace,
                      workspace_bytes);
}

int igemm_pack_i16(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                   const int16_t *B, int64_t ldb, int kernel, void *workspace,
                   int64_t workspace_bytes, void *stream) {
    return igemm::run_pack(2, m, n, k, A, lda, B, ldb, kernel, workspace, workspace_bytes, stream);
}

int igemm_pack_i8(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                  const int8_t *B, int64_t ldb, int kernel, void *workspace,
                  int64_t workspace_bytes, void *stream) {
    return igemm::run_pack(1, m, n, k, A, lda, B, ldb, kernel, workspace, workspace_bytes, stream);
}

int igemm_i16_prepacked(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                        int32_t *C, int64_t ldc, int kernel, const void *workspace,
                        int64_t workspace_bytes, void *stream) {
    return igemm::run_prepacked(2, m, n, k, A, lda, C, ldc, kernel, workspace, workspace_bytes,
                                stream);
}

int igemm_i8_prepacked(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                       int32_t *C, int64_t ldc, int kernel, const void *workspace,
                       int64_t workspace_bytes, void *stream) {
    return igemm::run_prepacked(1, m, n, k, A, lda, C, ldc, kernel, workspace, workspace_bytes,
                                stream);
}

int igemm_pack_b_i16(int64_t n, int64_t k, const int16_t *B, int64_t ldb, int kernel,
                     void *packed_b, int64_t packed_b_bytes, void *stream) {
    return igemm::run_pack_b(2, n, k, B, ldb, kernel, packed_b, packed_b_bytes, stream);
}

int igemm_pack_b_i8(int64_t n, int64_t k, const int8_t *B, int64_t ldb, int kernel,
                    void *packed_b, int64_t packed_b_bytes, void *stream) {
    return igemm::run_pack_b(1, n, k, B, ldb, kernel, packed_b, packed_b_bytes, stream);
}

int igemm_i16_packed_b(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                       const void *packed_b, int64_t packed_b_bytes, int32_t *C, int64_t ldc,
                       int kernel, void *workspace, int64_t workspace_bytes, void *stream) {
    return igemm::run_packed_b(2, m, n, k, A, lda, packed_b, packed_b_bytes, C, ldc, kernel,
                               workspace, workspace_bytes, stream);
}

int igemm_i8_packed_b(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                      const void *packed_b, int64_t packed_b_bytes, int32_t *C, int64_t ldc,
                      int kernel, void *workspace, int64_t workspace_bytes, void *stream) {
    return igemm::run_packed_b(1, m, n, k, A, lda, packed_b, packed_b_bytes, C, ldc, kernel,
                               workspace, workspace_bytes, stream);
}

}  // extern "C"
