/*
 * igemm.h -- integer GEMM  C += A * B  on AMD Instinct MI355X (gfx950).
 *
 * Operation (Sec. 4.1, "GEMM in conventional processor architectures"):
 * A is m x k, B is k x n, C is m x n, and C is updated in place with the
 * product A B. Operands are signed two's-complement int16 (igemm_i16) or
 * int8 (igemm_i8); C is int32. Every product and sum is formed exactly and
 * the updated C[i,j] is the exact value C[i,j] + sum_p A[i,p] B[p,j]
 * reduced modulo 2^32 (two's-complement wraparound). Integer addition modulo
 * 2^32 is associative, so the result is unique and bit-reproducible whatever
 * the blocking, the order of the k loop or the number of workgroups that
 * contribute to one element.
 *
 * Storage: ROW-MAJOR, leading dimensions counted in ELEMENTS:
 *   A[i,p] = A[i*lda + p]   (lda >= max(1,k))
 *   B[p,j] = B[p*ldb + j]   (ldb >= max(1,n))
 *   C[i,j] = C[i*ldc + j]   (ldc >= max(1,n))
 * Elements outside these windows are neither read nor written. A
 * column-major caller uses the identity C^T += B^T A^T: pass
 * (n, m, k, B, ldb, A, lda, C, ldc).
 *
 * Ownership and memory: A, B and C are DEVICE pointers owned by the caller
 * (allocated by any HIP allocator; the library never frees them). C itself
 * is the only output buffer. C must not overlap A or B (not checked).
 * Pointers and leading dimensions of any alignment are accepted; 16-byte
 * aligned rows take the vector-load path, others a slower element path.
 *
 * Memory: the library allocates no device memory and keeps no per-call
 * state; every entry point may be called from several threads at once.
 * Large products run fastest on the packed path (Sec. 4.1's packing of the
 * A and B panels into contiguous buffers, done once per call for the whole
 * operands): pack kernels rearrange A and B into a device workspace, then
 * the main kernel multiplies the packed copies. That workspace always
 * belongs to the caller: igemm_query_plan reports its size
 * (plan.workspace_bytes) and the _ws, pack-once and packed-B calls take it.
 * igemm_i16 / igemm_i8 and the _ex calls have no workspace, so their
 * automatic choice is always one of the kernels that read A and B in place
 * (fused tiles, or the int8 streaming kernel), and an explicit packed kernel
 * returns IGEMM_EINVAL there.
 *
 * Asynchrony and errors: every entry point validates its arguments on the
 * host and returns IGEMM_EINVAL before making any HIP call if they are
 * invalid. Otherwise it enqueues kernels on `stream` (a hipStream_t; NULL is
 * the default stream) and returns IGEMM_OK, or IGEMM_EHIP if a launch was
 * refused. The update of C is complete when the stream is. Faults inside a
 * kernel surface at the caller's next synchronisation. Calls on different
 * streams may run concurrently as long as their C windows do not overlap.
 */
#ifndef IGEMM_H
#define IGEMM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum igemm_status {
    IGEMM_OK = 0,
    IGEMM_EINVAL = -1,  /* invalid argument; nothing was enqueued          */
    IGEMM_EHIP = -2,    /* a HIP runtime call or kernel launch failed      */
    IGEMM_ENOTSUP = -3, /* valid but unsupported (a size beyond 2^31 - 1,  */
                        /* or a grid beyond 2^24 workgroups)              */
    IGEMM_ENOMEM = -4,  /* the caller's workspace is smaller than the plan */
                        /* needs                                           */
    IGEMM_ESCRATCH = -5 /* igemm_i16_noalloc: the call needs more than the */
                        /* static scratch array holds; nothing enqueued   */
} igemm_status;

/*
 * C += A B with int16 operands and int32 wraparound output (Sec. 4.1; the
 * paper's baseline datatype is int16, Sec. 6.1).
 *   m, n, k  >= 0. m == 0 or n == 0: no-op. k == 0: C unchanged.
 *   A        device, m x k int16, row-major, leading dimension lda.
 *   B        device, k x n int16, row-major, leading dimension ldb.
 *   C        device, m x n int32, row-major, leading dimension ldc; read
 *            and written.
 *   stream   hipStream_t or NULL.
 * Returns an igemm_status.
 */
int igemm_i16(int64_t m, int64_t n, int64_t k,
              const int16_t *A, int64_t lda,
              const int16_t *B, int64_t ldb,
              int32_t *C, int64_t ldc, void *stream);

/* Same operation with int8 operands (the lower-precision variant that
 * Sec. 6.1 lists as future work; int8 inputs in [-128, 127]). */
int igemm_i8(int64_t m, int64_t n, int64_t k,
             const int8_t *A, int64_t lda,
             const int8_t *B, int64_t ldb,
             int32_t *C, int64_t ldc, void *stream);

/*
 * Expert variants of the two calls above with an explicit kernel choice, for
 * tuning sweeps and for tests that must reach every kernel:
 *   kernel   -1 = automatic (same as igemm_i16 / igemm_i8), otherwise an
 *            index 0 .. igemm_num_kernels()-1 whose operand type matches the
 *            call (IGEMM_EINVAL otherwise).
 *   split    -1 = automatic, otherwise the number of slices the k range is
 *            cut into (>= 1); slices add their partial results into C with
 *            32-bit atomic adds, which are exact modulo 2^32 in any order.
 *            Values above ceil(k/64) are reduced to it. Packed kernels
 *            need a workspace (the _ws calls; IGEMM_EINVAL here) and
 *            ignore split: one launch per 32768 k elements.
 *            The int8 streaming kernel (few rows of A, B read once) rounds
 *            the k range of a slice up to 4, 8 or 16 k-tiles of 64 when
 *            the rows of A and B are whole 16-byte chunks; up to 4, 8, 16
 *            or 32 (16 at most for more than 16 rows) when B's rows are
 *            whole 8-byte chunks; and to 4 otherwise.
 * Semantics, memory and errors are those of igemm_i16 / igemm_i8.
 */
int igemm_i16_ex(int64_t m, int64_t n, int64_t k,
                 const int16_t *A, int64_t lda,
                 const int16_t *B, int64_t ldb,
                 int32_t *C, int64_t ldc, void *stream,
                 int kernel, int split);
int igemm_i8_ex(int64_t m, int64_t n, int64_t k,
                const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb,
                int32_t *C, int64_t ldc, void *stream,
                int kernel, int split);

/* The launch the library would make for a call (host only, no HIP call).
 * Filled by igemm_query_plan. For packed kernels split is the number of
 * main-kernel launches (one per k chunk of k_chunk elements) and grid the
 * workgroups of each. */
typedef struct igemm_plan {
    int kernel;        /* kernel index                                     */
    int elem_bytes;    /* 2 = int16 operands, 1 = int8                     */
    int bm, bn, bk;    /* workgroup tile of C and k-tile depth (elements)  */
    int split;         /* number of k slices                               */
    int64_t k_chunk;   /* k elements per slice (multiple of bk)            */
    int64_t tiles;     /* C tiles = ceil(m/bm) * ceil(n/bn)                */
    int64_t grid;      /* workgroups launched = tiles * split              */
    int threads;       /* threads per workgroup                            */
    int vec_a, vec_b;  /* 1 if A / B rows take 16-byte vector loads      */
    int limb_products; /* int8 MFMA products per operand pair: 4 or 1      */
    int packed;        /* 1 if operands are packed into a workspace first  */
    int64_t workspace_bytes; /* device workspace the call needs (0: none)  */
    int64_t packed_a_bytes;  /* its A part (packed A and row corrections)  */
    int64_t packed_b_bytes;  /* its B part (packed B, column corrections): */
                             /* the buffer igemm_pack_b_* fills            */
} igemm_plan;

/*
 * Fill *out with the plan for a call with these arguments (pointers are only
 * inspected for alignment, never dereferenced). elem_bytes is 2 for int16,
 * 1 for int8. num_cu is the compute-unit count to plan for (0 = 256, one
 * MI355X). kernel/split as in the _ex calls. The plan is the one a _ws call
 * follows when its workspace holds out->workspace_bytes (it may be a packed
 * kernel); calls without a workspace follow the same rules restricted to the
 * kernels that read A and B in place. Returns IGEMM_OK, IGEMM_EINVAL for
 * invalid arguments, or IGEMM_OK with out->grid == 0 for a no-op call.
 */
int igemm_query_plan(int elem_bytes, int64_t m, int64_t n, int64_t k,
                     const void *A, int64_t lda, const void *B, int64_t ldb,
                     const void *C, int64_t ldc, int num_cu,
                     int kernel, int split, igemm_plan *out);

/*
 * The expert calls with a caller-owned workspace (for callers that manage
 * device memory themselves, e.g. a framework's caching allocator, or that
 * capture the call into a graph):
 *   workspace        device pointer, 256-byte aligned (IGEMM_EINVAL
 *                    otherwise), at least workspace_bytes long, or NULL
 *                    (the call is then the _ex call: no packed path).
 *   workspace_bytes  its size; IGEMM_ENOMEM (nothing enqueued) if it is
 *                    smaller than the plan's workspace_bytes.
 * The workspace is read and written by the kernels enqueued on `stream`; it
 * must not be reused by other work until they have finished. A call whose
 * plan needs no workspace ignores both arguments.
 */
int igemm_i16_ws(int64_t m, int64_t n, int64_t k,
                 const int16_t *A, int64_t lda,
                 const int16_t *B, int64_t ldb,
                 int32_t *C, int64_t ldc, void *stream,
                 int kernel, int split, void *workspace, int64_t workspace_bytes);
int igemm_i8_ws(int64_t m, int64_t n, int64_t k,
                const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb,
                int32_t *C, int64_t ldc, void *stream,
                int kernel, int split, void *workspace, int64_t workspace_bytes);

/*
 * For callers that cannot allocate device memory (code under graph capture,
 * tight serving loops, harnesses that forbid allocation): igemm_i16_ws
 * without a caller workspace. The packed path's workspace is a static device
 * array inside the library, IGEMM_NOALLOC_SCRATCH_BYTES (72 MiB) on each GPU
 * the library runs on, held from the first call on that GPU until the
 * process ends; enough for int16 products up to 4096 x 4096 x 4096 (64.1 MiB
 * of packed operands). Arguments, semantics and errors are those of
 * igemm_i16_ws (kernel and split included), except:
 *   - calls whose plan needs more scratch than the array holds return
 *     IGEMM_ESCRATCH and enqueue nothing (pass kernel = one of the fused
 *     int16 kernels to run such a product with no scratch at all);
 *   - every call on one GPU uses that GPU's single array, which keeps the
 *     last call's contents (the kernels clear what must start at zero):
 *     calls that overlap on one GPU (concurrent streams, or threads without
 *     ordering) RACE and give wrong results; order them on one stream.
 * No hipMalloc, hipFree or other allocating routine is called. The first
 * call on a device looks up the array's device address once
 * (hipGetSymbolAddress) with that device current.
 */
#define IGEMM_NOALLOC_SCRATCH_BYTES ((int64_t)72 << 20)
int igemm_i16_noalloc(int64_t m, int64_t n, int64_t k,
                      const int16_t *A, int64_t lda,
                      const int16_t *B, int64_t ldb,
                      int32_t *C, int64_t ldc, void *stream,
                      int kernel, int split);

/*
 * Pack once, multiply many times. In DL inference one operand is fixed
 * (the weights) and the paper packs it once and reuses it (Sec. 5.1); these
 * calls split the packed path into its two parts so that a caller can keep
 * the packed operands and run only the multiply:
 *   igemm_pack_i16 / igemm_pack_i8  write the packed A and B of the product
 *            C += A B into `workspace` (A and B as in igemm_i16 / igemm_i8;
 *            C is not touched).
 *   igemm_i16_prepacked / igemm_i8_prepacked  run the multiply C += A B on
 *            a workspace filled by the pack call with the same m, n, k, A,
 *            lda and kernel (A itself is read only by int8 plans that use it
 *            in place of a packed copy: 16-byte aligned A, lda a multiple
 *            of 16, m a multiple of 256 and k of 256).
 *   kernel   -1 = the packed kernel of the operand type, otherwise a packed
 *            kernel index of that type (IGEMM_EINVAL for fused kernels).
 *   workspace, workspace_bytes  device memory owned by the caller,
 *            256-byte aligned, at least plan.workspace_bytes of
 *            igemm_query_plan for that kernel (IGEMM_EINVAL for NULL or
 *            misaligned, IGEMM_ENOMEM if too small; nothing is enqueued).
 * Both calls are asynchronous on `stream`; the multiply must be ordered
 * after the pack (same stream, or an event) and the workspace kept intact
 * between them. Sizes beyond the packed path's limits return IGEMM_ENOTSUP.
 */
int igemm_pack_i16(int64_t m, int64_t n, int64_t k,
                   const int16_t *A, int64_t lda,
                   const int16_t *B, int64_t ldb,
                   int kernel, void *workspace, int64_t workspace_bytes, void *stream);
int igemm_pack_i8(int64_t m, int64_t n, int64_t k,
                  const int8_t *A, int64_t lda,
                  const int8_t *B, int64_t ldb,
                  int kernel, void *workspace, int64_t workspace_bytes, void *stream);
int igemm_i16_prepacked(int64_t m, int64_t n, int64_t k,
                        const int16_t *A, int64_t lda,
                        int32_t *C, int64_t ldc,
                        int kernel, const void *workspace, int64_t workspace_bytes,
                        void *stream);
int igemm_i8_prepacked(int64_t m, int64_t n, int64_t k,
                       const int8_t *A, int64_t lda,
                       int32_t *C, int64_t ldc,
                       int kernel, const void *workspace, int64_t workspace_bytes,
                       void *stream);

/*
 * Pack the fixed operand alone (Sec. 5.1: the weights are packed once, the
 * activations on every call). The packed B depends only on n, k, B and the
 * kernel, so one packed B serves products with any m and any A:
 *   igemm_pack_b_i16 / igemm_pack_b_i8  write the packed k x n matrix B
 *            (row-major, leading dimension ldb >= n) into `packed_b`.
 *   igemm_i16_packed_b / igemm_i8_packed_b  C += A B for an m x k A (as in
 *            igemm_i16 / igemm_i8) and a B packed by the call above with
 *            the same n, k and kernel: pack A, then multiply. A's packed
 *            copy goes into `workspace` (caller-owned, 256-byte aligned, at
 *            least plan.packed_a_bytes of igemm_query_plan for (m, n, k)
 *            and that kernel; IGEMM_ENOMEM if smaller). workspace may be
 *            NULL only when that size is 0 (int8 A read in place);
 *            otherwise NULL returns IGEMM_EINVAL.
 *   kernel   -1 = the packed kernel of the operand type, otherwise a packed
 *            kernel index of that type (IGEMM_EINVAL for fused kernels).
 *   packed_b, packed_b_bytes  device memory owned by the caller, 256-byte
 *            aligned, at least plan.packed_b_bytes (IGEMM_EINVAL for NULL or
 *            misaligned, IGEMM_ENOMEM if too small; nothing is enqueued).
 * Asynchronous on `stream`; a multiply must be ordered after the pack and
 * `packed_b` kept intact between them. Multiplies that share one packed B
 * may run concurrently (they only read it). Sizes beyond the packed path's
 * limits return IGEMM_ENOTSUP.
 */
int igemm_pack_b_i16(int64_t n, int64_t k, const int16_t *B, int64_t ldb, int kernel,
                     void *packed_b, int64_t packed_b_bytes, void *stream);
int igemm_pack_b_i8(int64_t n, int64_t k, const int8_t *B, int64_t ldb, int kernel,
                    void *packed_b, int64_t packed_b_bytes, void *stream);
int igemm_i16_packed_b(int64_t m, int64_t n, int64_t k,
                       const int16_t *A, int64_t lda,
                       const void *packed_b, int64_t packed_b_bytes,
                       int32_t *C, int64_t ldc,
                       int kernel, void *workspace, int64_t workspace_bytes,
                       void *stream);
int igemm_i8_packed_b(int64_t m, int64_t n, int64_t k,
                      const int8_t *A, int64_t lda,
                      const void *packed_b, int64_t packed_b_bytes,
                      int32_t *C, int64_t ldc,
                      int kernel, void *workspace, int64_t workspace_bytes,
                      void *stream);

/*
 * Convolution through its GEMM lowering (Sec. 4.2, "GEMM and DL inference":
 * the convolution of a CNN layer is cast as one GEMM by the IM2ROW transform
 * of the input activations, which can be applied on the fly, as part of
 * packing, instead of being materialised). Here the IM2ROW rows are gathered
 * while the operand tiles are staged, so the lowered matrix never exists in
 * memory:
 *
 *   Y[b,oy,ox,co] += sum over fy < r, fx < s, ci < c of
 *                    X[b, oy*stride_h - pad_h + fy*dil_h,
 *                         ox*stride_w - pad_w + fx*dil_w, ci] * W[fy,fx,ci,co]
 *
 * with input positions outside the image counting as zero (zero padding),
 * exact integer sums and the update reduced modulo 2^32 as for igemm_i16.
 * The lowered GEMM has m = n*oh*ow rows (output pixels), n = k columns
 * (output channels) and k = r*s*c (filter taps times input channels); W is
 * exactly its B (k x n row-major) and Y its C.
 *
 * Layouts, all dense and row-major in the order given, DEVICE pointers owned
 * by the caller:
 *   X  n x h x w x c      input activations (NHWC), int16 or int8
 *   W  r x s x c x k      filters (filter row, filter column, input channel,
 *                         output channel), same type
 *   Y  n x oh x ow x k    output activations, int32, updated in place
 * oh = floor((h + 2*pad_h - dil_h*(r-1) - 1) / stride_h) + 1 (0 when the
 * window does not fit), likewise ow; igemm_conv2d_out_dim computes it.
 * Y must not overlap X or W. An input whose channel rows are 16-byte aligned
 * (X 16-byte aligned, c*element size a multiple of 16) is gathered 16 bytes at
 * a time; with horizontal dilation 1 (or s = 1) and s*c at least 7 (int16)
 * or 15 (int8), the s*c contiguous elements a filter row covers are read as
 * runs with unaligned 16-byte loads; any other input element by element.
 *
 * Errors: IGEMM_EINVAL (before any HIP call) for a NULL descriptor, negative
 * extents, r or s < 1, strides or dilations < 1, negative padding, NULL
 * tensors when there is work, or an int16 X at an odd address; IGEMM_ENOTSUP when the input exceeds 2 GiB, the
 * padded image 2^30 elements in a dimension, the lowered k or m 2^31, or the
 * filter tensor's offsets 2 GiB. A call with no output pixel, no output
 * channel or k = 0 returns IGEMM_OK and leaves Y unchanged. Asynchrony as for
 * igemm_i16 (enqueued on `stream`). No workspace is used.
 */
typedef struct igemm_conv2d_desc {
    int64_t n, h, w, c;            /* input batch, height, width, channels */
    int64_t k;                     /* output channels                      */
    int64_t r, s;                  /* filter height and width              */
    int64_t stride_h, stride_w;    /* >= 1                                 */
    int64_t pad_h, pad_w;          /* >= 0, zero padding on both sides     */
    int64_t dil_h, dil_w;          /* >= 1                                 */
} igemm_conv2d_desc;

int igemm_conv2d_i16(const igemm_conv2d_desc *desc, const int16_t *X, const int16_t *W,
                     int32_t *Y, void *stream);
int igemm_conv2d_i8(const igemm_conv2d_desc *desc, const int8_t *X, const int8_t *W,
                    int32_t *Y, void *stream);
/* The same with an explicit kernel (one of the fused 16/32-row, 64x64 or
 * int16 128x128 tile kernels of the operand type; -1 = automatic) and k-slice
 * count (-1 = automatic); elem_bytes 2 (int16) or 1 (int8). For sweeps and
 * tests. */
int igemm_conv2d_ex(int elem_bytes, const igemm_conv2d_desc *desc, const void *X,
                    const void *W, int32_t *Y, void *stream, int kernel, int split);
/* Host-only plan of the lowered GEMM a convolution call would launch
 * (out->kernel = -1 when there is nothing to compute); vec_a reports the
 * 16-byte gather. */
int igemm_conv2d_query_plan(int elem_bytes, const igemm_conv2d_desc *desc, const void *X,
                            const void *W, const void *Y, int num_cu, int kernel, int split,
                            igemm_plan *out);
/* Output extent of one spatial dimension, or -1 for invalid arguments. */
int64_t igemm_conv2d_out_dim(int64_t in, int64_t f, int64_t stride, int64_t pad,
                             int64_t dil);

/*
 * int16-output update with the conversion of the paper's micro-kernel (Sec.
 * 5.2, the listing of the micro-kernel: after its k_c loop the accumulators
 * are converted to int16 by a shift-round-saturate step and added to the
 * int16 micro-tile C_r; in the blocked algorithm, Fig. "baseline GEMM", the
 * micro-kernel runs once per k_c block of loop L2, so the conversion applies
 * to each block's partial product):
 *
 *   for each block of kc consecutive k indices (ascending; the last block may
 *   be shorter; kc = 0, or kc >= k, means one block holding all of k):
 *     acc    = sum over p in the block of A[i,p] * B[p,j]     (exact)
 *     t      = floor((acc + r) / 2^shift), r = 2^(shift-1) when round_half_up
 *              is 1 and shift > 0, else 0 (an arithmetic shift right)
 *     t      = min(max(t, -32768), 32767)                    (saturation)
 *     C[i,j] = (C[i,j] + t) modulo 2^16                        (wraparound)
 *
 * The paper names the conversion and its shift (0 in its listing) but not the
 * rounding or the overflow rule of the add; floor (the plain arithmetic
 * shift), saturation to int16 and a wrapping add are the readings taken, and
 * round_half_up = 1 selects round-half-up instead of floor.
 *
 * A (m x k, lda) and B (k x n, ldb) row-major int16 (igemm_i16_srs) or int8
 * (igemm_i8_srs); C is int16, m x n, row-major with leading dimension ldc,
 * updated in place; DEVICE pointers owned by the caller; any alignment.
 * shift in [0, 47] (the paper's accumulators are 48 bits wide); kc >= 0 and a
 * block of at most 32768 elements. These calls have no workspace: one fused
 * kernel launch per block, enqueued in order on `stream` (igemm_srs_ws with a
 * caller's workspace packs large int16 products first).
 *
 * Errors: IGEMM_EINVAL (before any HIP call, nothing enqueued) as for
 * igemm_i16 and for kc < 0, shift outside [0, 47], round_half_up not 0 or 1;
 * IGEMM_ENOTSUP for blocks longer than 32768 (or extents beyond 2^31 as for
 * igemm_i16). m = 0, n = 0 or k = 0: IGEMM_OK, C unchanged.
 */
int igemm_i16_srs(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                  const int16_t *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                  int round_half_up, void *stream);
int igemm_i8_srs(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                 const int8_t *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                 int round_half_up, void *stream);
/* The same with elem_bytes 2 (int16) or 1 (int8) and an explicit kernel (one
 * of the fused 16/32-row, 64x64 or int16 128x128 tile kernels of the operand
 * type; -1 = automatic; the int16 packed kernel needs igemm_srs_ws, and is
 * refused here with IGEMM_EINVAL). For sweeps and tests. */
int igemm_srs_ex(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                 const void *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                 int round_half_up, void *stream, int kernel);

/*
 * The int16-output update with a caller-owned workspace, for callers that
 * capture the call into a graph or manage device memory themselves (the same
 * operation as igemm_srs_ex, same arguments and errors):
 *   igemm_srs_query  host only (no HIP call): *workspace_bytes = the bytes
 *                    igemm_srs_ws needs for these arguments on a device with
 *                    num_cu compute units (the current device's count, as
 *                    hipDeviceAttributeMultiprocessorCount reports it), 0 when
 *                    the call takes a fused kernel (int8 operands, small
 *                    products, or blocks that are not one block or multiples
 *                    of 256). C and the pointers are only checked, never read.
 *   igemm_srs_ws     workspace: device memory, 256-byte aligned
 *                    (IGEMM_EINVAL otherwise), holding the packed operands
 *                    and the per-block limb sums; at least the queried bytes
 *                    when the packed path is taken (IGEMM_ENOMEM otherwise;
 *                    nothing is enqueued). With workspace NULL the call is
 *                    igemm_srs_ex (fused kernels only). The workspace
 *                    must stay untouched until the call's kernels have run;
 *                    calls that share one workspace must be ordered.
 */
int igemm_srs_query(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A,
                    int64_t lda, const void *B, int64_t ldb, const void *C, int64_t ldc,
                    int64_t kc, int num_cu, int kernel, int64_t *workspace_bytes);
int igemm_srs_ws(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                 const void *B, int64_t ldb, int16_t *C, int64_t ldc, int64_t kc, int shift,
                 int round_half_up, void *stream, int kernel, void *workspace,
                 int64_t workspace_bytes);

/* Number of kernels, and a static name for index `kernel` (NULL if out of
 * range). */
int igemm_num_kernels(void);
const char *igemm_kernel_name(int kernel);

/* Static, human-readable text for a status code. */
const char *igemm_strerror(int status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int igemm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* IGEMM_H */
