// Internal declarations shared by the host planner and the kernel launcher.
#pragma once

#include <stdint.h>

#include "igemm.h"

namespace igemm {

// One kernel family: operand size, workgroup tile of C and the tile of C
// each wave owns (four waves per workgroup; eight for i8_packed_256x256).
// Packed kernels multiply operands that a pack step has first rearranged
// into a workspace.
struct KernelDesc {
    const char *name;
    int es;      // operand bytes: 2 = int16 (two int8 limb planes), 1 = int8
    int bm, bn;  // workgroup tile of C
    int wm, wn;  // wave tile of C
    bool packed;
};

enum KernelId {
    K_I8_256x256 = 0,
    K_I8_128x128,
    K_I8_32x256,
    K_I8_16x256,
    K_I16_128x128,
    K_I16_64x64,
    K_I16_32x128,
    K_I16_16x128,
    K_I8_PACKED_256x256,
    K_I16_PACKED_128x128,
    K_I8_STREAM,
    K_I16_DIRECT_128x128,
    K_I8_DIRECT_256x256,
    K_I16_SMALL_64x64,
    K_I16_STREAM,
    K_COUNT
};

constexpr int kBK = 64;        // k elements per k-tile (one 16x16x64 MFMA step)
constexpr int kThreads = 256;  // four waves of 64
// Largest k range one workgroup accumulates in int32 MFMA accumulators. Each
// int16 limb sum is bounded by 2^15 per k element (2^14 for int8), so partial
// sums stay below 2^31 and never depend on how the hardware treats overflow.
constexpr int64_t kMaxKChunk = 32768;

extern const KernelDesc kKernels[K_COUNT];

// Workspace of the packed path, in two parts (byte offsets from 256-byte
// aligned bases), so that B can be packed once and reused:
//   A part (a_bytes): es planes of m_pad rows (int16: high limb, then offset
//     low limb), absent for int8 A that is already aligned and tile-shaped,
//     then m_pad row corrections (int16);
//   B part (b_bytes): es planes of n_pad rows (the columns of B), then n_pad
//     column corrections (int16; pack_b adds each k slice's column sums).
// Planes are k-contiguous int8 rows of k_pad bytes, zero beyond k. The
// one-call workspace is the A part followed by the B part.
struct PackedLayout {
    int64_t m_pad, n_pad, k_pad;
    int64_t kspan;     // k rows per pack_b workgroup
    int b_slices;      // k slices of pack_b
    bool pack_a;
    int64_t off_a, off_corr_a, a_bytes;  // within the A part
    int64_t off_b, off_corr_b, b_bytes;  // within the B part
    int64_t bytes;                        // a_bytes + b_bytes
};

// Division of a 32-bit unsigned integer by an invariant divisor d >= 1 with
// one multiply-high, an add and two shifts (Granlund and Montgomery,
// "Division by invariant integers using multiplication", 1994, the
// round-up method with a 33-bit multiplier whose top bit is applied as an
// add): q = (t + ((x - t) >> s1)) >> s2 with t = mulhi(x, mul). Exact for
// every x < 2^32.
struct DivU32 {
    uint32_t mul, s1, s2;
};
DivU32 make_div(uint32_t d);

// Geometry of a convolution lowered to C += A B by IM2ROW (Sec. 4.2): row i
// of A is output pixel i (image, output row, output column), column p is
// (filter row, filter column, input channel); A[i, p] is the input element
// that this output pixel reads through that filter tap, or zero outside the
// image. All extents fit in 31 bits (checked on the host).
struct ConvGeom {
    int h, w, c;          // input height, width, channels (NHWC)
    int ohw, ow;          // output pixels per image, output width
    int s;                // filter width
    int sh, sw, ph, pw, dh, dw;
    int x_bytes;          // bytes of the input tensor
    int sc;               // s * c: elements of one filter row's window run
    int run2;             // dh * w * c - s * c: from one filter row's run to the next
    DivU32 by_c, by_s, by_ohw, by_ow, by_sc;
};

// Validation and planning; pure host code, no HIP calls.
int validate(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
             const void *B, int64_t ldb, const void *C, int64_t ldc);
// allow_packed = false restricts automatic choice to the fused kernels (used
// when no workspace can be obtained, e.g. under stream capture).
int make_plan(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
              const void *B, int64_t ldb, int64_t ldc, int num_cu, int kernel, int split,
              bool allow_packed, igemm_plan *out);
void packed_layout(int es, int64_t m, int64_t n, int64_t k, int kernel, const void *A,
                   int64_t lda, PackedLayout *L);

// Plan of one k block (kb <= kMaxKChunk elements) of the int16-output
// update: a small-tile fused kernel, one workgroup per output tile.
bool srs_kernel(int id);
int make_srs_plan(int es, int64_t m, int64_t n, int64_t kb, const void *A, int64_t lda,
                  const void *B, int64_t ldb, int64_t ldc, int num_cu, int kernel,
                  igemm_plan *out);
// Output extent of one spatial dimension of a convolution (-1 if invalid).
int64_t conv_out_dim(int64_t in, int64_t f, int64_t stride, int64_t pad, int64_t dil);
// Plan of a convolution as its lowered GEMM, with the kernel's geometry.
// Returns IGEMM_OK with out->kernel = -1 when there is nothing to compute.
// *gather: how the kernel reads the IM2ROW rows (1: 16-byte vector loads,
// channel rows 16-byte aligned; 3: unaligned 16-byte loads of the contiguous
// runs that a filter row covers when the horizontal dilation is 1; 2: one
// load per element).
int make_conv_plan(int es, const igemm_conv2d_desc *d, const void *X, const void *W,
                   const void *Y, int num_cu, int kernel, int split, igemm_plan *out,
                   ConvGeom *g, int *gather);

// The direct kernels (raw row-major A and B moved into LDS unchanged, no
// workspace) apply to these arguments: 16-byte aligned operands with rows a
// multiple of 16 bytes, k a multiple of 256 (whole groups of four k-tiles
// per launch), n a multiple of 8 (int16) or 16 (int8) columns, and byte offsets
// that fit the kernel's 32-bit lane offsets.
bool direct_ok(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
               const void *B, int64_t ldb, int64_t ldc);

// The small-output int16 kernel (64 x 64 tiles, at most four k-tiles per
// workgroup, all loads at once) applies to these arguments: 16-byte aligned
// operands with rows a multiple of 16 bytes, k a multiple of 64, n a multiple
// of 8, and byte offsets that fit its 32-bit lane offsets and grid.
bool small_ok(int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
              int64_t ldb, int64_t ldc);
// Its ragged variant (A through registers): A at any element alignment and
// any k >= 1; B 16-byte aligned with rows of whole 16 bytes, n a multiple of 8.
bool small_rg_ok(int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
                 int64_t ldb, int64_t ldc);

// Kernel launches for a validated plan (stream is a hipStream_t). The packed
// launch needs a workspace of at least plan.workspace_bytes, 256-byte aligned.
// The streaming kernel for few-row int8 products.
int launch_stream(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                  void *stream);
int launch_tiled(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                 int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                 void *stream);
// Host stubs of the fused kernel variants (VA: A rows 16-byte aligned, or for
// convolutions the 16-byte gather; VB: B rows aligned; SPLIT: k sliced across
// workgroups), one translation unit per group of tile shapes; nullptr for
// ids outside the group.
const void *fused_i8_wide(int id, bool va, bool vb, bool split);
const void *fused_i8_rows(int id, bool va, bool vb, bool split);
const void *fused_i16_wide(int id, bool va, bool vb, bool split);
const void *fused_i16_rows(int id, bool va, bool vb, bool split);
const void *fused_conv_i16(int id, int gather, bool vb, bool split);
const void *fused_conv_i8(int id, int gather, bool vb, bool split);
const void *fused_srs(int id, bool va, bool vb);
// The same fused kernels with A gathered from the NHWC input X by IM2ROW
// (gather mode as make_conv_plan chose it).
int launch_conv(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const ConvGeom &g,
                int gather, const void *X, const void *W, int32_t *Y, int64_t ldy,
                void *stream);
// The int16-output update on packed int16 operands (a packed plan whose
// workspace the pack kernels have filled, with the exact per-block limb sums
// of both operands in `sums`, srs_sums_bytes): one multiply launch, or one
// per block. nblocks <= 64; blocks of kc elements, a multiple of 256 unless
// there is one block.
int64_t srs_sums_bytes(const igemm_plan &p, int64_t m, int64_t n, int64_t k, int64_t nblocks,
                       const void *A, int64_t lda);
int launch_srs_packed(const igemm_plan &p, int64_t m, int64_t n, int64_t k, int64_t kc,
                      int64_t nblocks, const void *A, int64_t lda, int16_t *C, int64_t ldc,
                      const void *a_part, const void *b_part, uint32_t *sums, int shift,
                      int round_half_up, void *stream);
// The int16-output update of one k block (plan without k slices): C16 +=
// srs(A B) modulo 2^16 with the given shift and rounding.
int launch_srs(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
               int64_t lda, const void *B, int64_t ldb, int16_t *C, int64_t ldc, int shift,
               int round_half_up, void *stream);
// The packed path: pack A into an A part (optionally clearing the B part's
// column corrections, which pack_b then adds into), pack B into a B part
// (clear_corr: clear the corrections itself first), multiply (one launch per
// k chunk) from the two parts. For the int16-output update (sums given, int16
// only) the pack kernels also write the exact limb sums of each block of kc
// elements (one block: all of k) into sums, A's then B's, as
// launch_srs_packed reads them.
int launch_pack_a(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, void *a_part, void *b_part_to_clear, void *stream,
                  uint32_t *sums = nullptr, int64_t kc = 0, int64_t nblocks = 0);
int launch_pack_b(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, const void *B, int64_t ldb, void *b_part, bool clear_corr,
                  void *stream, uint32_t *sums = nullptr, int64_t kc = 0,
                  int64_t nblocks = 0);
// The direct kernel: one launch per k chunk of plan.k_chunk elements.
int launch_direct(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                  void *stream);
// The small-output int16 kernel: one launch, k slices of plan.k_chunk; and
// its convolution variants (A gathered from X: gather 1, whole 64-channel
// taps by DMA; gather 3, input runs through registers).
int launch_small(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                 int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                 void *stream);
int launch_small_conv(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const ConvGeom &g,
                      int gather, const void *X, const void *W, int32_t *Y, int64_t ldy,
                      void *stream);
int launch_multiply(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                    int64_t lda, int32_t *C, int64_t ldc, const void *a_part, const void *b_part,
                    void *stream);

}  // namespace igemm
