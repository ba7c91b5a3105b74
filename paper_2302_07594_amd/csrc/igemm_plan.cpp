// Host-side argument validation and launch planning (no HIP calls).
//
// The planner plays the role of the paper's choice of cache configuration
// parameters (Sec. 4.1: mc, nc, kc around a fixed micro-kernel; Sec. 6.3 and
// 6.4 pick kc and mc from the sizes of the memory levels). On the GPU the
// workgroup tile (bm x bn) takes the place of mc x nc, the k-tile of 64
// elements the place of kc, and the number of k slices is chosen so that
// small-output shapes -- the deep-learning shapes with one large and two
// small dimensions (Sec. 2, Sec. 4.2) -- still occupy every compute unit.
#include <limits.h>
#include <stddef.h>
#include <stdint.h>

#include "igemm_internal.h"

namespace igemm {

const KernelDesc kKernels[K_COUNT] = {
    {"i8_256x256", 1, 256, 256, 128, 128, false},
    {"i8_128x128", 1, 128, 128, 64, 64, false},
    {"i8_32x256", 1, 32, 256, 32, 64, false},
    {"i8_16x256", 1, 16, 256, 16, 64, false},
    {"i16_128x128", 2, 128, 128, 64, 64, false},
    {"i16_64x64", 2, 64, 64, 32, 32, false},
    {"i16_32x128", 2, 32, 128, 32, 32, false},
    {"i16_16x128", 2, 16, 128, 16, 32, false},
    {"i8_packed_256x256", 1, 256, 256, 64, 128, true},
    {"i16_packed_128x128", 2, 128, 128, 64, 64, true},
    {"i8_stream_32x128", 1, 32, 128, 16, 128, false},
    {"i16_direct_128x128", 2, 128, 128, 64, 64, false},
    {"i8_direct_256x256", 1, 256, 256, 64, 128, false},
    {"i16_small_64x64", 2, 64, 64, 32, 32, false},
    {"i16_stream_32x64", 2, 32, 64, 16, 16, false},
};

// Largest grid (in workgroups) of one launch: the dispatch packet counts
// work-items in 32 bits.
static constexpr int64_t kMaxGrid = ((int64_t)1 << 32) / kThreads - 1;

static bool mul_ok(int64_t a, int64_t b, int64_t *out) {
    return !__builtin_mul_overflow(a, b, out);
}

// Byte extent of a rows x cols window with leading dimension ld; false on
// int64 overflow.
static bool extent_ok(int64_t rows, int64_t cols, int64_t ld, int64_t es) {
    int64_t t;
    if (!mul_ok(rows - 1, ld, &t)) return false;
    if (__builtin_add_overflow(t, cols, &t)) return false;
    return mul_ok(t, es, &t);
}

int validate(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
             const void *B, int64_t ldb, const void *C, int64_t ldc) {
    if (es != 1 && es != 2) return IGEMM_EINVAL;
    if (m < 0 || n < 0 || k < 0) return IGEMM_EINVAL;
    if (m == 0 || n == 0) return IGEMM_OK;
    if (C == NULL || ldc < n) return IGEMM_EINVAL;
    if (!extent_ok(m, n, ldc, 4)) return IGEMM_EINVAL;
    if (k > 0) {
        if (A == NULL || B == NULL) return IGEMM_EINVAL;
        if (lda < k || ldb < n) return IGEMM_EINVAL;
        if (!extent_ok(m, k, lda, es) || !extent_ok(k, n, ldb, es)) return IGEMM_EINVAL;
    }
    // k leaves headroom so that k-tile offsets computed in int never overflow.
    if (m > INT_MAX || n > INT_MAX || k > INT_MAX - 65536) return IGEMM_ENOTSUP;
    return IGEMM_OK;
}

static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

static int64_t tiles_of(int id, int64_t m, int64_t n) {
    return cdiv(m, kKernels[id].bm) * cdiv(n, kKernels[id].bn);
}

static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

void packed_layout(int es, int64_t m, int64_t n, int64_t k, int kernel, const void *A,
                   int64_t lda, PackedLayout *L) {
    const KernelDesc &d = kKernels[kernel];
    L->m_pad = cdiv(m, d.bm) * d.bm;
    L->n_pad = cdiv(n, d.bn) * d.bn;
    // A multiple of four 64-element k-tiles, so the main loop has no remainder.
    L->k_pad = cdiv(k, 256) * 256;
    // pack_b: 64 columns per workgroup and k slices of whole passes (a pass
    // covers 128 int16 or 256 int8 rows), enough slices for ~512 workgroups.
    const int64_t colblocks = L->n_pad / 64;
    const int64_t rows_per_pass = es == 2 ? 128 : 256;
    const int64_t passes = L->k_pad / rows_per_pass;
    int64_t s = cdiv(512, colblocks);
    if (s > passes) s = passes;
    if (s < 1) s = 1;
    L->kspan = cdiv(passes, s) * rows_per_pass;
    L->b_slices = (int)cdiv(L->k_pad, L->kspan);
    const uintptr_t a = (uintptr_t)A;
    L->pack_a = es == 2 || !(a % 16 == 0 && lda % 16 == 0 && m % d.bm == 0 && k % 256 == 0);
    int64_t off = 0;
    L->off_a = off;
    if (L->pack_a) off = align256(off + es * L->m_pad * L->k_pad);
    L->off_corr_a = off;
    if (es == 2) off = align256(off + 4 * L->m_pad);
    L->a_bytes = off;
    off = 0;
    L->off_b = off;
    off = align256(off + es * L->n_pad * L->k_pad);
    L->off_corr_b = off;
    if (es == 2) off = align256(off + 4 * L->n_pad);
    L->b_bytes = off;
    L->bytes = L->a_bytes + L->b_bytes;
}

// The packed path pays off once the product is large enough for the pack
// traffic (one read and one write of each operand) to be small next to the
// rest and there are enough tiles to fill the chip. Measured on int16
// m = n = 4096: packed against fused 128x128 tiles 61.6 against 68.7 us at
// k = 256, 77.3 against 84.3 at k = 290, 111 against 128 at k = 1024 (with
// k this short both are bound by the read and write of C).
static bool packed_pays(int es, int64_t m, int64_t n, int64_t k, int num_cu) {
    const int id = es == 2 ? K_I16_PACKED_128x128 : K_I8_PACKED_256x256;
    return k >= 256 && m >= 1024 && n >= 1024 && tiles_of(id, m, n) >= num_cu;
}

// The packed kernel addresses its C tile with 32-bit byte offsets.
static bool packed_fits(int id, int64_t ldc) {
    return (int64_t)kKernels[id].bm * ldc * 4 < INT_MAX;
}

static bool is_direct(int id) { return id == K_I16_DIRECT_128x128 || id == K_I8_DIRECT_256x256; }

bool direct_ok(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
               const void *B, int64_t ldb, int64_t ldc) {
    const int id = es == 2 ? K_I16_DIRECT_128x128 : K_I8_DIRECT_256x256;
    const uintptr_t a = (uintptr_t)A, b = (uintptr_t)B;
    if (a % 16 != 0 || b % 16 != 0 || (lda * es) % 16 != 0 || (ldb * es) % 16 != 0) return false;
    // Whole groups of four k-tiles per launch (the kernel's loop has no
    // remainder steps).
    if (k % (4 * kBK) != 0 || n % (16 / es) != 0) return false;
    // 32-bit lane offsets: rows of A from its base, 64 rows of B plus a column.
    if (m * lda * es >= ((int64_t)1 << 31) || (kBK + 1) * ldb * es >= ((int64_t)1 << 31))
        return false;
    return packed_fits(id, ldc) && tiles_of(id, m, n) <= kMaxGrid;
}

// Most k-tiles one workgroup of the small-output kernel takes (its LDS holds
// them all at once).
static constexpr int64_t kSmallKtMax = 4;

bool small_ok(int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
              int64_t ldb, int64_t ldc) {
    const uintptr_t a = (uintptr_t)A, b = (uintptr_t)B;
    if (a % 16 != 0 || b % 16 != 0 || (lda * 2) % 16 != 0 || (ldb * 2) % 16 != 0) return false;
    if (k % kBK != 0 || n % 8 != 0) return false;
    // 32-bit lane offsets: rows of A from the k-tile's base, 64 rows of B plus
    // a column, 64 rows of C; grid: column tiles, row tiles, k slices.
    if (m * lda * 2 >= ((int64_t)1 << 31) || (kBK * ldb + n) * 2 >= ((int64_t)1 << 31) ||
        64 * ldc * 4 >= ((int64_t)1 << 31))
        return false;
    return cdiv(n, 64) <= kMaxGrid && cdiv(m, 64) <= 65535 &&
           cdiv(k / kBK, kSmallKtMax) <= 65535;
}

// The ragged variant of the small-output kernel: A's rows at any element
// alignment and any k >= 1 (A read through registers); B as for the DMA
// variant but with rows past k read as zeros, so its k-tiles may overrun k.
bool small_rg_ok(int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                        const void *B, int64_t ldb, int64_t ldc) {
    const uintptr_t a = (uintptr_t)A, b = (uintptr_t)B;
    if (k < 1 || a % 2 != 0 || b % 16 != 0 || (ldb * 2) % 16 != 0 || n % 8 != 0) return false;
    const int64_t ktiles = cdiv(k, kBK);
    // 32-bit offsets: A's rows and k-tiles (plus a 20-byte read), B's k-tiles
    // plus a column, 64 rows of C; the resources' ranges.
    if ((m * lda + ktiles * kBK) * 2 + 32 >= ((int64_t)1 << 31) ||
        ((ktiles + 1) * kBK * ldb + n) * 2 >= ((int64_t)1 << 31) ||
        64 * ldc * 4 >= ((int64_t)1 << 31))
        return false;
    return cdiv(n, 64) <= kMaxGrid && cdiv(m, 64) <= 65535 &&
           cdiv(ktiles, kSmallKtMax) <= 65535;
}

// k elements per launch of the direct kernels: as few launches as the
// 32768-element limit allows, split evenly in groups of four k-tiles.
static int64_t direct_chunk(int64_t k) {
    const int64_t launches = cdiv(k, kMaxKChunk);
    return cdiv(k / (4 * kBK), launches) * 4 * kBK;
}

// Streaming kernel: row blocks of 16 or 32 rows, column blocks of 128, and
// workgroups of 4 or 8 waves that each take 1, 2 or 4 k-steps of 64 (4, 8,
// 16 or 32 steps per workgroup). Returns false if its 32-bit window offsets
// do not fit.
// Operands the int16 column-per-wave kernel takes: A and B 16-byte aligned
// with rows of whole 16-byte chunks, k a multiple of 64 and n of 8.
static bool i16_stream_ok(int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
                          int64_t ldb) {
    return (uintptr_t)A % 16 == 0 && (uintptr_t)B % 16 == 0 && lda % 8 == 0 && ldb % 8 == 0 &&
           k % kBK == 0 && n % 8 == 0 && k <= lda && n <= ldb;
}

// The int16 column-per-wave kernel's launch: 64-column blocks of 16 or 32
// rows, 4 k-steps of 64 per workgroup (8 when an explicit k-slice count asks
// for longer ranges). Four steps measured faster than eight on every
// weight-streaming shape (k = 4096, us, 4 / 8 steps): 1 x 4096 8.6 / 9.1,
// 8 x 4096 9.4 / 9.6, 1 x 11008 17.7 / 19.6, 8 x 11008 19.1 / 20.9,
// 32 x 11008 25.5 / 35.5 (eight steps of two 16-row blocks hold 96 KB of
// LDS: one workgroup per compute unit).
static int i16_stream_plan(int64_t m, int64_t n, int64_t k, int64_t lda, int64_t ldb,
                           int split, igemm_plan *out) {
    const int64_t ksteps = k / kBK;
    const int64_t spw = split > 0 && cdiv(ksteps, split) > 4 ? 8 : 4;
    const int bm = m <= 16 ? 16 : 32;
    // (32-bit byte offsets into a workgroup's k range of B and rows of A)
    int64_t t;
    if (ldb >= 0x7fff0000 / (2 * spw * kBK) || lda >= 0x7fff0000 / 64 - 64 ||
        !mul_ok(cdiv(m, bm), cdiv(n, 64), &t) || t > kMaxGrid ||
        t * cdiv(ksteps, spw) > kMaxGrid)
        return IGEMM_ENOTSUP;
    out->kernel = K_I16_STREAM;
    out->bm = bm;
    out->bn = 64;
    out->threads = 256;
    out->k_chunk = spw * kBK;
    out->split = (int)cdiv(ksteps, spw);
    out->tiles = t;
    out->grid = t * out->split;
    out->vec_a = 1;
    out->vec_b = 1;
    return IGEMM_OK;
}

struct StreamShape {
    int bm, threads;
    int64_t spw, slices, tiles;
    bool lds;  // the column-per-wave kernel (else the register kernel)
};
static bool stream_shape(int64_t m, int64_t n, int64_t k, int64_t lda, int64_t ldb, bool va,
                         bool vb16, bool vb, int split, int num_cu, StreamShape *out) {
    int bm = m <= 16 ? 16 : 32;
    const int64_t ksteps = cdiv(k, kBK);
    int64_t spw = 4;
    // 17 to 32 rows over few column blocks (at most one workgroup per compute
    // unit with 32-row blocks of 8 steps) take the register kernel's two
    // 16-row blocks of 16 steps even when the column-per-wave kernel could
    // run: 32 x 4096 x 4096 7.07-7.26 us against 7.22-7.71 us.
    const bool two_blocks =
        va && vb && bm == 32 && split <= 0 && cdiv(n, 128) * cdiv(ksteps, 8) <= num_cu;
    out->lds = va && vb16 && !two_blocks;
    if (out->lds) {
        // The column-per-wave kernel (A and B rows of whole 16-byte chunks):
        // eight waves, 4, 8 or 16 steps of 64 k per workgroup, all of them in
        // LDS at once (up to 160 KB). 8 steps by default; measured with k =
        // 4096 (us, 4 / 8 / 16 steps): 1 x 4096 4.76 / 4.92 / 5.82, 32 x 4096
        // 8.98 / 7.34 / 7.79, 1 x 11008 9.94 / 10.16 / 12.79, 32 x 11008
        // 19.07 / 14.76 / 16.63.
        int64_t want = split > 0 ? cdiv(ksteps, split) : 8;
        // 17 to 32 rows over 64 to 128 column blocks: as many k slices as
        // give one workgroup per compute unit (two for 11008 columns, four
        // for 8192), each a long range (through the ring variant beyond 16
        // steps), so that C takes fewer atomic adds (32 x 11008 x 4096:
        // 12.4 us with two slices against 14.4 us with eight slices of 8
        // steps; three slices, 258 workgroups on 256 units, 17.0 us;
        // 32 x 8192 x 4096: 10.7 us with four slices of 16 steps against
        // 11.5 us with eight).
        const int64_t cbs = cdiv(n, 128), per_unit = num_cu / cbs;
        if (split <= 0 && bm == 32 && cbs >= 64 && cbs <= 128 && per_unit >= 1 &&
            cdiv(ksteps, per_unit) > 8)
            want = cdiv(ksteps, per_unit);
        while (spw < want && spw < 16) spw *= 2;
        // Longer ranges (more than 16 steps) take the ring variant, which
        // streams any number of steps through eight LDS stages (measured
        // with k = 4096, slices of 64, 32 or 22 steps against 8: slower on
        // the 4096-column shapes, whose 32 column blocks then leave most
        // compute units idle, and within 5 % on 1 and 8 x 11008).
        if (want > 16) spw = want;
        // (This kernel with two 16-row blocks took 7.44 us on 32 x 4096 x 4096.)
        if (ldb >= (0x7fff0000 - 256) / (spw * kBK) || lda >= 0x7fff0000 / 64 ||
            32 * lda + spw * kBK >= 0x7fff0000)
            return false;
        out->bm = bm;
        out->threads = 512;
        out->spw = spw;
        out->slices = cdiv(ksteps, spw);
        out->tiles = cdiv(m, bm) * cdiv(n, 128);
        return out->tiles * out->slices <= ((int64_t)1 << 32) / 512 - 1;
    }
    if (va && vb) {
        // The register kernel with 8-byte loads of B.
        // Few slices keep the atomic adds into C cheap; enough workgroups keep
        // the loads of B in flight. Measured on the 4096- and 11008-column
        // shapes with k = 4096: 8 steps per workgroup (4 and 16 are up to 10%
        // slower, 32 up to 2x).
        int64_t want = split > 0 ? cdiv(ksteps, split) : 8;
        // 17 to 32 rows over few column blocks (at most one workgroup per
        // compute unit with 32-row blocks of 8 steps): two 16-row blocks of
        // 16 steps instead, half the adds per workgroup and no two-phase
        // reduction (32 x 4096 x 4096: 7.1 us against 8.2 us; on 32 x 11008,
        // where B's second pass costs bandwidth, 16.8 against 15.2 us).
        if (two_blocks) {
            bm = 16;
            want = 16;
        }
        const int64_t cap = bm == 16 ? 32 : 16;
        while (spw < want && spw < cap) spw *= 2;
    }
    if ((spw * kBK) * ldb + 128 >= 0x7fff0000 || (int64_t)bm * lda + spw * kBK >= 0x7fff0000)
        return false;
    out->bm = bm;
    out->threads = spw == 4 ? 256 : 512;
    out->spw = spw;
    out->slices = cdiv(ksteps, spw);
    out->tiles = cdiv(m, bm) * cdiv(n, 128);
    return out->tiles * out->slices <= ((int64_t)1 << 32) / 512 - 1;
}

// k slices for the 128x128 tiles (int16 and int8) below one tile per compute
// unit. One workgroup fits on a compute unit, so a grid beyond num_cu would
// run a second, mostly empty round: slice up to num_cu / tiles, keeping at
// least 512 k per slice. Measured, int16: (1568, 512, 4608) 36 us with 4
// slices (208 workgroups) against 45 us with 5 (260) and 46 with 2;
// (6272, 256, 2304) 36 us with 2 slices against 46-49 us with 1, 3 or 4.
// int8: (1568, 512, 4608) 22.4 us with 4 slices against 26.0 with 2 and 25.0
// with 5; (6272, 256, 2304) 24.2 us with 2 against 32.1 with 1;
// (1024, 1024, 8192) 33.7 us with 4 against 47.8 with 2 and 41.1 with 5.
static int64_t big_tile_split(int64_t tiles, int64_t k, int num_cu) {
    if (tiles >= num_cu) return 1;
    int64_t s = num_cu / tiles;
    const int64_t cap = cdiv(k, kBK) / 8;
    if (s > cap) s = cap;
    return s < 1 ? 1 : s;
}

// k-tiles per workgroup of the small-output kernel: its atomic adds into C
// cost about as much as the extra parallelism of more k slices buys, so the
// fewest slices that still give 128 workgroups (or one k-tile each, when
// the product has fewer), spread evenly. Measured (us): (49, 512, 4608)
// 5.96 with 4 k-tiles per workgroup, 6.02 with 3, 6.63 with 2, 8.92 with 1;
// (784, 128, 1152) 5.50 / 5.63 / 6.04 / 8.01; (3136, 64, 576) 5.59 with 3
// against 5.92 with 2; 256^3 4.17 with 1 against 4.23 with 2.
static int64_t small_ktpw(int64_t tiles, int64_t ktiles) {
    const int64_t want = tiles * ktiles < 128 ? tiles * ktiles : 128;
    int64_t t = kSmallKtMax;
    while (t > 1 && tiles * cdiv(ktiles, t) < want) --t;
    return cdiv(ktiles, cdiv(ktiles, t));
}

// The small-output kernel takes int16 products whose whole grid, at four
// k-tiles per workgroup, fits in two workgroups per compute unit.
static bool small_pays(int64_t m, int64_t n, int64_t k, int num_cu) {
    const int64_t tiles = cdiv(m, 64) * cdiv(n, 64);
    return tiles * cdiv(cdiv(k, kBK), kSmallKtMax) <= 2 * (int64_t)num_cu;
}

static int auto_kernel(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
                       const void *B, int64_t ldb, int64_t ldc, int num_cu, bool allow_packed) {
    const int pid = es == 2 ? K_I16_PACKED_128x128 : K_I8_PACKED_256x256;
    // Large products: int8 takes the direct kernel whenever the operands
    // allow it (int8 8192^3: 519 us against 566 us for pack + packed
    // multiply, and 534 us for the packed multiply alone); int16 takes the
    // packed path when a workspace is given (4096^3: pack 26 us + multiply
    // 239 us against 282 us direct: the direct kernel's in-register limb
    // split costs matrix-core issue slots) and the direct kernel otherwise
    // (fused 128x128 tiles: 337 us).
    const bool large = packed_pays(es, m, n, k, num_cu);
    const bool direct = large && direct_ok(es, m, n, k, A, lda, B, ldb, ldc);
    if (es == 1 && direct) return K_I8_DIRECT_256x256;
    // Up to k = 1024 the pack pass costs the packed path more than the
    // direct kernel's in-register split (int16 m = n = 4096, one call, us:
    // k = 256 61.6 packed against 57.9 direct, 512 77.9 / 74.7, 1024
    // 106.9 / 106.0, 2048 161.8 / 164.6).
    if (es == 2 && direct && k <= 1024) return K_I16_DIRECT_128x128;
    if (allow_packed && large && packed_fits(pid, ldc) &&
        16 * (k > lda ? k : lda) < ((int64_t)1 << 31))
        return pid;
    if (direct) return K_I16_DIRECT_128x128;
    if (es == 2 && !large && small_pays(m, n, k, num_cu) &&
        (small_ok(m, n, k, A, lda, B, ldb, ldc) || small_rg_ok(m, n, k, A, lda, B, ldb, ldc)))
        return K_I16_SMALL_64x64;
    if (es == 1) {
        StreamShape ss;
        if (m <= 32 && n >= 512 && k >= 256 && (uintptr_t)B % 8 == 0 && ldb % 8 == 0 &&
            (uintptr_t)A % 16 == 0 && lda % 16 == 0 &&
            stream_shape(m, n, k, lda, ldb, true, (uintptr_t)B % 16 == 0 && ldb % 16 == 0, true,
                         -1, num_cu, &ss))
            return K_I8_STREAM;
        if (m <= 16) return K_I8_16x256;
        if (m <= 32) return K_I8_32x256;
        if (tiles_of(K_I8_256x256, m, n) >= num_cu) return K_I8_256x256;
        return K_I8_128x128;
    }
    // Up to 16 rows over wide B (the weight-streaming shapes): the int16
    // column-per-wave kernel where the operands allow it (k = 4096, us:
    // 1 x 11008 17.7 against 26.4 on 16x128 tiles, 8 x 4096 9.4 against
    // 12.3). With 17 to 32 rows the fused 32x128 tiles stay (32 x 11008 24.6
    // against 25.5 us).
    igemm_plan sp{};
    if (m <= 16 && n >= 512 && k >= 256 && i16_stream_ok(n, k, A, lda, B, ldb) &&
        i16_stream_plan(m, n, k, lda, ldb, -1, &sp) == IGEMM_OK)
        return K_I16_STREAM;
    if (m <= 16) return K_I16_16x128;
    if (m <= 32) return K_I16_32x128;
    // 128-column tiles on n <= 64 would multiply padding for half their
    // columns (measured on (401408, 64, 147): 205 us against 120 us with
    // 64x64 tiles; (100352, 64, 576): 92 against 64 us). Otherwise 128x128
    // tiles pay from three quarters of a tile per compute unit: n = 128 and
    // 256 with k = 512..2304 and 192-255 tiles ran 13-35% faster than 64x64
    // tiles; at half a tile per unit the two were within +-20% either way.
    // Up to k = 256 the 64x64 tiles' single pass (every load at once, C
    // fetched alongside) wins instead: (100352, 256, 64) 78 against 84 us.
    // With k slices (big_tile_split) the same holds for fewer tiles: three
    // quarters of the compute units busy with slices of at least 512 k.
    if (n > 64 && k > 256) {
        const int64_t t128 = tiles_of(K_I16_128x128, m, n);
        if (4 * t128 * big_tile_split(t128, k, num_cu) >= 3 * (int64_t)num_cu)
            return K_I16_128x128;
    }
    // Small outputs: time goes into each workgroup's latency chain (load,
    // stage, multiply, write back), so twice the workgroups of half the size
    // finish sooner (measured: 256x256x256 3.9 us against 5.6 us with 64x64
    // tiles; 784x128x1152 and 196x256x2304 13% and 9% faster).
    if (tiles_of(K_I16_64x64, m, n) < 32) return m <= 64 ? K_I16_32x128 : K_I16_16x128;
    // A single k-tile cannot be sliced, so when the 64x64 tiles leave compute
    // units idle only smaller tiles add workgroups: (3136, 256, 64) with
    // 16x128 tiles 5.6 us against 6.1 us.
    if (k <= kBK && tiles_of(K_I16_64x64, m, n) < num_cu) return K_I16_16x128;
    return K_I16_64x64;
}

int make_plan(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
              const void *B, int64_t ldb, int64_t ldc, int num_cu, int kernel, int split,
              bool allow_packed, igemm_plan *out) {
    if (out == NULL) return IGEMM_EINVAL;
    if (num_cu <= 0) num_cu = 256;
    *out = igemm_plan{};
    out->elem_bytes = es;
    out->bk = kBK;
    out->threads = kThreads;
    out->limb_products = es == 2 ? 4 : 1;
    if (m == 0 || n == 0 || k == 0) {
        out->kernel = -1;
        return IGEMM_OK;  // no-op: nothing is launched
    }
    if (kernel < -1 || kernel >= K_COUNT || split < -1 || split == 0) return IGEMM_EINVAL;
    int id = kernel >= 0 ? kernel : auto_kernel(es, m, n, k, A, lda, B, ldb, ldc, num_cu, allow_packed);
    if (kKernels[id].es != es) return IGEMM_EINVAL;
    const KernelDesc &d = kKernels[id];
    const int64_t tiles = tiles_of(id, m, n);
    const uintptr_t a = (uintptr_t)A, b = (uintptr_t)B;
    if (is_direct(id)) {
        if (!direct_ok(es, m, n, k, A, lda, B, ldb, ldc)) return IGEMM_EINVAL;
        out->kernel = id;
        out->bm = d.bm;
        out->bn = d.bn;
        out->threads = (d.bm / d.wm) * (d.bn / d.wn) * 64;
        out->k_chunk = direct_chunk(k);
        out->split = (int)cdiv(k, out->k_chunk);
        // int16 launches of at most eight k-tiles run eight waves of 64 x 32
        if (es == 2 && out->k_chunk <= 8 * kBK) out->threads = 512;
        out->tiles = tiles;
        out->grid = tiles;
        out->vec_a = 1;
        out->vec_b = 1;
        return IGEMM_OK;
    }
    if (id == K_I16_SMALL_64x64) {
        // vec_a = 1: A by DMA; 0: the ragged variant
        const bool dma_a = small_ok(m, n, k, A, lda, B, ldb, ldc);
        if (!dma_a && !small_rg_ok(m, n, k, A, lda, B, ldb, ldc)) return IGEMM_EINVAL;
        // k-tiles per workgroup: an explicit split asks for that many slices
        // (at least k / 256 of them: a workgroup takes at most four k-tiles).
        const int64_t ktiles = cdiv(k, kBK);
        int64_t ktpw = split > 0 ? cdiv(ktiles, split) : small_ktpw(tiles, ktiles);
        if (ktpw > kSmallKtMax) ktpw = kSmallKtMax;
        if (ktpw < 1) ktpw = 1;
        out->kernel = id;
        out->bm = d.bm;
        out->bn = d.bn;
        out->threads = 256;
        out->k_chunk = ktpw * kBK;
        out->split = (int)cdiv(ktiles, ktpw);
        out->tiles = tiles;
        out->grid = tiles * out->split;
        out->vec_a = dma_a ? 1 : 0;
        out->vec_b = 1;
        return IGEMM_OK;
    }
    if (d.packed) {
        // Pack once, then one launch of the main kernel per k chunk of at most
        // kMaxKChunk elements; the launches add into C in stream order.
        PackedLayout L;
        packed_layout(es, m, n, k, id, A, lda, &L);
        // The multiply kernel addresses 16 rows of a plane with 32-bit lane
        // offsets.
        const int64_t plane_ld = L.pack_a ? L.k_pad : (L.k_pad > lda ? L.k_pad : lda);
        if (tiles > kMaxGrid || L.m_pad > kMaxGrid || L.n_pad / 64 > kMaxGrid ||
            L.b_slices > 65535 || !packed_fits(id, ldc) || 16 * plane_ld >= ((int64_t)1 << 32))
            return IGEMM_ENOTSUP;
        out->kernel = id;
        out->bm = d.bm;
        out->bn = d.bn;
        out->threads = (d.bm / d.wm) * (d.bn / d.wn) * 64;
        out->k_chunk = L.k_pad < kMaxKChunk ? L.k_pad : kMaxKChunk;
        out->split = (int)cdiv(L.k_pad, out->k_chunk);
        out->tiles = tiles;
        out->grid = tiles;
        out->vec_a = (a % 16 == 0) && ((lda * es) % 16 == 0);
        out->vec_b = (b % 16 == 0) && ((ldb * es) % 16 == 0);
        out->packed = 1;
        out->workspace_bytes = L.bytes;
        out->packed_a_bytes = L.a_bytes;
        out->packed_b_bytes = L.b_bytes;
        return IGEMM_OK;
    }
    if (id == K_I16_STREAM) {
        if (!i16_stream_ok(n, k, A, lda, B, ldb)) return IGEMM_EINVAL;
        return i16_stream_plan(m, n, k, lda, ldb, split, out);
    }
    if (id == K_I8_STREAM) {
        // vec_b = 1: B's rows are whole 16-byte chunks (with vec_a, the
        // column-per-wave kernel); otherwise the register kernel
        const bool va = a % 16 == 0 && lda % 16 == 0;
        const bool vb = b % 16 == 0 && ldb % 16 == 0;
        const bool vb8 = b % 8 == 0 && ldb % 8 == 0;
        StreamShape ss;
        if (!stream_shape(m, n, k, lda, ldb, va, vb, vb8, split, num_cu, &ss))
            return IGEMM_ENOTSUP;
        out->kernel = id;
        out->bm = ss.bm;
        out->bn = 128;
        out->split = (int)ss.slices;
        out->k_chunk = ss.spw * kBK;
        out->tiles = ss.tiles;
        out->grid = ss.tiles * ss.slices;
        out->threads = ss.threads;
        out->vec_a = va;
        // vec_b = 1: the column-per-wave kernel (B's rows whole 16-byte chunks)
        out->vec_b = ss.lds ? 1 : 0;
        return IGEMM_OK;
    }
    const int64_t ktiles = cdiv(k, kBK);
    const int64_t min_split = cdiv(k, kMaxKChunk);
    int64_t s;
    if (split > 0) {
        s = split;
    } else if (tiles >= num_cu) {
        s = 1;
    } else if ((id == K_I16_128x128 || id == K_I8_128x128) &&
               2 * tiles * big_tile_split(tiles, k, num_cu) >= num_cu) {
        // (Outputs too small to keep half the units busy this way keep the
        // rule below.)
        s = big_tile_split(tiles, k, num_cu);
    } else {
        // Aim for two workgroups per compute unit, but keep at least two
        // k-tiles per slice so each slice still pipelines its loads (the
        // 16- and 32-row int16 tiles take short ranges in one pass, where a
        // single k-tile per slice measured fastest on small cubes).
        // (The cap rounds up: with nine k-tiles, five slices of at most two
        // rather than three slices of three; (3136, 64, 576) on 64x64 tiles
        // 7.0 against 7.6 us, (12544, 64, 147) 8.3 against 8.5 us.)
        s = cdiv(2 * (int64_t)num_cu, tiles);
        const bool one_tile = id == K_I16_16x128 || id == K_I16_32x128;
        const int64_t cap = one_tile ? ktiles : cdiv(ktiles, 2);
        if (s > cap) s = cap;
    }
    // Small-tile kernels take a k range of at most four k-tiles in one go
    // (all loads issued at once); prefer that when the grid stays modest.
    const bool short_tiles = (int64_t)d.bm * d.bn <= 32 * 256;
    // Four-tile ranges also beat shorter ones when they still give a
    // workgroup per CU (fewer slices add into C).
    if (split <= 0 && short_tiles && cdiv(ktiles, s) > 4 &&
        tiles * cdiv(ktiles, 4) <= 4 * (int64_t)num_cu)
        s = cdiv(ktiles, 4);
    if (split <= 0 && short_tiles && cdiv(ktiles, s) < 4 &&
        tiles * cdiv(ktiles, 4) >= (int64_t)num_cu)
        s = cdiv(ktiles, 4);
    // Every k slice adds its partial tile into C with atomics; their cost
    // grows with m * n * slices (measured: past ~2^21 element updates it
    // outweighs the extra parallelism).
    // (The 128x128 slices of the rule above are long enough to carry their
    // adds.)
    const bool big_slices = (id == K_I16_128x128 || id == K_I8_128x128) && tiles < num_cu &&
                            2 * tiles * big_tile_split(tiles, k, num_cu) >= num_cu;
    if (split <= 0 && !big_slices) {
        const int64_t cap = ((int64_t)1 << 21) / (m * n);
        if (s > cap) s = cap > 1 ? cap : 1;
    }
    if (s < min_split) s = min_split;
    if (s > ktiles) s = ktiles;
    if (s < 1) s = 1;
    const int64_t kchunk = cdiv(ktiles, s) * kBK;
    s = cdiv(k, kchunk);
    const int64_t grid = tiles * s;
    if (grid > kMaxGrid) return IGEMM_ENOTSUP;
    out->kernel = id;
    out->bm = d.bm;
    out->bn = d.bn;
    out->split = (int)s;
    out->k_chunk = kchunk;
    out->tiles = tiles;
    out->grid = grid;
    // Vector path: 16-byte aligned rows, and per-lane row offsets within one
    // workgroup tile that fit in 32 bits (bm rows of A, 64 rows of B).
    out->vec_a = (a % 16 == 0) && ((lda * es) % 16 == 0) && ((int64_t)d.bm * lda * es < INT_MAX);
    out->vec_b = (b % 16 == 0) && ((ldb * es) % 16 == 0) && ((int64_t)kBK * ldb * es < INT_MAX);
    return IGEMM_OK;
}

DivU32 make_div(uint32_t d) {
    DivU32 r = {0u, 0u, 0u};
    if (d <= 1) return r;  // x / 1: t = 0, q = x
    int l = 0;
    while (((uint64_t)1 << l) < d) ++l;  // l = ceil(log2 d), 1 <= l <= 32
    r.mul = (uint32_t)((((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d + 1);
    r.s1 = 1;
    r.s2 = (uint32_t)(l - 1);
    return r;
}

int64_t conv_out_dim(int64_t in, int64_t f, int64_t stride, int64_t pad, int64_t dil) {
    if (in < 0 || f < 1 || stride < 1 || pad < 0 || dil < 1) return -1;
    int64_t t, padded;
    if (__builtin_mul_overflow(dil, f - 1, &t) || __builtin_mul_overflow(pad, 2, &padded) ||
        __builtin_add_overflow(in, padded, &padded))
        return -1;
    const int64_t span = padded - t - 1;  // no overflow: padded >= 0, t >= 0
    return span < 0 ? 0 : span / stride + 1;
}

// One k block of the int16-output update (the conversion of Sec. 5.2 applies
// per block, so a block is never sliced across workgroups): int16 64x64 tiles
// when there are enough of them, else 32- or 16-row tiles; int8 32- or 16-row
// tiles. (128x128 tiles, one workgroup per compute unit, took 95 us against
// 89 us for 64x64 on the paper's shape (4096, 4096, 290): the 64-bit
// conversion is better hidden behind a second workgroup.)
bool srs_kernel(int id) {
    return id == K_I16_128x128 || id == K_I16_64x64 || id == K_I16_32x128 ||
           id == K_I16_16x128 || id == K_I8_32x256 || id == K_I8_16x256;
}

int make_srs_plan(int es, int64_t m, int64_t n, int64_t kb, const void *A, int64_t lda,
                  const void *B, int64_t ldb, int64_t ldc, int num_cu, int kernel,
                  igemm_plan *out) {
    if (kb > kMaxKChunk) return IGEMM_ENOTSUP;
    if (num_cu <= 0) num_cu = 256;
    int id = kernel;
    if (id < 0) {
        if (es == 2)
            id = tiles_of(K_I16_64x64, m, n) >= 32 ? K_I16_64x64
                                                    : (m <= 16 ? K_I16_16x128 : K_I16_32x128);
        else
            id = m <= 16 ? K_I8_16x256 : K_I8_32x256;
    }
    if (id >= K_COUNT || !srs_kernel(id) || kKernels[id].es != es) return IGEMM_EINVAL;
    const int st = make_plan(es, m, n, kb, A, lda, B, ldb, ldc, num_cu, id, 1, false, out);
    if (st != IGEMM_OK) return st;
    if (out->kernel >= 0 && out->split != 1) return IGEMM_ENOTSUP;
    return IGEMM_OK;
}

// A convolution planned as the GEMM its IM2ROW lowering gives (Sec. 4.2):
// m = n * oh * ow output pixels, n_gemm = output channels, k = r * s * c.
int make_conv_plan(int es, const igemm_conv2d_desc *d, const void *X, const void *W,
                   const void *Y, int num_cu, int kernel, int split, igemm_plan *out,
                   ConvGeom *g, int *gather) {
    if (out == NULL || d == NULL || (es != 1 && es != 2)) return IGEMM_EINVAL;
    *out = igemm_plan{};
    out->kernel = -1;
    out->elem_bytes = es;
    if (d->n < 0 || d->h < 0 || d->w < 0 || d->c < 0 || d->k < 0 || d->r < 1 || d->s < 1)
        return IGEMM_EINVAL;
    const int64_t oh = conv_out_dim(d->h, d->r, d->stride_h, d->pad_h, d->dil_h);
    const int64_t ow = conv_out_dim(d->w, d->s, d->stride_w, d->pad_w, d->dil_w);
    if (oh < 0 || ow < 0) return IGEMM_EINVAL;
    const int64_t N = d->k;
    int64_t M, K;
    if (__builtin_mul_overflow(d->n, oh, &M) || __builtin_mul_overflow(M, ow, &M) ||
        __builtin_mul_overflow(d->r, d->s, &K) || __builtin_mul_overflow(K, d->c, &K)) {
        // Sizes beyond int64: unsupported unless one factor makes them empty.
        if (d->n == 0 || oh == 0 || ow == 0 || N == 0 || d->c == 0) return IGEMM_OK;
        return IGEMM_ENOTSUP;
    }
    if (M == 0 || N == 0 || K == 0) return IGEMM_OK;  // nothing to add
    if (X == NULL || W == NULL || Y == NULL) return IGEMM_EINVAL;
    // The element gather reads X one element at a time: int16 X must be
    // 2-byte aligned (as its C type requires).
    if (es == 2 && ((uintptr_t)X & 1) != 0) return IGEMM_EINVAL;
    // 31-bit extents: input bytes and window arithmetic (the kernel addresses
    // the input through one buffer resource), the lowered GEMM's sizes.
    const int64_t lim = (int64_t)1 << 30;
    if (d->h + 2 * d->pad_h >= lim || d->w + 2 * d->pad_w >= lim || d->c >= lim ||
        d->s >= lim || d->stride_h >= lim || d->stride_w >= lim)
        return IGEMM_ENOTSUP;
    int64_t xb;
    if (__builtin_mul_overflow(d->n, d->h, &xb) || __builtin_mul_overflow(xb, d->w, &xb) ||
        __builtin_mul_overflow(xb, d->c, &xb) || xb > (0x7fff0000 - 64) / es)
        return IGEMM_ENOTSUP;
    if (M > INT_MAX || K > INT_MAX - 65536 || N > INT_MAX) return IGEMM_ENOTSUP;
    // Filter window offsets; (K + 2) * N < 2^62 after the bounds above.
    if ((K + 2) * N * es + 64 >= 0x7fff0000) return IGEMM_ENOTSUP;
    // Runs: with horizontal dilation 1 the taps of one filter row are
    // s * c consecutive input elements; the jump to the next filter row must
    // fit in 31 bits.
    // (dh as the kernel uses it: 1 for a one-row filter, else below 2^30.)
    const int64_t dh = d->r == 1 ? 1 : d->dil_h;
    const int64_t run2 = dh * d->w * d->c - d->s * d->c;
    // A 16-byte chunk then spans at most two runs if s * c >= 16 / es - 1.
    const bool runs = (d->s == 1 || d->dil_w == 1) && dh * d->w * d->c < ((int64_t)1 << 30) &&
                      d->s * d->c < ((int64_t)1 << 30) && d->s * d->c >= 16 / es - 1;
    // The small-output kernel gathers whole 64-channel k-tiles of one filter
    // tap (channels a multiple of 64, 16-byte aligned input and weights), or,
    // in its ragged variant, input runs through registers (any channel count;
    // 16-byte aligned weights with rows of whole 16 bytes).
    const bool small_conv = es == 2 && d->c % 64 == 0 && (uintptr_t)X % 16 == 0 &&
                            small_ok(M, N, K, X, K, W, N, N);
    const bool small_runs = es == 2 && !small_conv && runs &&
                            small_rg_ok(M, N, K, X, K, W, N, N);
    int id = kernel;
    if (id < 0) {
        // The rules of the GEMM planner's fused kernels (no packed path: the
        // lowered matrix never exists).
        const int64_t ncu = num_cu > 0 ? num_cu : 256;
        if (es == 2 && (small_conv || small_runs) && small_pays(M, N, K, (int)ncu))
            id = K_I16_SMALL_64x64;
        else if (es == 2) {
            if (M <= 16) id = K_I16_16x128;
            else if (M <= 32) id = K_I16_32x128;
            else if (N > 64 && K > 256 &&
                     4 * tiles_of(K_I16_128x128, M, N) *
                             big_tile_split(tiles_of(K_I16_128x128, M, N), K, (int)ncu) >=
                         3 * ncu)
                id = K_I16_128x128;
            else if (tiles_of(K_I16_64x64, M, N) < 32) id = M <= 64 ? K_I16_32x128 : K_I16_16x128;
            else if (K <= kBK && tiles_of(K_I16_64x64, M, N) < ncu) id = K_I16_16x128;
            else id = K_I16_64x64;
        } else {
            id = M <= 16 ? K_I8_16x256 : K_I8_32x256;
        }
    }
    const bool conv_id = id == K_I16_128x128 || id == K_I16_64x64 || id == K_I16_32x128 ||
                         id == K_I16_16x128 || id == K_I8_32x256 || id == K_I8_16x256 ||
                         (id == K_I16_SMALL_64x64 && (small_conv || small_runs));
    if (!conv_id || kKernels[id].es != es) return IGEMM_EINVAL;
    int st = make_plan(es, M, N, K, X, K, W, N, N, num_cu, id, split, false, out);
    if (st != IGEMM_OK) return st;
    out->vec_a = (((uintptr_t)X % 16) == 0 && (d->c * es) % 16 == 0) ? 1 : 0;
    *gather = out->vec_a != 0 ? 1 : (runs ? 3 : 2);
    // the small-output kernel: whole taps by DMA, or runs
    if (id == K_I16_SMALL_64x64) *gather = small_conv ? 1 : 3;
    g->sc = (int)(d->s * d->c);
    g->run2 = (int)run2;
    g->by_sc = make_div((uint32_t)(d->s * d->c));
    g->h = (int)d->h;
    g->w = (int)d->w;
    g->c = (int)d->c;
    g->ohw = (int)(oh * ow);
    g->ow = (int)ow;
    g->s = (int)d->s;
    g->sh = (int)d->stride_h;
    g->sw = (int)d->stride_w;
    g->ph = (int)d->pad_h;
    g->pw = (int)d->pad_w;
    // A one-tap dimension never multiplies its dilation by anything but 0;
    // any dilation of a wider filter is below 2^30 since the window fits.
    g->dh = d->r == 1 ? 1 : (int)d->dil_h;
    g->dw = d->s == 1 ? 1 : (int)d->dil_w;
    g->x_bytes = (int)(xb * es);
    g->by_c = make_div((uint32_t)d->c);
    g->by_s = make_div((uint32_t)d->s);
    g->by_ohw = make_div((uint32_t)(oh * ow));
    g->by_ow = make_div((uint32_t)ow);
    return IGEMM_OK;
}

}  // namespace igemm

extern "C" {

int igemm_query_plan(int elem_bytes, int64_t m, int64_t n, int64_t k, const void *A,
                     int64_t lda, const void *B, int64_t ldb, const void *C, int64_t ldc,
                     int num_cu, int kernel, int split, igemm_plan *out) {
    if (out == NULL) return IGEMM_EINVAL;
    int st = igemm::validate(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc);
    if (st != IGEMM_OK) return st;
    return igemm::make_plan(elem_bytes, m, n, k, A, lda, B, ldb, ldc, num_cu, kernel, split,
                            true, out);
}

int igemm_num_kernels(void) { return igemm::K_COUNT; }

const char *igemm_kernel_name(int kernel) {
    if (kernel < 0 || kernel >= igemm::K_COUNT) return NULL;
    return igemm::kKernels[kernel].name;
}

const char *igemm_strerror(int status) {
    switch (status) {
        case IGEMM_OK: return "success";
        case IGEMM_EINVAL: return "invalid argument (nothing was enqueued)";
        case IGEMM_EHIP: return "HIP runtime call or kernel launch failed";
        case IGEMM_ENOTSUP:
            return "unsupported size (a dimension exceeds 2^31 - 1 or the grid 2^24 workgroups)";
        case IGEMM_ENOMEM: return "the caller's workspace is smaller than the call needs";
        case IGEMM_ESCRATCH:
            return "the call needs more scratch than the library's static device array holds "
                   "(IGEMM_NOALLOC_SCRATCH_BYTES)";
        default: return "unknown status";
    }
}

int igemm_version(void) { return 300; }

int64_t igemm_conv2d_out_dim(int64_t in, int64_t f, int64_t stride, int64_t pad, int64_t dil) {
    return igemm::conv_out_dim(in, f, stride, pad, dil);
}

int igemm_conv2d_query_plan(int elem_bytes, const igemm_conv2d_desc *desc, const void *X,
                            const void *W, const void *Y, int num_cu, int kernel, int split,
                            igemm_plan *out) {
    igemm::ConvGeom g;
    int gather = 0;
    return igemm::make_conv_plan(elem_bytes, desc, X, W, Y, num_cu, kernel, split, out, &g,
                                 &gather);
}

}  // extern "C"
