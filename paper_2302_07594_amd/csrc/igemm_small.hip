// Small-output int16 kernel: C += A B for products whose output is too small
// to occupy the chip with whole-k tiles -- the lowered convolution layers
// with one large and two small dimensions (Sec. 2, Sec. 4.2), e.g. m = 49 to
// 3136 output pixels, n = 64 to 512 channels, k = 64 to 4608.
//
// Such a product is bound neither by the matrix cores nor by HBM: a few MB
// move and the work spreads over a few hundred workgroups, so the time is
// the launch plus each workgroup's latency chain. This kernel keeps that
// chain to one memory round trip in, one multiply pass and one write:
//   * each workgroup owns a 64 x 64 tile of C and a range of at most KTMAX
//     k-tiles of 64 (the k range is sliced across workgroups, gridDim.z);
//   * it issues every load at once: all its k-tiles of A and B move global
//     -> LDS unchanged by DMA (global_load_lds_dwordx4), and, when it is the
//     only slice, its C tile into registers alongside;
//   * after one wait it multiplies out of LDS: A fragments with
//     ds_read_b128, B fragments with transpose reads, each int16 element
//     split into its high and offset-low int8 limbs in registers, four
//     v_mfma_i32_32x32x32_i8 per 32 k (wave tile 32 x 32);
//   * the epilogue adds the limb corrections of its own k range (exact row
//     sums of A and column sums of B, from the raw fragments) and updates C
//     modulo 2^32: read-add-write from the prefetched values, or 32-bit
//     atomic adds when k is sliced.
// Exactness (Sec. 4.1 definition, int16 limb identity): with h = x >> 8 and
// l' = (x & 255) - 128,
//   sum_p x_p y_p = 65536 S_hh + 256 (S_hl' + S_l'h) + S_l'l'
//                   + 128 sum_p x_p + 128 sum_p y_p - 16384 k     (mod 2^32),
// summed per slice; the partial sums of at most 256 k never overflow.
//
// Preconditions (checked by the planner): A and B 16-byte aligned, rows a
// multiple of 16 bytes, k a multiple of 64, n a multiple of 8, and 32-bit
// byte offsets within one k-tile of each operand and within a C tile. The
// convolution variant gathers A from an NHWC input with a multiple of 64
// channels (below 2 GB). The ragged variant (RG) lifts the conditions on A
// and k: A's rows may start at any element and k may end inside a k-tile
// (the lowered 7x7 stem layer: k = 147, rows of 294 bytes); each lane then
// moves its 16-byte chunk of A through registers instead of by DMA, and B
// (still 16-byte aligned rows, n a multiple of 8) is read through a buffer
// resource whose range ends at its last element.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm.h"
#include "igemm_device.h"
#include "igemm_internal.h"
#include "igemm_lds.h"

namespace igemm {
namespace small {

using namespace lds;

constexpr int BM = 64, BN = 64;
constexpr int RA = 128;               // LDS bytes of one A row per k-tile (64 int16)
constexpr int RB = 128;               // LDS bytes of one B row (64 int16 columns)
constexpr int APL = BM * RA;          // 8 KB
constexpr int BPL = 64 * RB;          // 8 KB
constexpr int STAGE = APL + BPL;      // one k-tile of A and B

// 16-byte chunk c of LDS row r sits at c ^ swz(r). A: the fragment reads (16
// consecutive rows at one chunk per LDS cycle) cover 16 distinct 16-byte bank
// groups. B: a transpose read takes 4 consecutive k rows x 64 bytes for 32
// lanes; rows 2 apart share banks, so rows with bit 1 set move to the other
// half of their 128 bytes, and the 4 rows cover all 64 banks.
__device__ __forceinline__ int swz_a(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int swz_b(int row) { return 4 * ((row >> 1) & 1); }

// x / d for the invariant divisor d described by `dv` (the host's make_div).
__device__ __forceinline__ u32 div_inv(u32 x, DivU32 dv) {
    const u32 t = __umulhi(x, dv.mul);
    return (t + ((x - t) >> dv.s1)) >> dv.s2;
}

// KT: k-tiles per workgroup (the last k slice may hold fewer). CONV: A is the
// IM2ROW matrix of a convolution (Sec. 4.2) gathered from the NHWC input A
// with geometry g, whose channel count is a multiple of 64, so that each
// k-tile is 64 channels of one filter tap and each of its rows 128
// contiguous bytes of one input pixel, or zeros outside the image.
// RG: ragged A and k (see above); k is the true depth (ktiles = ceil(k / 64)).
template <int KT, bool SPLIT, bool CONV, bool RG = false>
__global__ void __launch_bounds__(256, 2)
igemm_small_i16(const char *__restrict__ A, int64_t lda, const char *__restrict__ B,
                int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int ktiles,
                ConvGeom g, int k) {
    // RG && CONV: the convolution's IM2ROW rows gathered as input runs (any
    // channel count; horizontal dilation 1 and s c >= 7, checked on the host).
    typedef Mfma<32> M;
    typedef M::acc_t acc_t;
    static_assert(KT >= 1 && KT <= 4, "at most four k-tiles in LDS");
    // One LDS array per k-tile: the compiler tells the DMA into each apart
    // and waits only for the one a read needs.
    __shared__ __attribute__((aligned(16))) char st0[STAGE];
    __shared__ __attribute__((aligned(16))) char st1[KT > 1 ? STAGE : 16];
    __shared__ __attribute__((aligned(16))) char st2[KT > 2 ? STAGE : 16];
    __shared__ __attribute__((aligned(16))) char st3[KT > 3 ? STAGE : 16];
    auto stage = [&](int kt) -> char * {
        return kt == 0 ? st0 : kt == 1 ? st1 : kt == 2 ? st2 : st3;
    };
    __shared__ u32 sums[BM + BN];

    // Every kernel argument is named up front so that their loads issue together.
    asm volatile("" ::"s"(A), "s"(lda), "s"(B), "s"(ldb), "s"(C), "s"(ldc), "s"(m), "s"(n),
                 "s"(ktiles), "s"(k));
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
    const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
    const int kt0 = blockIdx.z * KT;
    const int nkt = min(ktiles - kt0, KT);  // >= 1 (planner)

    // ---- every load, issued at once (below, before the multiply) -------------
    // Per k-tile each wave moves two 1 KB blocks of A (8 rows of 128 bytes
    // each) and two of B (8 k rows of 128 bytes). Lane i of a block writes LDS
    // bytes [16 i, 16 i + 16): row i / 8, physical chunk i % 8, and fetches the
    // logical chunk that the swizzle puts there. Rows of A beyond m read row
    // m - 1 and column chunks of B beyond n read the last chunk; their
    // products only reach outputs that are never written.
    u32 off[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const int b = 2 * wave + (d & 1);
        const int row = 8 * b + lane / 8, pc = lane % 8;
        if (d < 2) {
            const int grow = min(m0 + row, m - 1);
            off[d] = CONV ? 16u * (u32)(pc ^ swz_a(row))
                          : (u32)grow * (u32)(lda * 2) + 16u * (u32)(pc ^ swz_a(row));
        } else {
            const int col = min(n0 + 8 * (pc ^ swz_b(row)), n - 8);
            off[d] = (u32)row * (u32)(ldb * 2) + 2u * (u32)col;
        }
    }
    // IM2ROW: the output pixel of each of this lane's two A rows, decoded
    // once: first input row and column of its window and its image's first
    // pixel (a row past m gets a window outside the image). The input is
    // read through a buffer resource, so that taps outside the image (an
    // offset past its range) land in LDS as zeros.
    // RG: [cv_lo, cv_hi), the positions of a filter row's run of s c input
    // elements that lie inside the image horizontally.
    int cv_iy0[2], cv_ix0[2], cv_pix[2], cv_lo[2], cv_hi[2];
    __amdgpu_buffer_rsrc_t Xrs;
    u32 x_dl = 0;
    if constexpr (CONV) {
#pragma unroll
        for (int d = 0; d < 2; ++d) {
            const u32 p = (u32)(m0 + 8 * (2 * wave + d) + lane / 8);
            const bool ok = p < (u32)m;
            const u32 img = div_inv(p, g.by_ohw);
            const u32 rem = p - img * (u32)g.ohw;
            const u32 oy = div_inv(rem, g.by_ow);
            const u32 ox = rem - oy * (u32)g.ow;
            cv_iy0[d] = ok ? (int)oy * g.sh - g.ph : -(1 << 30);
            cv_ix0[d] = (int)ox * g.sw - g.pw;
            cv_pix[d] = ok ? (int)img * g.h * g.w : 0;
            cv_lo[d] = min(max(-cv_ix0[d], 0), g.s) * g.c;
            cv_hi[d] = min(max(g.w - cv_ix0[d], 0), g.s) * g.c;
        }
        // RG: based at the dword below X (X is 2-byte aligned)
        x_dl = RG ? (u32)((uintptr_t)A & 3) : 0u;
        Xrs = __builtin_amdgcn_make_buffer_rsrc((void *)(A - x_dl), 0,
                                                (int)(((u32)g.x_bytes + x_dl + 3) & ~3u),
                                                0x00020000);
    }
    // RG && CONV: chunk d's 8 IM2ROW elements from column p are the tail of
    // filter row fy's run (input elements base1 + t) and the head of run
    // fy + 1 (base2 + t), valid in [a1, b1) and [a2, b2) (inside the image
    // and before k); a run that starts before the tensor (the first image's
    // top-left corner, where its leading elements are padding) is read
    // element by element instead (bad).
    struct Runs {
        int base1, base2, a1, b1, a2, b2;
        bool need1, need2, bad;
    };
    auto runs = [&](int d, u32 p) -> Runs {
        Runs r;
        const u32 fy = div_inv(p, g.by_sc);
        const int q1 = (int)(p - fy * (u32)g.sc);
        const int iy1 = cv_iy0[d] + (int)fy * g.dh;
        const bool r1 = (u32)iy1 < (u32)g.h, r2 = (u32)(iy1 + g.dh) < (u32)g.h;
        // (modulo 2^32: exact for rows inside the image, unused otherwise)
        r.base1 = (int)((u32)cv_pix[d] * (u32)g.c +
                        ((u32)iy1 * (u32)g.w + (u32)cv_ix0[d]) * (u32)g.c + (u32)q1);
        r.base2 = (int)((u32)r.base1 + (u32)g.run2);
        const int split = g.sc - q1;
        const int kmax = k - (int)p;
        r.a1 = max(cv_lo[d] - q1, 0);
        r.b1 = r1 ? min(min(cv_hi[d] - q1, split), kmax) : 0;
        r.a2 = split + cv_lo[d];
        r.b2 = r2 ? min(split + cv_hi[d], kmax) : 0;
        r.need1 = r.a1 < r.b1 && r.a1 < 8;
        r.need2 = r.a2 < r.b2 && r.a2 < 8;
        r.bad = (r.need1 && r.base1 < 0) || (r.need2 && r.base2 < 0);
        return r;
    };
    // RG: A through a resource based at the dword below A (dl: A's offset in
    // that dword) that ends at A's last element; B through one that ends at
    // B's last element (its rows past k read as zeros).
    __amdgpu_buffer_rsrc_t Ars, Brs;
    u32 a_dl = 0;
    v4i av[RG ? KT : 1][2];
    u32 ah[RG ? KT : 1][2];
    v4i av2[RG && CONV ? KT : 1][2];
    u32 ah2[RG && CONV ? KT : 1][2];
    if constexpr (RG) {
        a_dl = (u32)((uintptr_t)A & 3);
        const int64_t a_ext = ((int64_t)(m - 1) * lda + k) * 2 + a_dl;
        const int64_t b_ext = ((int64_t)(k - 1) * ldb + n) * 2;
        if constexpr (!CONV)
            Ars = __builtin_amdgcn_make_buffer_rsrc((void *)(A - a_dl), 0,
                                                    (int)((a_ext + 3) & ~3), 0x00020000);
        Brs = __builtin_amdgcn_make_buffer_rsrc((void *)B, 0, (int)((b_ext + 3) & ~3),
                                                0x00020000);
    }
    // Every one of the KT tiles is moved, a short last slice repeating its
    // last tile (read, never multiplied), so that the waits below are fixed
    // counts.
    const int64_t b_step = 64 * ldb * 2;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
        const int64_t t = kt0 + min(kt, nkt - 1);
        // Opaque scalar bases: the loads take a scalar base and a 32-bit lane
        // offset instead of 64-bit vector addresses.
        const char *ak = A + t * 128;
        const char *bk = B + t * b_step;
        asm volatile("" : "+s"(ak), "+s"(bk));
        char *st = stage(kt);
        // B first: its addresses need no decoding.
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            const int dd = d ^ 2;   // B blocks (2, 3), then A blocks (0, 1)
            if ((CONV || RG) && dd < 2) continue;
            u32 o = off[dd];
            asm volatile("" : "+v"(o));
            const int b = 2 * wave + (dd & 1);
            if constexpr (RG)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    Brs, (lds_void *)(st + APL + b * 1024), 16, (int)((u32)t * (u32)b_step + o),
                    0, 0, 0);
            else
                dma16((dd < 2 ? ak : bk) + o, (lds_void *)(st + (dd < 2 ? 0 : APL) + b * 1024));
        }
        if constexpr (RG && CONV) {
            // each run's 16 bytes: an aligned 16-byte and 4-byte load each
            // (a run not needed, or read element by element, loads nothing)
#pragma unroll
            for (int d = 0; d < 2; ++d) {
                const int row = 8 * (2 * wave + d) + lane / 8;
                const u32 p = (u32)t * 64u + 8u * (u32)((lane % 8) ^ swz_a(row));
                const Runs r = runs(d, p);
                const u32 o1 = r.need1 && !r.bad ? ((u32)r.base1 * 2u + x_dl) & ~3u : 0x80000000u;
                const u32 o2 = r.need2 && !r.bad ? ((u32)r.base2 * 2u + x_dl) & ~3u : 0x80000000u;
                av[kt][d] = __builtin_amdgcn_raw_buffer_load_b128(Xrs, o1, 0, 0);
                ah[kt][d] = (u32)__builtin_amdgcn_raw_buffer_load_b32(Xrs, o1 + 16, 0, 0);
                av2[kt][d] = __builtin_amdgcn_raw_buffer_load_b128(Xrs, o2, 0, 0);
                ah2[kt][d] = (u32)__builtin_amdgcn_raw_buffer_load_b32(Xrs, o2 + 16, 0, 0);
            }
        } else if constexpr (RG) {
            // this lane's chunk of each of its two A rows: an aligned 16-byte
            // and 4-byte load (past A's end: zeros), shifted into place below
#pragma unroll
            for (int d = 0; d < 2; ++d) {
                const u32 oa = ((u32)t * 128u + off[d] + a_dl) & ~3u;
                av[kt][d] = __builtin_amdgcn_raw_buffer_load_b128(Ars, oa, 0, 0);
                ah[kt][d] = (u32)__builtin_amdgcn_raw_buffer_load_b32(Ars, oa + 16, 0, 0);
            }
        }
        if constexpr (CONV && !RG) {
            // k-tile t: channels [c0, c0 + 64) of filter tap (fy, fx)
            const u32 tap = div_inv((u32)t * 64u, g.by_c);
            const int c0 = (int)((u32)t * 64u - tap * (u32)g.c);
            const u32 fy = div_inv(tap, g.by_s);
            const int fx = (int)(tap - fy * (u32)g.s);
#pragma unroll
            for (int d = 0; d < 2; ++d) {
                const int iy = cv_iy0[d] + (int)fy * g.dh, ix = cv_ix0[d] + fx * g.dw;
                const bool in = (u32)iy < (u32)g.h && (u32)ix < (u32)g.w;
                const u32 o = in ? (u32)((cv_pix[d] + iy * g.w + ix) * g.c + c0) * 2u + off[d]
                                 : 0x80000000u;
                const int b = 2 * wave + d;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(Xrs, (lds_void *)(st + b * 1024), 16,
                                                         (int)o, 0, 0, 0);
            }
        }
    }
    // Nothing below moves above the loads: the address arithmetic of the
    // rest of the kernel would otherwise delay them.
    __builtin_amdgcn_sched_barrier(0);
    // C tile: a buffer resource at the tile's corner; elements outside C get
    // an offset beyond the range (loads return zero, stores are dropped).
    // Without k slices C is prefetched right behind the DMA.
    const __amdgpu_buffer_rsrc_t Crs = __builtin_amdgcn_make_buffer_rsrc(
        (char *)C + ((int64_t)m0 * ldc + n0) * 4, 0, 0x7fffffff, 0x00020000);
    const int ldc32 = (int)ldc;
    const int ocol = wn0 + M::out_col(lane);
    u32 coff[M::REGS];
#pragma unroll
    for (int r = 0; r < M::REGS; ++r) {
        const int orow = wm0 + M::out_row(lane, r);
        coff[r] = (m0 + orow < m && n0 + ocol < n) ? (u32)(orow * ldc32 + ocol) * 4u
                                                    : 0x80000000u;
    }
    int32_t cv[SPLIT ? 1 : M::REGS];
    if constexpr (!SPLIT) {
#pragma unroll
        for (int r = 0; r < M::REGS; ++r)
            cv[r] = __builtin_amdgcn_raw_buffer_load_b32(Crs, coff[r], 0, 0);
        __builtin_amdgcn_sched_barrier(0);
    }
    constexpr int NC = SPLIT ? 0 : M::REGS;  // loads issued after the DMA

    // ---- multiply -----------------------------------------------------------
    // A: lane row fr = lane % 32, k chunk q = 2 ks + lane / 32 of 16 elements
    // (32 bytes: two ds_read_b128). B: group g = lane / 16 covers columns
    // 16 (g % 2) + [0, 16) of the wave's 32 and k chunk 2 ks + g / 2; lane
    // u = lane % 16 addresses k row 16 q + 4 r + u / 4 at columns 4 (u % 4).
    const int fr = lane & 31, grp = lane >> 4, u = lane & 15;
    int a_rd[2][2], b_rd[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int q = 2 * ks + (lane >> 5);
        const int row = wm0 + fr;
#pragma unroll
        for (int h = 0; h < 2; ++h) a_rd[ks][h] = row * RA + 16 * ((2 * q + h) ^ swz_a(row));
        const int qb = 2 * ks + (grp >> 1);
        const int col = wn0 + 16 * (grp & 1) + 4 * (u & 3);
        const int krow = 16 * qb + (u >> 2);
        b_rd[ks] = APL + krow * RB + 16 * ((col >> 3) ^ swz_b(krow)) + 2 * (col & 7);
    }
    // Four accumulator sets (hh, hl', l'h, l'l'): no two consecutive matrix
    // instructions of a sub-step depend on each other.
    acc_t acc[4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int r = 0; r < M::REGS; ++r) acc[a][r] = 0;
    int rsum = 0, csum = 0;  // raw sums: row fr of A, column (lane % 32) of B
    // One k-tile from LDS: raw fragments of both sub-steps (32 k each), limb
    // split, the four limb products, and the raw sums.
    auto tile = [&](const char *st) {
        u32 ra[2][8], rb[2][8];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const v4i x = *(const v4i *)(st + a_rd[ks][h]);
                ra[ks][4 * h] = (u32)x.x;
                ra[ks][4 * h + 1] = (u32)x.y;
                ra[ks][4 * h + 2] = (u32)x.z;
                ra[ks][4 * h + 3] = (u32)x.w;
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const v2i y = tr16(st + b_rd[ks] + r * 4 * RB);
                rb[ks][2 * r] = (u32)y.x;
                rb[ks][2 * r + 1] = (u32)y.y;
            }
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const u32 *a = ra[ks], *b = rb[ks];
            const v4i ah = v4(hi4(a[1], a[0]), hi4(a[3], a[2]), hi4(a[5], a[4]), hi4(a[7], a[6]));
            const v4i al = v4(lo4(a[1], a[0]), lo4(a[3], a[2]), lo4(a[5], a[4]), lo4(a[7], a[6]));
            const v4i bh = v4(hi4(b[1], b[0]), hi4(b[3], b[2]), hi4(b[5], b[4]), hi4(b[7], b[6]));
            const v4i bl = v4(lo4(b[1], b[0]), lo4(b[3], b[2]), lo4(b[5], b[4]), lo4(b[7], b[6]));
            acc[0] = M::mma(ah, bh, acc[0]);
            acc[1] = M::mma(ah, bl, acc[1]);
            acc[2] = M::mma(al, bh, acc[2]);
            acc[3] = M::mma(al, bl, acc[3]);
#pragma unroll
            for (int x = 0; x < 8; ++x) {
                rsum = sum2(a[x], rsum);
                csum = sum2(b[x], csum);
            }
        }
    };
    // Loads complete in order: tile kt has landed once at most (KT - 1 - kt)
    // DMA groups of four and the C loads remain outstanding, so each tile is
    // multiplied as soon as every wave's share of it is in LDS.
    auto wait_vm = [](auto cnt) {
        constexpr int N = decltype(cnt)::value;
        __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
    };
    if constexpr (RG) {
        // Every A chunk and B tile has landed once only the C loads remain;
        // each lane shifts its A chunks into place, zeroes the elements at or
        // beyond k (their B rows are zeros or repeat nothing that counts: a
        // zero element of A contributes nothing, and the limb identity holds
        // element by element) and stores them where the DMA would have.
        wait_vm(ic<NC>{});
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
            const int t = kt0 + min(kt, nkt - 1);
#pragma unroll
            for (int d = 0; d < 2; ++d) {
                const int b = 2 * wave + d;
                const int row = 8 * b + lane / 8;
                if constexpr (CONV) {
                    const u32 p = (u32)t * 64u + 8u * (u32)((lane % 8) ^ swz_a(row));
                    const Runs r = runs(d, p);
                    u32 w[4] = {0u, 0u, 0u, 0u};
                    if (r.bad) {
                        // element by element (every valid element lies inside X)
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const bool in1 = e >= r.a1 && e < r.b1, in2 = e >= r.a2 && e < r.b2;
                            const u32 o = in1 ? (u32)(r.base1 + e) * 2u + x_dl
                                              : (in2 ? (u32)(r.base2 + e) * 2u + x_dl
                                                     : 0x80000000u);
                            w[e >> 1] |= (u32)__builtin_amdgcn_raw_buffer_load_b16(Xrs, o, 0, 0)
                                         << (16 * (e & 1));
                        }
                    } else {
                        const u32 s1 = ((u32)r.base1 * 2u + x_dl) & 3u;
                        const u32 s2 = ((u32)r.base2 * 2u + x_dl) & 3u;
                        const v4i x1 = av[kt][d], x2 = av2[kt][d];
                        const u32 v1[4] = {
                            __builtin_amdgcn_alignbyte((u32)x1.y, (u32)x1.x, s1),
                            __builtin_amdgcn_alignbyte((u32)x1.z, (u32)x1.y, s1),
                            __builtin_amdgcn_alignbyte((u32)x1.w, (u32)x1.z, s1),
                            __builtin_amdgcn_alignbyte(ah[kt][d], (u32)x1.w, s1)};
                        const u32 v2[4] = {
                            __builtin_amdgcn_alignbyte((u32)x2.y, (u32)x2.x, s2),
                            __builtin_amdgcn_alignbyte((u32)x2.z, (u32)x2.y, s2),
                            __builtin_amdgcn_alignbyte((u32)x2.w, (u32)x2.z, s2),
                            __builtin_amdgcn_alignbyte(ah2[kt][d], (u32)x2.w, s2)};
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const u32 em = 0xffffu << (16 * (e & 1));
                            const bool in1 = e >= r.a1 && e < r.b1, in2 = e >= r.a2 && e < r.b2;
                            w[e >> 1] |= (in1 ? v1[e >> 1] & em : 0u) | (in2 ? v2[e >> 1] & em : 0u);
                        }
                    }
                    *(v4i *)(stage(kt) + b * 1024 + lane * 16) = v4(w[0], w[1], w[2], w[3]);
                    continue;
                }
                const u32 sh = ((u32)t * 128u + off[d] + a_dl) & 3u;
                const v4i x = av[kt][d];
                const int valid = k - (64 * t + 8 * ((lane % 8) ^ swz_a(row)));
                v4i y;
                y.x = (int)(__builtin_amdgcn_alignbyte((u32)x.y, (u32)x.x, sh) &
                            byte_mask(2 * valid));
                y.y = (int)(__builtin_amdgcn_alignbyte((u32)x.z, (u32)x.y, sh) &
                            byte_mask(2 * (valid - 2)));
                y.z = (int)(__builtin_amdgcn_alignbyte((u32)x.w, (u32)x.z, sh) &
                            byte_mask(2 * (valid - 4)));
                y.w = (int)(__builtin_amdgcn_alignbyte(ah[kt][d], (u32)x.w, sh) &
                            byte_mask(2 * (valid - 6)));
                *(v4i *)(stage(kt) + b * 1024 + lane * 16) = y;
            }
        }
        // lgkmcnt(0): the stores are in LDS before the barrier
        __builtin_amdgcn_s_waitcnt((0xf) | (0x7 << 4) | (0x3 << 14));
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
            if (kt < nkt) tile(stage(kt));
    } else {
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
            if (kt == 0) wait_vm(ic<4 * (KT - 1) + NC>{});
            if (kt == 1) wait_vm(ic<4 * (KT > 2 ? KT - 2 : 0) + NC>{});
            if (kt == 2) wait_vm(ic<4 * (KT > 3 ? KT - 3 : 0) + NC>{});
            if (kt == 3) wait_vm(ic<NC>{});
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");  // no LDS read moves above the wait
            if (kt < nkt) tile(stage(kt));
        }
    }

    // ---- epilogue -----------------------------------------------------------
    // Lanes l and l + 32 hold complementary k chunks of the same row and
    // column. The waves of wave column 0 publish the row sums of their 32
    // rows, those of wave row 0 the column sums of their 32 columns.
    {
        const u32 rs = 128u * (u32)(rsum + __shfl_xor(rsum, 32));
        const u32 cs = 128u * (u32)(csum + __shfl_xor(csum, 32));
        if (lane < 32) {
            if (wn0 == 0) sums[wm0 + lane] = rs;
            if (wm0 == 0) sums[BM + wn0 + lane] = cs;
        }
    }
    __syncthreads();
    const u32 colt = (0u - 16384u * (u32)(64 * nkt)) + sums[BM + ocol];
#pragma unroll
    for (int r = 0; r < M::REGS; ++r) {
        const u32 v = 65536u * (u32)acc[0][r] + 256u * ((u32)acc[1][r] + (u32)acc[2][r]) +
                      (u32)acc[3][r] + colt + sums[wm0 + M::out_row(lane, r)];
        if constexpr (SPLIT)
            __builtin_amdgcn_raw_ptr_buffer_atomic_add_i32((int)v, Crs, (int)coff[r], 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b32((int)((u32)cv[r] + v), Crs, coff[r], 0, 0);
    }
}

}  // namespace small

using namespace small;

// One launch: grid (column tiles, row tiles, k slices of plan.k_chunk).
template <int KT, bool CONV, bool RG>
static void launch_kt(dim3 grid, bool split, hipStream_t s, const char *A, int64_t lda,
                      const char *B, int64_t ldb, int32_t *C, int64_t ldc, int m, int n,
                      int ktiles, const ConvGeom &g, int k) {
    if (split)
        igemm_small_i16<KT, true, CONV, RG><<<grid, 256, 0, s>>>(A, lda, B, ldb, C, ldc, m, n,
                                                                 ktiles, g, k);
    else
        igemm_small_i16<KT, false, CONV, RG><<<grid, 256, 0, s>>>(A, lda, B, ldb, C, ldc, m, n,
                                                                  ktiles, g, k);
}

// RG: the ragged variant (A at any alignment, any k).
template <bool CONV, bool RG>
static int launch_any(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                      int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                      const ConvGeom &g, void *stream) {
    const int64_t ktiles = (k + 63) / 64, ktpw = p.k_chunk / 64;
    // (the planner prevents both)
    if ((!RG && k % 64 != 0) || ktpw < 1 || ktpw > 4) return IGEMM_EINVAL;
    const int64_t slices = (ktiles + ktpw - 1) / ktpw;
    const dim3 grid((unsigned)((n + BN - 1) / BN), (unsigned)((m + BM - 1) / BM),
                    (unsigned)slices);
    const char *a = (const char *)A, *b = (const char *)B;
    hipStream_t s = (hipStream_t)stream;
    const bool split = slices > 1;
    const int mi = (int)m, ni = (int)n, kti = (int)ktiles, ki = (int)k;
    switch (ktpw) {
        case 1:
            launch_kt<1, CONV, RG>(grid, split, s, a, lda, b, ldb, C, ldc, mi, ni, kti, g, ki);
            break;
        case 2:
            launch_kt<2, CONV, RG>(grid, split, s, a, lda, b, ldb, C, ldc, mi, ni, kti, g, ki);
            break;
        case 3:
            launch_kt<3, CONV, RG>(grid, split, s, a, lda, b, ldb, C, ldc, mi, ni, kti, g, ki);
            break;
        default:
            launch_kt<4, CONV, RG>(grid, split, s, a, lda, b, ldb, C, ldc, mi, ni, kti, g, ki);
            break;
    }
    return hipGetLastError() == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

int launch_small(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                 int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                 void *stream) {
    const ConvGeom g = {};
    // vec_a = 0: A's rows are not whole aligned 16-byte chunks, or k ends
    // inside a k-tile (the ragged variant)
    if (p.vec_a == 0) return launch_any<false, true>(p, m, n, k, A, lda, B, ldb, C, ldc, g, stream);
    return launch_any<false, false>(p, m, n, k, A, lda, B, ldb, C, ldc, g, stream);
}

int launch_small_conv(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const ConvGeom &g,
                      int gather, const void *X, const void *W, int32_t *Y, int64_t ldy,
                      void *stream) {
    // gather 1: whole 64-channel taps by DMA; 3: input runs through registers
    if (gather == 3) return launch_any<true, true>(p, m, n, k, X, k, W, n, Y, ldy, g, stream);
    if (gather != 1) return IGEMM_EINVAL;
    return launch_any<true, false>(p, m, n, k, X, k, W, n, Y, ldy, g, stream);
}

}  // namespace igemm
