// Integer GEMM C += A B on gfx950 (CDNA4) int8 matrix cores: the fused
// kernel template. The instantiations live in igemm_fused_*.hip, a few tile
// shapes per translation unit so that the library compiles in parallel.
//
// Structure (the MI355X counterpart of the paper's blocked algorithm, Fig.
// "baseline GEMM", and of its micro-kernel, Sec. 5.2):
//   * each workgroup of four waves owns a bm x bn tile of C (loops L1/L3
//     become the grid; loop L2 over k becomes the in-kernel k loop);
//   * per k-tile of 64 elements the workgroup stages its A and B panels from
//     HBM into LDS (the packing routines of Sec. 4.1): A rows are already
//     k-contiguous, B rows are n-contiguous and are transposed in registers
//     with byte permutes so that LDS holds B k-contiguous per column, which is
//     the operand layout of the MFMA instructions; LDS rows are XOR-swizzled
//     in 16-byte chunks so that the staging writes and the fragment reads are
//     free of bank conflicts;
//   * each wave keeps its C tile in accumulator registers and runs int8
//     matrix-core instructions (v_mfma_i32_32x32x32_i8, or
//     v_mfma_i32_16x16x64_i8 for 16-row tiles) over the k-tile (loop L6:
//     rank-64 updates instead of rank-1);
//   * the epilogue adds the accumulators into C with int32 wraparound (the
//     C_r load / update / store of Sec. 5.2), by plain read-add-write, or by
//     32-bit atomic adds when the k range is sliced across workgroups.
//
// int16 operands run on the same int8 matrix cores through an exact limb
// split. With h = x >> 8 (arithmetic) and l = (x & 0xff) - 128, both in
// [-128, 127], x = 256 h + l + 128, and for one pair of operands
//   x y = 65536 hx hy + 256 (hx ly + lx hy) + lx ly
//         + 32768 (hx + hy) + 128 (lx + ly) + 16384.
// Summed over k this is four int8 products into three accumulator sets
// (S_hh, S_x, S_ll) plus row sums of A's limbs, column sums of B's limbs and
// a constant, all combined modulo 2^32 in the epilogue. Limbs of elements
// beyond k are zero, so they add nothing to any term. Partial sums in one
// workgroup stay below 2^31 because the host caps the k range per workgroup
// (kMaxKChunk).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "igemm.h"
#include "igemm_device.h"
#include "igemm_internal.h"

namespace igemm {
namespace {

// x / d for the invariant divisor d described by `dv` (exact for every x).
__device__ __forceinline__ u32 divu(u32 x, DivU32 dv) {
    const u32 t = __umulhi(x, dv.mul);
    return (t + ((x - t) >> dv.s1)) >> dv.s2;
}

// Value of `v` in lane (lane ^ X) within each group of 32 lanes (ds_swizzle
// in bit-mask mode: and-mask 0x1f, or-mask 0, xor-mask X).
template <int X>
__device__ __forceinline__ u32 swz_xor(u32 v) {
    static_assert(X > 0 && X < 32, "xor within 32 lanes");
    return (u32)__builtin_amdgcn_ds_swizzle((int)v, 0x1f | (X << 10));
}

// ---------------------------------------------------------------------------
// Small tiles (bm * bn <= 8192, LDS <= 64 KB) are held to 256 registers per
// lane so that two workgroups share a compute unit; larger tiles take one.
// AM selects where A comes from: 0, the row-major matrix A (lda); 1, 2 and 3,
// the IM2ROW rows of a convolution gathered from the NHWC input Ap (geometry
// g): 16 bytes at a time (1: the channel count is a multiple of a 16-byte
// chunk, so a chunk never straddles two filter taps), element by element (2),
// or (3, horizontal dilation 1) as the contiguous input runs that one filter
// row covers, with at most two unaligned 16-byte loads per chunk.
// EPI selects the update of C: 0, int32 C += A B modulo 2^32; 1, int16 C
// (passed through the int32 pointer) += srs(A B), the product converted to
// int16 by an arithmetic shift right by (epi & 0xff) bits, after adding half
// a unit when bit 8 of epi is set, and saturation, then added modulo 2^16.
template <int ES, int BM, int BN, int WM, int WN, int MF, bool VA, bool VB, bool SPLIT, int AM,
          int EPI = 0>
__global__ void __launch_bounds__(256, BM * BN <= 32 * 256 ? 2 : 1)
igemm_tiled(const void *__restrict__ Ap, int64_t lda, const void *__restrict__ Bp,
            int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int k,
            int kchunk, int tiles_m, int tiles_n, ConvGeom g, int epi) {
    constexpr int P = ES;                  // limb planes per operand
    constexpr int NACC = ES == 2 ? 3 : 1;  // accumulator sets
    typedef Mfma<MF> M;
    typedef typename M::acc_t acc_t;
    constexpr int TM = WM / MF, TN = WN / MF;
    static_assert(WM % MF == 0 && WN % MF == 0, "wave tile is a whole number of MFMA tiles");
    constexpr int WGN = BN / WN;
    static_assert((BM / WM) * WGN == 4, "four waves per workgroup");
    constexpr int APL = BM * 64, BPL = BN * 64;  // bytes per LDS plane
    constexpr int STAGE = P * (APL + BPL);
    constexpr int ACH = BM * 4 * ES;  // 16-byte A chunks per k-tile
    constexpr int ACT = (ACH + 255) / 256;
    constexpr int BUN = BN * ES;  // B units (4 rows x 16 bytes) per k-tile
    constexpr int BUT = (BUN + 255) / 256;
    constexpr int CPU = 16 / ES;  // columns per B unit
    static_assert((ACH & (ACH - 1)) == 0 && (BUN & (BUN - 1)) == 0, "power-of-two staging");
    constexpr int NST = 4;  // LDS stages of the pipeline
    static_assert(NST * STAGE >= 4 * 2 * (BM + BN), "LDS reuse for the limb sums");
    static_assert(NST * STAGE <= 160 * 1024, "gfx950 LDS");
    // The int16 conversion is not additive: one workgroup owns each output.
    static_assert(EPI == 0 || !SPLIT, "no k slices with the int16-output update");

    __shared__ __attribute__((aligned(16))) char smem[NST * STAGE];

    // The kernel arguments are read from memory: loaded where first used, two
    // or three dependent round trips would open every workgroup. Naming them
    // all here issues their loads together.
    asm volatile("" ::"s"(Ap), "s"(lda), "s"(Bp), "s"(ldb), "s"(C), "s"(ldc), "s"(m), "s"(n),
                 "s"(k), "s"(kchunk), "s"(tiles_m), "s"(tiles_n), "s"(gridDim.x), "s"(epi));
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm0 = (wave / WGN) * WM;
    const int wn0 = (wave % WGN) * WN;

    // Workgroup -> (tile, k slice). Consecutive workgroup ids are dealt to the
    // eight XCDs in turn; renumber them so each XCD receives a contiguous range
    // of tiles, then walk tiles in groups of 8 tile-rows so that the tiles
    // running together on one XCD share A rows and B columns in its L2.
    int bid = blockIdx.x;
    const int G = gridDim.x;
    if ((G & 7) == 0) bid = (bid & 7) * (G >> 3) + (bid >> 3);
    const int tiles = tiles_m * tiles_n;
    const int z = bid / tiles;
    const int t = bid - z * tiles;
    constexpr int GROUP = 8;
    const int span = GROUP * tiles_n;
    const int first_m = (t / span) * GROUP;
    const int gsize = min(tiles_m - first_m, GROUP);
    const int tm = first_m + (t % span) % gsize;
    const int tn = (t % span) / gsize;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = z * kchunk;
    const int kend = min(k, kbeg + kchunk);
    if (kbeg >= kend) return;  // uniform over the workgroup

    const int8_t *A8 = (const int8_t *)Ap;
    const int8_t *B8 = (const int8_t *)Bp;

    // ---- per-thread staging geometry (fixed over the k loop) ---------------
    // Slots beyond the tile (fewer chunks than threads) repeat a real chunk;
    // they write the same bytes to the same LDS address and are left out of
    // the limb sums.
    int a_row[ACT], a_q[ACT], a_woff[ACT];
    bool a_dup[ACT];
#pragma unroll
    for (int s = 0; s < ACT; ++s) {
        const int c = tid + 256 * s;
        a_dup[s] = c >= ACH;
        const int ce = c & (ACH - 1);
        a_row[s] = ce / (4 * ES);
        a_q[s] = ce % (4 * ES);
        a_woff[s] = ES == 1 ? lds_off(a_row[s], a_q[s])
                            : lds_off(a_row[s], a_q[s] >> 1) + ((a_q[s] & 1) << 3);
    }
    int b_rg[BUT], b_cc[BUT];
    bool b_dup[BUT];
    int b_wbase[BUT][4];  // [slot][compile-time swizzle class of the column]
#pragma unroll
    for (int s = 0; s < BUT; ++s) {
        const int u = tid + 256 * s;
        b_dup[s] = u >= BUN;
        const int ue = u & (BUN - 1);
        // Consecutive lanes take consecutive row groups: their transposed LDS
        // writes then spread over all banks. (Taking consecutive column chunks
        // instead reads whole cache lines per load, but puts sixteen lanes of
        // one LDS write on the same banks, which measured slower.)
        b_rg[s] = ue & 15;
        b_cc[s] = ue >> 4;
        // Column col = cc*CPU + c' of the unit goes to LDS row col, chunk
        // q ^ swz(col). For CPU = 16, swz(col) = g(c'); for CPU = 8,
        // swz(col) = g(c') ^ 2*(cc & 1), with g(c') = ((c' >> 1) ^ (c' >> 2)) & 3.
        // So the offset is a per-thread base for each g plus c' * 64.
        const int q = (b_rg[s] >> 2) ^ (CPU == 8 ? ((b_cc[s] & 1) << 1) : 0);
        const int base = b_cc[s] * CPU * 64 + ((b_rg[s] & 3) << 2);
#pragma unroll
        for (int g = 0; g < 4; ++g) b_wbase[s][g] = base + ((q ^ g) << 4);
    }
    // Fragment read bases (LDS byte offsets within a stage).
    // Fragment read bases: the MFMA tile rows start at multiples of 16, so
    // swz(row) depends only on the lane's row within the tile.
    const int fr = M::frag_row(lane);
    int a_rbase[M::KSTEPS], b_rbase[M::KSTEPS];
#pragma unroll
    for (int ks = 0; ks < M::KSTEPS; ++ks) {
        const int cq = (M::frag_chunk(lane, ks) ^ swz(fr)) << 4;
        a_rbase[ks] = (wm0 + fr) * 64 + cq;
        b_rbase[ks] = (wn0 + fr) * 64 + cq;
    }

    // Register sets for staged k-tiles: two for the pipeline; the short path
    // (a k range of at most NST tiles) loads every tile at once.
    constexpr bool SHORT = BM * BN <= 32 * 256;
    constexpr int NPAR = SHORT ? NST : 2;
    v4i ra[NPAR][ACT];
    v4i rb[NPAR][BUT][4];
    int sah[ACT], sal[ACT];
    int sbh[BUT][8], sbl[BUT][8];
#pragma unroll
    for (int s = 0; s < ACT; ++s) sah[s] = sal[s] = 0;
#pragma unroll
    for (int s = 0; s < BUT; ++s)
#pragma unroll
        for (int c = 0; c < 8; ++c) sbh[s][c] = sbl[s][c] = 0;

    acc_t acc[NACC][TM][TN];
#pragma unroll
    for (int a = 0; a < NACC; ++a)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < M::REGS; ++r) acc[a][i][j][r] = 0;

    // ---- global -> registers, interior tiles: no bounds checks --------------
    // Row offsets fit in 32 bits (checked on the host), so each load is a
    // uniform 64-bit base plus a 32-bit per-lane offset.
    uint32_t a_goff[ACT], b_goff[BUT];
#pragma unroll
    for (int s = 0; s < ACT; ++s)
        a_goff[s] = (uint32_t)(((int64_t)a_row[s] * lda + a_q[s] * (16 / ES)) * ES);
#pragma unroll
    for (int s = 0; s < BUT; ++s)
        b_goff[s] = (uint32_t)(((int64_t)(4 * b_rg[s]) * ldb + b_cc[s] * CPU) * ES);
    const int64_t ldb_bytes = ldb * ES;
    const int8_t *a_tile0 = A8 + (int64_t)m0 * lda * ES;
    const int8_t *b_tile0 = B8 + (int64_t)n0 * ES;

    auto load_fast = [&](auto par, int k0) __attribute__((always_inline)) {
        constexpr int R = decltype(par)::value;
        const int8_t *ab = a_tile0 + (int64_t)k0 * ES;
#pragma unroll
        for (int s = 0; s < ACT; ++s) ra[R][s] = *(const v4i *)(ab + a_goff[s]);
        const int8_t *bb = b_tile0 + (int64_t)k0 * ldb_bytes;
#pragma unroll
        for (int s = 0; s < BUT; ++s)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                rb[R][s][r] = *(const v4i *)(bb + r * ldb_bytes + b_goff[s]);
    };

    // ---- global -> registers, any tile: per-element bounds -------------------
    auto load_safe = [&](auto par, int k0) __attribute__((always_inline)) {
        constexpr int R = decltype(par)::value;
        const int klen = kend - k0;
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            const int gi = m0 + a_row[s];
            const int len = gi < m ? klen : 0;
            const int gic = gi < m ? gi : m - 1;
            const void *rowp = A8 + ((int64_t)gic * lda + k0) * ES;
            ra[R][s] = load16<ES, VA>(rowp, a_q[s] * (16 / ES), len);
        }
        const int nlen = n - n0;
#pragma unroll
        for (int s = 0; s < BUT; ++s) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int p = k0 + 4 * b_rg[s] + r;
                const int len = p < kend ? nlen : 0;
                const int pc = p < kend ? p : kend - 1;
                const void *rowp = B8 + ((int64_t)pc * ldb + n0) * ES;
                rb[R][s][r] = load16<ES, VB>(rowp, b_cc[s] * CPU, len);
            }
        }
    };

    // ---- range-checked loads through buffer resources ---------------------------
    // Buffer resources at the corner of this workgroup's A rows and B columns
    // (from kbeg), with 32-bit lane offsets. Rows of A beyond m, elements
    // beyond kend and rows of B beyond kend get an offset past the resource's
    // range, which the hardware returns as zero (per dword), so the loads need
    // no branches; the range ends at the matrix's last byte (rounded up to a
    // dword), so no load reaches past the allocation. Columns of B beyond n
    // only feed outputs beyond n, which are never stored. Used whenever the
    // workgroup's windows span less than 2 GiB.
    const int klen = kend - kbeg;
    const int64_t a_span = (int64_t)BM * lda * ES + (int64_t)klen * ES + 64;
    const int64_t b_span = (int64_t)(klen + 1) * ldb * ES + BN * ES + 64;
    const bool rs_ok = (AM != 0 || a_span < 0x7fff0000) && b_span < 0x7fff0000;
    const char *a_base = (const char *)Ap + ((int64_t)m0 * lda + kbeg) * ES;
    const char *b_base = (const char *)Bp + ((int64_t)kbeg * ldb + n0) * ES;
    const int64_t a_ext = ((int64_t)(m - 1 - m0) * lda + (k - kbeg)) * ES;
    const int64_t b_ext = ((int64_t)(k - 1 - kbeg) * ldb + (n - n0)) * ES;
    // Rows that are not 16-byte aligned are read with dword-aligned loads
    // from a dword-aligned resource base and shifted into place
    // (v_alignbyte), five dwords per 16 bytes.
    const u32 a_dl = AM == 3 ? (u32)((uintptr_t)Ap & 3)
                             : (AM != 0 ? 0u : (u32)((uintptr_t)a_base & 3));
    const u32 b_dl = (u32)((uintptr_t)b_base & 3);
    const int a_rec = AM != 0 ? ((g.x_bytes + (int)a_dl + 3) & ~3)
                              : (int)min((a_ext + a_dl + 3) & ~(int64_t)3, (int64_t)0x7ffffff0);
    const int b_rec = (int)min((b_ext + b_dl + 3) & ~(int64_t)3, (int64_t)0x7ffffff0);
    const __amdgpu_buffer_rsrc_t Ars = __builtin_amdgcn_make_buffer_rsrc(
        AM != 0 ? (void *)((const char *)Ap - a_dl) : (void *)(a_base - a_dl), 0, a_rec,
        0x00020000);
    const __amdgpu_buffer_rsrc_t Brs =
        __builtin_amdgcn_make_buffer_rsrc((void *)(b_base - b_dl), 0, b_rec, 0x00020000);
    const int lda_b = (int)(lda * ES), ldb_b = (int)(ldb * ES);
    // 16 bytes at byte offset `off` (from the unaligned base; dl is the base's
    // misalignment), every load unconditional: one vector load when rows are
    // 16-byte aligned (VEC, dl = 0), else an aligned 16-byte and 4-byte load
    // and a byte shift. The out-of-range offset 0x80000000 stays out of range
    // after adding dl and 16.
    auto load16_rs = [&](auto vec, __amdgpu_buffer_rsrc_t rs, u32 off, u32 dl)
                         __attribute__((always_inline)) -> v4i {
        if constexpr (decltype(vec)::value != 0) {
            return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
        } else {
            const u32 o = off + dl;
            const u32 oa = o & ~3u, sh = o & 3u;
            const v4i lo = __builtin_amdgcn_raw_buffer_load_b128(rs, oa, 0, 0);
            const u32 hi = (u32)__builtin_amdgcn_raw_buffer_load_b32(rs, oa + 16, 0, 0);
            v4i v;
            v.x = (int)__builtin_amdgcn_alignbyte((u32)lo.y, (u32)lo.x, sh);
            v.y = (int)__builtin_amdgcn_alignbyte((u32)lo.z, (u32)lo.y, sh);
            v.z = (int)__builtin_amdgcn_alignbyte((u32)lo.w, (u32)lo.z, sh);
            v.w = (int)__builtin_amdgcn_alignbyte(hi, (u32)lo.w, sh);
            return v;
        }
    };
    // IM2ROW: the output pixel of each A row this thread stages, decoded
    // once: first input row and column of its window (a row past m gets a
    // window that lies outside the image), and its image's first element.
    int cv_iy0[AM != 0 ? ACT : 1], cv_ix0[AM != 0 ? ACT : 1], cv_img[AM != 0 ? ACT : 1];
    // AM 3: positions [cv_lo, cv_hi) of a filter row's run of s*c elements
    // that fall inside the image horizontally.
    int cv_lo[AM == 3 ? ACT : 1], cv_hi[AM == 3 ? ACT : 1];
    if constexpr (AM != 0) {
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            const u32 i = (u32)(m0 + a_row[s]);
            const u32 img = divu(i, g.by_ohw);
            const u32 rem = i - img * (u32)g.ohw;
            const u32 oy = divu(rem, g.by_ow);
            const u32 ox = rem - oy * (u32)g.ow;
            const bool ok = (int)i < m;
            cv_iy0[s] = ok ? (int)oy * g.sh - g.ph : -(1 << 30);
            cv_ix0[s] = (int)ox * g.sw - g.pw;
            cv_img[s] = ok ? (int)img * g.h * g.w * g.c : 0;
            if constexpr (AM == 3) {
                const int x0 = cv_ix0[s];
                cv_lo[s] = min(max(-x0, 0), g.s) * g.c;
                cv_hi[s] = min(max(g.w - x0, 0), g.s) * g.c;
            }
        }
    }
    // Element offset in X of A[row of chunk s, column p], or -1 where the
    // filter tap falls outside the image (zero padding) or p is past the end.
    auto tap = [&](int s, u32 p) __attribute__((always_inline)) -> int {
        const u32 fyx = divu(p, g.by_c);
        const int ci = (int)(p - fyx * (u32)g.c);
        const u32 fy = divu(fyx, g.by_s);
        const int fx = (int)(fyx - fy * (u32)g.s);
        const int iy = cv_iy0[s] + (int)fy * g.dh;
        const int ix = cv_ix0[s] + fx * g.dw;
        const bool in = (u32)iy < (u32)g.h && (u32)ix < (u32)g.w;
        return in ? cv_img[s] + (iy * g.w + ix) * g.c + ci : -1;
    };
    // One load per element of the 16 bytes at column p (AM 2, and the rare
    // chunks AM 3 cannot read as runs).
    auto gather_elems = [&](int s, int e, u32 p) __attribute__((always_inline)) -> v4i {
        u32 w4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int t = 0; t < 16 / ES; ++t) {
            const int o = e + t < klen ? tap(s, p + t) : -1;
            const u32 off = o >= 0 ? (u32)o * ES + a_dl : 0x80000000u;
            u32 v;
            if constexpr (ES == 2)
                v = (u32)__builtin_amdgcn_raw_buffer_load_b16(Ars, off, 0, 0);
            else
                v = (u32)__builtin_amdgcn_raw_buffer_load_b8(Ars, off, 0, 0);
            w4[(t * ES) >> 2] |= v << (8 * ((t * ES) & 3));
        }
        v4i r;
        r.x = (int)w4[0];
        r.y = (int)w4[1];
        r.z = (int)w4[2];
        r.w = (int)w4[3];
        return r;
    };
    // 16 bytes of IM2ROW row a_row[s] from element e of this workgroup's k
    // range: one vector load (AM 1: the chunk lies within one filter tap),
    // one load per element (AM 2), or runs (AM 3); out-of-image elements and
    // elements past the k range read as zero.
    auto gather16 = [&](int s, int e) __attribute__((always_inline)) -> v4i {
        const u32 p = (u32)(kbeg + e);
        if constexpr (AM == 1) {
            const int o = e < klen ? tap(s, p) : -1;
            return __builtin_amdgcn_raw_buffer_load_b128(
                Ars, o >= 0 ? (u32)o * ES : 0x80000000u, 0, 0);
        } else if constexpr (AM == 3) {
            // With horizontal dilation 1, the s*c columns of filter row fy
            // are consecutive input elements (one run), so the chunk is the
            // tail of run fy and the head of run fy + 1 (s*c >= 16/ES - 1,
            // checked on the host): element t comes from run 1 at
            // base1 + t or from run 2 at base2 + t, and is valid inside the
            // intervals [a1, b1) and [a2, b2).
            constexpr int E = 16 / ES;
            const u32 fy = divu(p, g.by_sc);
            const int q1 = (int)(p - fy * (u32)g.sc);
            const int iy1 = cv_iy0[s] + (int)fy * g.dh;
            const bool r1 = (u32)iy1 < (u32)g.h, r2 = (u32)(iy1 + g.dh) < (u32)g.h;
            // (modulo 2^32: exact for rows inside the image, unused otherwise)
            const int base1 = (int)((u32)cv_img[s] +
                                    ((u32)iy1 * (u32)g.w + (u32)cv_ix0[s]) * (u32)g.c + (u32)q1);
            const int base2 = (int)((u32)base1 + (u32)g.run2);
            const int split = g.sc - q1;  // elements of run 1 in the chunk
            const int kmax = klen - e;    // elements before the end of the k range
            const int a1 = max(cv_lo[s] - q1, 0);
            const int b1 = r1 ? min(min(cv_hi[s] - q1, split), kmax) : 0;
            const int a2 = split + cv_lo[s];
            const int b2 = r2 ? min(split + cv_hi[s], kmax) : 0;
            const bool need1 = a1 < b1 && a1 < E, need2 = a2 < b2 && a2 < E;
            // A run that starts before the tensor (only at the first image's
            // top-left corner, where leading elements are padding): elements.
            if ((need1 && base1 < 0) || (need2 && base2 < 0)) return gather_elems(s, e, p);
            const v4i v1 = load16_rs(ic<0>{}, Ars, need1 ? (u32)base1 * ES : 0x80000000u, a_dl);
            const v4i v2 = load16_rs(ic<0>{}, Ars, need2 ? (u32)base2 * ES : 0x80000000u, a_dl);
            const u32 w1[4] = {(u32)v1.x, (u32)v1.y, (u32)v1.z, (u32)v1.w};
            const u32 w2[4] = {(u32)v2.x, (u32)v2.y, (u32)v2.z, (u32)v2.w};
            u32 w4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int t = 0; t < E; ++t) {
                const int j = (t * ES) >> 2;
                const u32 em = (ES == 2 ? 0xffffu : 0xffu) << (8 * ((t * ES) & 3));
                const bool ok1 = t >= a1 && t < b1, ok2 = t >= a2 && t < b2;
                w4[j] |= (ok1 ? (w1[j] & em) : 0u) | (ok2 ? (w2[j] & em) : 0u);
            }
            v4i r;
            r.x = (int)w4[0];
            r.y = (int)w4[1];
            r.z = (int)w4[2];
            r.w = (int)w4[3];
            return r;
        } else {
            return gather_elems(s, e, p);
        }
    };
    // The k-tile starting kt0 elements after kbeg into register set R.
    auto load_rs = [&](auto par, int kt0) __attribute__((always_inline)) {
        constexpr int R = decltype(par)::value;
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            const int e = kt0 + a_q[s] * (16 / ES);  // first element, from kbeg
            if constexpr (AM == 0) {
                const u32 off = (m0 + a_row[s] < m && e < klen)
                                    ? (u32)(a_row[s] * lda_b + e * ES)
                                    : 0x80000000u;
                ra[R][s] = load16_rs(ic<VA>{}, Ars, off, a_dl);
            } else {
                ra[R][s] = gather16(s, e);
            }
        }
#pragma unroll
        for (int s = 0; s < BUT; ++s) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int p = kt0 + 4 * b_rg[s] + r;  // row of B, from kbeg
                const u32 off = p < klen ? (u32)(p * ldb_b + b_cc[s] * CPU * ES) : 0x80000000u;
                rb[R][s][r] = load16_rs(ic<VB>{}, Brs, off, b_dl);
            }
        }
    };

    // ---- registers -> LDS (limb split, B transpose, limb sums) --------------
    // MASK: zero the limbs of elements at or beyond kend (last k-tile only).
    auto store_tile = [&](auto par, auto buf, auto mask, int k0) __attribute__((always_inline)) {
        constexpr int R = decltype(par)::value;
        constexpr int BUF = decltype(buf)::value;
        constexpr bool MASK = decltype(mask)::value != 0;
        char *As = smem + BUF * STAGE;
        char *Bs = As + P * APL;
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            if constexpr (ES == 1) {
                *(v4i *)(As + a_woff[s]) = ra[R][s];
            } else {
                const u32 y0 = ra[R][s].x, y1 = ra[R][s].y, y2 = ra[R][s].z, y3 = ra[R][s].w;
                u32 h0 = perm(y1, y0, 0x07050301u), h1 = perm(y3, y2, 0x07050301u);
                u32 l0 = perm(y1, y0, 0x06040200u) ^ 0x80808080u;
                u32 l1 = perm(y3, y2, 0x06040200u) ^ 0x80808080u;
                if constexpr (MASK) {
                    const int v = kend - k0 - a_q[s] * 8;
                    const u32 m0k = byte_mask(v), m1k = byte_mask(v - 4);
                    h0 &= m0k;
                    l0 &= m0k;
                    h1 &= m1k;
                    l1 &= m1k;
                }
                sah[s] = sum4(h1, sum4(h0, sah[s]));
                sal[s] = sum4(l1, sum4(l0, sal[s]));
                *(uint2 *)(As + a_woff[s]) = make_uint2(h0, h1);
                *(uint2 *)(As + APL + a_woff[s]) = make_uint2(l0, l1);
            }
        }
#pragma unroll
        for (int s = 0; s < BUT; ++s) {
            u32 rmask = 0xffffffffu;
            if constexpr (ES == 2 && MASK) rmask = byte_mask(kend - (k0 + 4 * b_rg[s]));
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                u32 y[4];
                transpose4x4((u32)rb[R][s][0][d], (u32)rb[R][s][1][d], (u32)rb[R][s][2][d],
                             (u32)rb[R][s][3][d], y[0], y[1], y[2], y[3]);
                if constexpr (ES == 1) {
#pragma unroll
                    for (int t4 = 0; t4 < 4; ++t4) {
                        const int cp = 4 * d + t4;  // column within the unit
                        *(u32 *)(Bs + b_wbase[s][((cp >> 1) ^ (cp >> 2)) & 3] + cp * 64) = y[t4];
                    }
                } else {
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        // y[2h]: low bytes of column 2d+h, y[2h+1]: high bytes.
                        const u32 lo = (y[2 * h] ^ 0x80808080u) & rmask;
                        const u32 hi = y[2 * h + 1] & rmask;
                        const int cp = 2 * d + h;
                        sbh[s][cp] = sum4(hi, sbh[s][cp]);
                        sbl[s][cp] = sum4(lo, sbl[s][cp]);
                        const int off = b_wbase[s][((cp >> 1) ^ (cp >> 2)) & 3] + cp * 64;
                        *(u32 *)(Bs + off) = hi;
                        *(u32 *)(Bs + BPL + off) = lo;
                    }
                }
            }
        }
    };

    // ---- MFMA over one k-tile ----------------------------------------------
    // ---- LDS -> fragment registers, and the MFMAs of one k sub-step ---------
    // Two fragment slots: the MFMAs of one sub-step run on one slot while the
    // next sub-step's fragments load into the other.
    v4i fa[2][P][TM], fb[2][P][TN];
    auto read_frags = [&](auto slot, auto buf, auto ks) __attribute__((always_inline)) {
        constexpr int SL = decltype(slot)::value;
        constexpr int BUF = decltype(buf)::value;
        constexpr int KS = decltype(ks)::value;
        const char *As = smem + BUF * STAGE;
        const char *Bs = As + P * APL;
#pragma unroll
        for (int p = 0; p < P; ++p) {
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[SL][p][j] = *(const v4i *)(Bs + p * BPL + b_rbase[KS] + j * MF * 64);
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[SL][p][i] = *(const v4i *)(As + p * APL + a_rbase[KS] + i * MF * 64);
        }
    };
    auto mfmas = [&](auto slot) __attribute__((always_inline)) {
        constexpr int SL = decltype(slot)::value;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if constexpr (ES == 1) {
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] = M::mma(fa[SL][0][i], fb[SL][0][j], acc[0][i][j]);
            } else {
                // plane 0 = high limbs, plane 1 = offset low limbs
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] = M::mma(fa[SL][0][i], fb[SL][0][j], acc[0][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[1][i][j] = M::mma(fa[SL][0][i], fb[SL][1][j], acc[1][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[2][i][j] = M::mma(fa[SL][1][i], fb[SL][1][j], acc[2][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[1][i][j] = M::mma(fa[SL][1][i], fb[SL][0][j], acc[1][i][j]);
            }
        }
    };

    // One pipelined k-tile kt with S = kt mod 4. On entry LDS stages S and
    // S+1 hold tiles kt and kt+1, register set S&1 holds (or is receiving)
    // tile kt+2, and fragment slot 0 holds sub-step 0 of tile kt. The step
    // starts loading tile kt+3 into register set (S+1)&1, runs the MFMAs of
    // tile kt while reading the next sub-step's fragments (the last one from
    // stage S+1, already complete), writes tile kt+2 into stage S+2, and ends
    // with one barrier.
    // Pipeline loads (through the buffer resources; the plain vector loads
    // remain available for interior workgroups with aligned rows).
    auto load_p = [&](auto use_rs, auto par, int k0) __attribute__((always_inline)) {
        if constexpr (decltype(use_rs)::value != 0)
            load_rs(par, k0 - kbeg);
        else
            load_fast(par, k0);
    };
    auto step = [&](auto phase, auto do_load, auto do_store, auto do_pref, int kt, auto use_rs) __attribute__((always_inline)) {
        constexpr int S = decltype(phase)::value;
        if constexpr (M::KSTEPS == 2) {
            constexpr int NM = TM * TN * (ES == 2 ? 4 : 1);  // MFMAs per sub-step
            constexpr int NR = P * (TM + TN);                // fragment reads
            constexpr int NV = ACT + 4 * BUT;                 // global loads
            // staging work of one tile: perms, xors, limb sums, LDS writes
            constexpr int VALU = ES == 2 ? (10 * ACT + 56 * BUT) : (36 * BUT);
            constexpr int DSW = ES == 2 ? (2 * ACT + 16 * BUT) : (ACT + 16 * BUT);
            // sub-step 0 on slot 0 while sub-step 1 loads into slot 1 and the
            // global loads of tile kt+3 go out
            if (decltype(do_load)::value) load_p(use_rs, ic<(S + 1) & 1>{}, kbeg + (kt + 3) * 64);
            read_frags(ic<1>{}, ic<S>{}, ic<1>{});
            mfmas(ic<0>{});
            interleave<NM, NR, decltype(do_load)::value ? NV : 0, 0, 0>();
            __builtin_amdgcn_sched_barrier(0);
            // sub-step 1 on slot 1 while the next tile's sub-step 0 loads into
            // slot 0 and tile kt+2 is staged into LDS
            if (decltype(do_pref)::value) read_frags(ic<0>{}, ic<(S + 1) & 3>{}, ic<0>{});
            if (decltype(do_store)::value)
                store_tile(ic<S & 1>{}, ic<(S + 2) & 3>{}, ic<0>{}, kbeg + (kt + 2) * 64);
            mfmas(ic<1>{});
            interleave<NM, decltype(do_pref)::value ? NR : 0, 0,
                       decltype(do_store)::value ? (VALU + NM - 1) / NM : 0,
                       decltype(do_store)::value ? (DSW + NM - 1) / NM : 0>();
            __builtin_amdgcn_sched_barrier(0);
        } else {
            if (decltype(do_load)::value) load_p(use_rs, ic<(S + 1) & 1>{}, kbeg + (kt + 3) * 64);
            // one sub-step per tile; tiles alternate between the slots
            constexpr int SL = S & 1;
            if (decltype(do_store)::value)
                store_tile(ic<S & 1>{}, ic<(S + 2) & 3>{}, ic<0>{}, kbeg + (kt + 2) * 64);
            if (decltype(do_pref)::value) read_frags(ic<1 - SL>{}, ic<(S + 1) & 3>{}, ic<0>{});
            mfmas(ic<SL>{});
        }
        __syncthreads();
    };

    // One unpipelined k-tile through LDS stage 0, loads range-checked.
    auto safe_tile = [&](int k0) __attribute__((always_inline)) {
        if (rs_ok) {
            load_rs(ic<0>{}, k0 - kbeg);
        } else {
            if constexpr (AM == 0) load_safe(ic<0>{}, k0);
        }
        if (k0 + 64 > kend)
            store_tile(ic<0>{}, ic<0>{}, ic<1>{}, k0);
        else
            store_tile(ic<0>{}, ic<0>{}, ic<0>{}, k0);
        __syncthreads();
        read_frags(ic<0>{}, ic<0>{}, ic<0>{});
        mfmas(ic<0>{});
        if constexpr (M::KSTEPS == 2) {
            read_frags(ic<0>{}, ic<0>{}, ic<1>{});
            mfmas(ic<0>{});
        }
        __syncthreads();
    };

    // ---- epilogue (C += result), as a function of where C comes from ----------
    // cpre: C values loaded before the k loop (short path), or none.
    int32_t cpre[SHORT ? TM : 1][SHORT ? TN : 1][SHORT ? M::REGS : 1];
    // C is addressed through a buffer resource based at the tile's corner with
    // 32-bit byte offsets when bm rows of C span less than 2 GiB (the usual
    // case); elements outside m x n then get an offset beyond the resource's
    // range, which the hardware reads as zero and does not write, so loads
    // and stores need no branch per element. Otherwise 64-bit addresses with
    // a branch per element.
    constexpr int CE = EPI == 1 ? 2 : 4;  // bytes per C element
    int16_t *const C16 = (int16_t *)C;
    const bool c_rsrc = (int64_t)BM * ldc * CE < 0x7fff0000;
    const __amdgpu_buffer_rsrc_t Crs = __builtin_amdgcn_make_buffer_rsrc(
        (char *)C + ((int64_t)m0 * ldc + n0) * CE, 0, 0x7fffffff, 0x00020000);
    const int ldc32 = (int)ldc;
    auto c_off = [&](int lr, int lc) __attribute__((always_inline)) -> u32 {
        return (m0 + lr < m && n0 + lc < n) ? (u32)(lr * ldc32 + lc) * (u32)CE : 0x80000000u;
    };
    // One element of C through the resource (int16 C sign-extended).
    auto c_load = [&](u32 off) __attribute__((always_inline)) -> int32_t {
        if constexpr (EPI == 1)
            return (int32_t)(int16_t)__builtin_amdgcn_raw_buffer_load_b16(Crs, off, 0, 0);
        else
            return __builtin_amdgcn_raw_buffer_load_b32(Crs, off, 0, 0);
    };
    // The int16 conversion: shift and rounding offset.
    const int srs_shift = epi & 0xff;
    const int64_t srs_half =
        ((epi >> 8) & 1) != 0 && srs_shift > 0 ? (int64_t)1 << (srs_shift - 1) : 0;
    auto srs16 = [&](int64_t a) __attribute__((always_inline)) -> int32_t {
        const int64_t t = (a + srs_half) >> srs_shift;  // arithmetic: floor
        return (int32_t)(t > 32767 ? 32767 : (t < -32768 ? -32768 : t));
    };
    auto epilogue = [&](auto pre) __attribute__((always_inline)) {
        constexpr bool PRE = decltype(pre)::value != 0;
        // int16 correction terms of this k range, per row and per column,
        // parked in LDS: row i gets 32768 sum(H_A[i,:]) + 128 sum(L_A[i,:]),
        // column j the same of B plus the constant 16384 * (k range).
        // With the int16 conversion the sums stay separate and exact (two
        // words per row and per column): the conversion needs the product
        // itself, not its residue modulo 2^32.
        constexpr int RW = EPI == 1 ? 2 : 1;
        u32 *sR = (u32 *)smem;
        u32 *sK = sR + RW * BM;
        if constexpr (ES == 2) {
            // The eight 16-byte chunks of one row of A were staged by eight
            // consecutive lanes: a butterfly over them gives the row total.
#pragma unroll
            for (int s = 0; s < ACT; ++s) {
                if constexpr (EPI == 1) {
                    u32 vh = (u32)sah[s], vl = (u32)sal[s];
                    vh += swz_xor<1>(vh);
                    vl += swz_xor<1>(vl);
                    vh += swz_xor<2>(vh);
                    vl += swz_xor<2>(vl);
                    vh += swz_xor<4>(vh);
                    vl += swz_xor<4>(vl);
                    if (!a_dup[s] && a_q[s] == 0) {
                        sR[2 * a_row[s]] = vh;
                        sR[2 * a_row[s] + 1] = vl;
                    }
                } else {
                    u32 v = 32768u * (u32)sah[s] + 128u * (u32)sal[s];
                    v += swz_xor<1>(v);
                    v += swz_xor<2>(v);
                    v += swz_xor<4>(v);
                    if (!a_dup[s] && a_q[s] == 0) sR[a_row[s]] = v;
                }
            }
            // Sixteen consecutive lanes staged four rows each of the same
            // eight columns of B: a reduce-scatter over them (halving the
            // columns held at each exchange) leaves each even lane with the
            // total of one column.
            const u32 kconst = 16384u * (u32)(kend - kbeg);
            const bool h8 = (lane & 8) != 0, h4 = (lane & 4) != 0, h2 = (lane & 2) != 0;
            auto col_total = [&](const u32 *v8) __attribute__((always_inline)) -> u32 {
                u32 v4[4], v2[2];
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    v4[c] = (h8 ? v8[c + 4] : v8[c]) + swz_xor<8>(h8 ? v8[c] : v8[c + 4]);
#pragma unroll
                for (int c = 0; c < 2; ++c)
                    v2[c] = (h4 ? v4[c + 2] : v4[c]) + swz_xor<4>(h4 ? v4[c] : v4[c + 2]);
                u32 v1 = (h2 ? v2[1] : v2[0]) + swz_xor<2>(h2 ? v2[0] : v2[1]);
                return v1 + swz_xor<1>(v1);
            };
#pragma unroll
            for (int s = 0; s < BUT; ++s) {
                const int c = (h8 ? 4 : 0) + (h4 ? 2 : 0) + (h2 ? 1 : 0);
                const bool w = !b_dup[s] && (lane & 1) == 0;
                if constexpr (EPI == 1) {
                    u32 vh[8], vl[8];
#pragma unroll
                    for (int cc = 0; cc < 8; ++cc) {
                        vh[cc] = (u32)sbh[s][cc];
                        vl[cc] = (u32)sbl[s][cc];
                    }
                    const u32 th = col_total(vh), tl = col_total(vl);
                    if (w) {
                        sK[2 * (b_cc[s] * 8 + c)] = th;
                        sK[2 * (b_cc[s] * 8 + c) + 1] = tl;
                    }
                } else {
                    u32 v8[8];
#pragma unroll
                    for (int cc = 0; cc < 8; ++cc)
                        v8[cc] = 32768u * (u32)sbh[s][cc] + 128u * (u32)sbl[s][cc];
                    const u32 v1 = col_total(v8);
                    if (w) sK[b_cc[s] * 8 + c] = v1 + kconst;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            // row terms of this lane's REGS output rows of block i (groups of
            // four consecutive rows)
            u32 rowt[M::REGS];
            int rowh[EPI == 1 ? M::REGS : 1], rowl[EPI == 1 ? M::REGS : 1];
            if constexpr (ES == 2 && EPI == 1) {
#pragma unroll
                for (int r = 0; r < M::REGS; r += 4) {
                    const u32 *q = sR + 2 * (wm0 + MF * i + M::out_row(lane, r));
                    const uint4 q0 = *(const uint4 *)q, q1 = *(const uint4 *)(q + 4);
                    rowh[r] = (int)q0.x;
                    rowl[r] = (int)q0.y;
                    rowh[r + 1] = (int)q0.z;
                    rowl[r + 1] = (int)q0.w;
                    rowh[r + 2] = (int)q1.x;
                    rowl[r + 2] = (int)q1.y;
                    rowh[r + 3] = (int)q1.z;
                    rowl[r + 3] = (int)q1.w;
                }
            } else if constexpr (ES == 2) {
#pragma unroll
                for (int r = 0; r < M::REGS; r += 4) {
                    const uint4 q = *(const uint4 *)(sR + wm0 + MF * i + M::out_row(lane, r));
                    rowt[r] = q.x;
                    rowt[r + 1] = q.y;
                    rowt[r + 2] = q.z;
                    rowt[r + 3] = q.w;
                }
            }
            int32_t cl[TN][M::REGS];
            if constexpr (!PRE && !SPLIT) {
                if (c_rsrc) {
#pragma unroll
                    for (int j = 0; j < TN; ++j) {
                        const int lc = wn0 + MF * j + M::out_col(lane);
#pragma unroll
                        for (int r = 0; r < M::REGS; ++r)
                            cl[j][r] = c_load(c_off(wm0 + MF * i + M::out_row(lane, r), lc));
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int lc = wn0 + MF * j + M::out_col(lane);
                const int gc = n0 + lc;
                const u32 colt = ES == 2 && EPI == 0 ? sK[lc] : 0u;
                int colh = 0, coll = 0;
                if constexpr (ES == 2 && EPI == 1) {
                    const uint2 q = *(const uint2 *)(sK + 2 * lc);
                    colh = (int)q.x;
                    coll = (int)q.y;
                }
#pragma unroll
                for (int r = 0; r < M::REGS; ++r) {
                    const int lr = wm0 + MF * i + M::out_row(lane, r);
                    const int gr = m0 + lr;
                    if constexpr (EPI == 1) {
                        // The exact product of this k range, then the int16
                        // conversion and the update modulo 2^16.
                        int64_t a64;
                        if constexpr (ES == 1) {
                            a64 = (int64_t)acc[0][i][j][r];
                        } else {
                            a64 = (int64_t)acc[0][i][j][r] * 65536 +
                                  (int64_t)acc[1][i][j][r] * 256 + (int64_t)acc[2][i][j][r] +
                                  (int64_t)(rowh[r] + colh) * 32768 +
                                  (int64_t)(rowl[r] + coll) * 128 +
                                  (int64_t)(kend - kbeg) * 16384;
                        }
                        const int32_t tv = srs16(a64);
                        if (c_rsrc) {
                            const int32_t old = PRE ? cpre[i][j][r] : cl[j][r];
                            __builtin_amdgcn_raw_buffer_store_b16(
                                (unsigned short)(u32)(old + tv), Crs, c_off(lr, lc), 0, 0);
                        } else if (gr < m && gc < n) {
                            int16_t *cp = C16 + (int64_t)gr * ldc + gc;
                            const int32_t old = PRE ? cpre[i][j][r] : (int32_t)*cp;
                            *cp = (int16_t)(unsigned short)(u32)(old + tv);
                        }
                        continue;
                    }
                    u32 v;
                    if constexpr (ES == 1) {
                        v = (u32)acc[0][i][j][r];
                    } else {
                        v = 65536u * (u32)acc[0][i][j][r] + 256u * (u32)acc[1][i][j][r] +
                            (u32)acc[2][i][j][r] + rowt[r] + colt;
                    }
                    if constexpr (SPLIT) {
                        if (gr < m && gc < n) atomicAdd(C + (int64_t)gr * ldc + gc, (int)v);
                    } else if (c_rsrc) {
                        const u32 old = PRE ? (u32)cpre[i][j][r] : (u32)cl[j][r];
                        __builtin_amdgcn_raw_buffer_store_b32((int)(old + v), Crs, c_off(lr, lc), 0,
                                                              0);
                    } else if (gr < m && gc < n) {
                        int32_t *cp = C + (int64_t)gr * ldc + gc;
                        const u32 old = PRE ? (u32)cpre[i][j][r] : (u32)*cp;
                        *cp = (int32_t)(old + v);
                    }
                }
            }
            // Keep the scheduler from hoisting every C load of the tile at once.
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // C of this workgroup's tile into cpre (short path), to be consumed by the
    // epilogue: issued before the first operand loads, its round trip
    // overlaps theirs.
    auto prefetch_c = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int lc = wn0 + MF * j + M::out_col(lane);
#pragma unroll
                for (int r = 0; r < M::REGS; ++r) {
                    const int lr = wm0 + MF * i + M::out_row(lane, r);
                    if (c_rsrc) {
                        cpre[i][j][r] = c_load(c_off(lr, lc));
                    } else {
                        const int gr = min(m0 + lr, m - 1), gc = min(n0 + lc, n - 1);
                        if constexpr (EPI == 1)
                            cpre[i][j][r] = C16[(int64_t)gr * ldc + gc];
                        else
                            cpre[i][j][r] = C[(int64_t)gr * ldc + gc];
                    }
                }
            }
    };

    // ---- short path: a k range of at most NST k-tiles -------------------------
    // Small products (skinny, convolution-shaped, small cubes) give each
    // workgroup only a few k-tiles, too few to fill a pipeline: one global
    // round trip per tile would dominate. Here every tile of the range is
    // loaded at once with branch-free range-checked loads (a branch per load
    // would make the compiler wait for each load before issuing the next), C
    // is fetched at the same time, and one barrier precedes all the MFMAs.
    if constexpr (SHORT) {
        const int nkt = (kend - kbeg + 63) >> 6;
        if (nkt <= NST && rs_ok) {
            if constexpr (!SPLIT) prefetch_c();
            // Only the k-tiles of the range (nkt is uniform over the workgroup).
            load_rs(ic<0>{}, 0);
            if (nkt > 1) load_rs(ic<1>{}, 64);
            if (nkt > 2) load_rs(ic<2>{}, 128);
            if (nkt > 3) load_rs(ic<3>{}, 192);
            __builtin_amdgcn_sched_barrier(0);  // every load goes out before the first wait
            // Elements of A at or beyond kend (the next k slice) count as zero.
            auto mask_short = [&](auto par, auto tile) __attribute__((always_inline)) {
                constexpr int R = decltype(par)::value, T = decltype(tile)::value;
#pragma unroll
                for (int s = 0; s < ACT; ++s) {
                    const int vb = (klen - (T * 64 + a_q[s] * (16 / ES))) * ES;
                    ra[R][s].x &= (int)byte_mask(vb);
                    ra[R][s].y &= (int)byte_mask(vb - 4);
                    ra[R][s].z &= (int)byte_mask(vb - 8);
                    ra[R][s].w &= (int)byte_mask(vb - 12);
                }
            };
            mask_short(ic<0>{}, ic<0>{});
            store_tile(ic<0>{}, ic<0>{}, ic<1>{}, kbeg);
            if (nkt > 1) {
                mask_short(ic<1>{}, ic<1>{});
                store_tile(ic<1>{}, ic<1>{}, ic<1>{}, kbeg + 64);
            }
            if (nkt > 2) {
                mask_short(ic<2>{}, ic<2>{});
                store_tile(ic<2>{}, ic<2>{}, ic<1>{}, kbeg + 128);
            }
            if (nkt > 3) {
                mask_short(ic<3>{}, ic<3>{});
                store_tile(ic<3>{}, ic<3>{}, ic<1>{}, kbeg + 192);
            }
            __syncthreads();
            auto tile_mfmas = [&](auto buf) __attribute__((always_inline)) {
                read_frags(ic<0>{}, buf, ic<0>{});
                mfmas(ic<0>{});
                if constexpr (M::KSTEPS == 2) {
                    read_frags(ic<1>{}, buf, ic<1>{});
                    mfmas(ic<1>{});
                }
            };
            tile_mfmas(ic<0>{});
            if (nkt > 1) tile_mfmas(ic<1>{});
            if (nkt > 2) tile_mfmas(ic<2>{});
            if (nkt > 3) tile_mfmas(ic<3>{});
            __syncthreads();  // the epilogue reuses stage 0 for the limb sums
            epilogue(ic<1>{});
            return;
        }
    }

    // ---- main loop ------------------------------------------------------------
    // A multiple of four full k-tiles runs through the pipeline, with loads
    // through the buffer resources (any alignment, edge workgroups
    // included); the leading remainder of full tiles and the partial last
    // tile take the single-tile path, and so does everything when a window
    // spans 2 GiB or more.
    const int nfull = (kend - kbeg) >> 6;  // k-tiles with all 64 elements inside
    const int npipe = rs_ok ? (nfull & ~3) : 0;
    const int klead = kbeg + (nfull - npipe) * 64 * (npipe > 0);
    if (npipe > 0)
        for (int k0 = kbeg; k0 < klead; k0 += 64) safe_tile(k0);
    auto pipe = [&](auto use_rs) __attribute__((always_inline)) {
        const int kb = klead;  // first pipelined k-tile
        // Prologue: tiles 0, 1 into stages 0, 1; tile 2 into register
        // set 0; fragments of tile 0, sub-step 0 into slot 0.
        load_p(use_rs, ic<0>{}, kb);
        load_p(use_rs, ic<1>{}, kb + 64);
        store_tile(ic<0>{}, ic<0>{}, ic<0>{}, kb);
        store_tile(ic<1>{}, ic<1>{}, ic<0>{}, kb + 64);
        load_p(use_rs, ic<0>{}, kb + 128);
        __syncthreads();
        read_frags(ic<0>{}, ic<0>{}, ic<0>{});
        // The steps address tiles relative to kbeg; shift by the lead.
        const int t0 = (kb - kbeg) >> 6;
        int kt = 0;
        for (; kt < npipe - 4; kt += 4) {
            step(ic<0>{}, ic<1>{}, ic<1>{}, ic<1>{}, t0 + kt, use_rs);
            step(ic<1>{}, ic<1>{}, ic<1>{}, ic<1>{}, t0 + kt + 1, use_rs);
            step(ic<2>{}, ic<1>{}, ic<1>{}, ic<1>{}, t0 + kt + 2, use_rs);
            step(ic<3>{}, ic<1>{}, ic<1>{}, ic<1>{}, t0 + kt + 3, use_rs);
        }
        step(ic<0>{}, ic<1>{}, ic<1>{}, ic<1>{}, t0 + kt, use_rs);
        step(ic<1>{}, ic<0>{}, ic<1>{}, ic<1>{}, t0 + kt + 1, use_rs);
        step(ic<2>{}, ic<0>{}, ic<0>{}, ic<1>{}, t0 + kt + 2, use_rs);
        step(ic<3>{}, ic<0>{}, ic<0>{}, ic<0>{}, t0 + kt + 3, use_rs);
    };
    if (npipe > 0) pipe(ic<1>{});
    const int ktail = npipe > 0 ? klead + npipe * 64 : kbeg;
    for (int k0 = ktail; k0 < kend; k0 += 64) safe_tile(k0);

    epilogue(ic<0>{});
}

// ---------------------------------------------------------------------------
// Host stub of one GEMM variant (A row-major).
template <int ES, int BM, int BN, int WM, int WN, int MF>
const void *pick(bool va, bool vb, bool split) {
#define IGEMM_K(a, b, s) (const void *)&igemm_tiled<ES, BM, BN, WM, WN, MF, a, b, s, 0>
    if (split) {
        if (va) return vb ? IGEMM_K(true, true, true) : IGEMM_K(true, false, true);
        return vb ? IGEMM_K(false, true, true) : IGEMM_K(false, false, true);
    }
    if (va) return vb ? IGEMM_K(true, true, false) : IGEMM_K(true, false, false);
    return vb ? IGEMM_K(false, true, false) : IGEMM_K(false, false, false);
#undef IGEMM_K
}

// Convolution variants (A gathered by IM2ROW; VA is unused) of the small
// tiles, which the planner chooses for lowered convolutions.
template <int ES, int BM, int BN, int WM, int WN, int MF, int AM>
const void *pick_conv_am(bool vb, bool split) {
#define IGEMM_C(b, s) (const void *)&igemm_tiled<ES, BM, BN, WM, WN, MF, false, b, s, AM>
    if (split) return vb ? IGEMM_C(true, true) : IGEMM_C(false, true);
    return vb ? IGEMM_C(true, false) : IGEMM_C(false, false);
#undef IGEMM_C
}

template <int ES, int BM, int BN, int WM, int WN, int MF>
const void *pick_conv(int gather, bool vb, bool split) {
    switch (gather) {
        case 1: return pick_conv_am<ES, BM, BN, WM, WN, MF, 1>(vb, split);
        case 2: return pick_conv_am<ES, BM, BN, WM, WN, MF, 2>(vb, split);
        case 3: return pick_conv_am<ES, BM, BN, WM, WN, MF, 3>(vb, split);
        default: return nullptr;
    }
}

// int16-output variants (Sec. 5.2 conversion) of the small tiles: A row-major,
// no k slices.
template <int ES, int BM, int BN, int WM, int WN, int MF>
const void *pick_srs(bool va, bool vb) {
#define IGEMM_S(a, b) (const void *)&igemm_tiled<ES, BM, BN, WM, WN, MF, a, b, false, 0, 1>
    if (va) return vb ? IGEMM_S(true, true) : IGEMM_S(true, false);
    return vb ? IGEMM_S(false, true) : IGEMM_S(false, false);
#undef IGEMM_S
}

}  // namespace
}  // namespace igemm
