// Streaming kernel for int8 C += A B with few rows (blocks of 16 or 32 rows
// of A): the shapes of deep-learning inference with one large and two small
// dimensions (Sec. 2, Sec. 4.2), where B -- the weights -- is read exactly
// once and the time is the time to stream it from HBM.
//
// Such a product has too little reuse for the LDS-staged tile kernels to
// pay: what matters is how many bytes of B are in flight. So every wave
// streams its own 64-row steps of a 128-column block of B straight into
// registers, with all of its loads issued before the first use, and no
// wave ever waits for another until the end:
//   * lane l loads 8 consecutive bytes (columns 8(l%16) .. 8(l%16)+7) of
//     16 consecutive rows (16(l/16) .. 16(l/16)+15 of the step); sixteen
//     lanes of one load instruction cover one whole 128-byte row segment;
//   * 4x4 byte transposes in registers turn those 16 rows x 8 columns into
//     eight k-contiguous 16-byte column fragments, the B operand of
//     v_mfma_i32_16x16x64_i8 -- fragment c of lane l is column 8(l%16)+c,
//     so MFMA c computes the columns {8j + c};
//   * the A operand (a block of 16 or 32 rows of A) is read with one
//     16-byte load per lane and step; it stays in L2 across workgroups
//     (larger m is covered by more row blocks, each streaming B again);
//   * the waves of a workgroup take interleaved steps of one k range and
//     sum their accumulators through LDS at the end; each workgroup then
//     adds its m x 128 result into C (32-bit atomic adds when several
//     workgroups share a column block, else a plain read-add-write).
// Rows of B beyond k are read through a buffer resource whose range ends at
// B's last byte, so the hardware returns zeros for them; A's elements
// beyond k are masked to zero, which also cancels whatever the rows of B
// past k would contribute. Columns beyond n and rows beyond m produce
// accumulator entries that are never written back.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm.h"
#include "igemm_device.h"
#include "igemm_internal.h"
#include "igemm_lds.h"

namespace igemm {
namespace stream {

typedef unsigned int v2u __attribute__((ext_vector_type(2)));
typedef int v2i_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// 8 bytes at byte offset `off`: one 8-byte load (VEC) or eight byte loads.
template <bool VEC>
__device__ __forceinline__ v2u load8(__amdgpu_buffer_rsrc_t rs, u32 off) {
    if constexpr (VEC) {
        return __builtin_bit_cast(v2u, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
    } else {
        u32 w[2] = {0u, 0u};
#pragma unroll
        for (int b = 0; b < 8; ++b)
            w[b >> 2] |= (u32)__builtin_amdgcn_raw_buffer_load_b8(rs, off + b, 0, 0) << (8 * (b & 3));
        v2u r;
        r.x = w[0];
        r.y = w[1];
        return r;
    }
}

// 16 bytes at byte offset `off`: one 16-byte load (VEC) or sixteen byte loads.
template <bool VEC>
__device__ __forceinline__ v4u load16(__amdgpu_buffer_rsrc_t rs, u32 off) {
    if constexpr (VEC) {
        return __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    } else {
        u32 w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int b = 0; b < 16; ++b)
            w[b >> 2] |= (u32)__builtin_amdgcn_raw_buffer_load_b8(rs, off + b, 0, 0) << (8 * (b & 3));
        v4u r;
        r.x = w[0];
        r.y = w[1];
        r.z = w[2];
        r.w = w[3];
        return r;
    }
}

// MB: 16-row MFMA blocks per row block (16 * MB rows); WAVES: waves per
// workgroup; S: 64-row steps per wave; VA / VB: 16-byte aligned A rows / 8-byte aligned B
// rows; SPLIT: several workgroups add into one column block of C.
template <int MB, int WAVES, int S, bool VA, bool VB, bool SPLIT>
__global__ void __launch_bounds__(64 * WAVES)
igemm_stream_i8(const int8_t *__restrict__ A, int64_t lda, const int8_t *__restrict__ B,
                int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int k,
                int colblocks, int rowblocks) {
    constexpr int SPW = WAVES * S;  // steps per workgroup
    constexpr int NP = MB * 8;      // accumulator fragments per wave
    // Two blocks of 16 rows with eight waves sum over the waves in two phases
    // so that the LDS buffers hold half of the waves' accumulators (64 KB, two
    // workgroups per compute unit); otherwise every wave stores its own.
    constexpr bool TWO = MB == 2 && WAVES == 8;
    constexpr int H = TWO ? WAVES / 2 : WAVES;  // LDS buffers
    __shared__ v4u red[H][NP][64];

    // Fetch every kernel argument at once (each load where first used would
    // cost a memory round trip of its own).
    asm volatile("" ::"s"(A), "s"(lda), "s"(B), "s"(ldb), "s"(C), "s"(ldc), "s"(m), "s"(n),
                 "s"(k), "s"(colblocks), "s"(rowblocks));

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int q = lane >> 4;  // k chunk of the MFMA fragments
    const int i = lane & 15;  // row of A / column group of B
    // workgroup -> (column block, row block, k range), column blocks fastest
    const unsigned t = blockIdx.x / (unsigned)colblocks;
    const int cb = (int)(blockIdx.x - t * (unsigned)colblocks);
    const int rb = (int)(t % (unsigned)rowblocks);
    const int ks = (int)(t / (unsigned)rowblocks);
    const int j0 = cb * 128;
    const int i0 = rb * 16 * MB;
    const int mrows = min(m - i0, 16 * MB);  // rows of this block
    const int kbeg = ks * SPW * 64;

    // Resources based at the workgroup's window, ending at each matrix's last
    // byte (rounded up to a dword: the hardware range-checks whole dwords).
    const int8_t *bw = B + (int64_t)kbeg * ldb + j0;
    const int64_t b_ext = (int64_t)(k - 1 - kbeg) * ldb + (n - j0);
    const int b_rec = (int)min((b_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0);
    const __amdgpu_buffer_rsrc_t Brs =
        __builtin_amdgcn_make_buffer_rsrc((void *)bw, 0, b_rec, 0x00020000);
    const int8_t *aw = A + (int64_t)i0 * lda + kbeg;
    const int64_t a_ext = (int64_t)(mrows - 1) * lda + (k - kbeg);
    const int a_rec = (int)min((a_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0);
    const __amdgpu_buffer_rsrc_t Ars =
        __builtin_amdgcn_make_buffer_rsrc((void *)aw, 0, a_rec, 0x00020000);
    const u32 ldb32 = (u32)ldb, lda32 = (u32)lda;

    // ---- every load of the wave, issued up front ---------------------------
    v2u bv[S][16];
    v4u av[S][MB];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const int kl = (s * WAVES + wave) * 64;  // step's k offset in the window
        const u32 boff = (u32)(kl + 16 * q) * ldb32 + (u32)(8 * i);
#pragma unroll
        for (int r = 0; r < 16; ++r) bv[s][r] = load8<VB>(Brs, boff + (u32)r * ldb32);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            av[s][mb] = load16<VA>(Ars, (u32)(16 * mb + i) * lda32 + (u32)(kl + 16 * q));
    }

    // ---- transpose and multiply --------------------------------------------
    v4i acc[MB][8];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[mb][c] = v4i{0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < S; ++s) {
        // elements of A at or beyond k are zeroed
        const int valid = k - (kbeg + (s * WAVES + wave) * 64 + 16 * q);
        u32 amask[4];
#pragma unroll
        for (int d = 0; d < 4; ++d) amask[d] = byte_mask(valid - 4 * d);
        v4i a[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            a[mb].x = (int)(av[s][mb].x & amask[0]);
            a[mb].y = (int)(av[s][mb].y & amask[1]);
            a[mb].z = (int)(av[s][mb].z & amask[2]);
            a[mb].w = (int)(av[s][mb].w & amask[3]);
        }
        u32 frag[8][4];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int d = 0; d < 4; ++d)
                transpose4x4(bv[s][4 * d][h], bv[s][4 * d + 1][h], bv[s][4 * d + 2][h],
                             bv[s][4 * d + 3][h], frag[4 * h][d], frag[4 * h + 1][d],
                             frag[4 * h + 2][d], frag[4 * h + 3][d]);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const v4i b = v4i{(int)frag[c][0], (int)frag[c][1], (int)frag[c][2], (int)frag[c][3]};
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[mb][c] = Mfma<16>::mma(a[mb], b, acc[mb][c]);
        }
    }

    // ---- sum over the waves, then into C ------------------------------------
    // Fragment c of lane (q, i) is stored in slot 16q + (i ^ 2c) of row p of
    // a buffer: one fragment's writes fill 64 distinct slots, and the reads
    // below -- sixteen consecutive threads take c = 0..7 of two column groups
    // -- hit sixteen distinct 16-byte bank groups. In two phases the upper
    // half of the waves stores its sums first and the lower half adds its own.
    if (!TWO || wave >= WAVES - H) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
            red[wave - (WAVES - H)][p][16 * q + (i ^ (2 * (p & 7)))] =
                __builtin_bit_cast(v4u, acc[p >> 3][p & 7]);
    }
    __syncthreads();
    if constexpr (TWO) {
        if (wave < H) {
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                v4u &slot = red[wave][p][16 * q + (i ^ (2 * (p & 7)))];
                slot = slot + __builtin_bit_cast(v4u, acc[p >> 3][p & 7]);
            }
        }
        __syncthreads();
    }
    // Thread -> (fragment, lane) with the column 8i + c running fastest: each
    // write-back instruction covers 64 consecutive columns of one row of C.
    constexpr int NT = 64 * WAVES;
    static_assert((NP * 64) % NT == 0, "whole passes");
#pragma unroll
    for (int e0 = 0; e0 < NP * 64; e0 += NT) {
        const int e = e0 + (int)threadIdx.x;
        const int c = e & 7, ii = (e >> 3) & 15, qq = (e >> 7) & 3, mb = e >> 9;
        const int p = mb * 8 + c;
        const int slot = 16 * qq + (ii ^ (2 * c));
        v4u sum = red[0][p][slot];
#pragma unroll
        for (int w = 1; w < H; ++w) sum += red[w][p][slot];
        const int col = j0 + 8 * ii + c;
        const int row0 = 16 * mb + 4 * qq;  // output row of component 0
        if (col < n) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (row0 + r < mrows) {
                    int32_t *dst = C + (int64_t)(i0 + row0 + r) * ldc + col;
                    if constexpr (SPLIT)
                        atomicAdd(dst, (int)sum[r]);
                    else
                        *dst = (int)((u32)*dst + sum[r]);
                }
            }
        }
    }
}

template <int MB, int WAVES, int S, bool VA, bool VB>
const void *pick_split(bool split) {
    return split ? (const void *)igemm_stream_i8<MB, WAVES, S, VA, VB, true>
                 : (const void *)igemm_stream_i8<MB, WAVES, S, VA, VB, false>;
}

template <int MB>
const void *pick(int waves, int s, bool va, bool vb, bool split) {
    if (!va || !vb) {
        // unaligned operands: one configuration, byte loads where needed
        if (waves != 4 || s != 1) return nullptr;
        if (va) return pick_split<MB, 4, 1, true, false>(split);
        if (vb) return pick_split<MB, 4, 1, false, true>(split);
        return pick_split<MB, 4, 1, false, false>(split);
    }
    if (waves == 4 && s == 1) return pick_split<MB, 4, 1, true, true>(split);
    if (waves == 8 && s == 1) return pick_split<MB, 8, 1, true, true>(split);
    if (waves == 8 && s == 2) return pick_split<MB, 8, 2, true, true>(split);
    if constexpr (MB == 1)
        if (waves == 8 && s == 4) return pick_split<MB, 8, 4, true, true>(split);
    return nullptr;
}


// ---------------------------------------------------------------------------
// Column-per-wave variant (16-byte aligned operands with rows of whole 16
// bytes). The register kernel above gives every wave its own k steps of the
// whole 128-column block, so the waves' partial 16 MB x 128 results must be
// summed through LDS at the end -- for 32 rows that sum moves more LDS bytes
// than B itself. Here every wave owns 16 of the 128 columns for all of the
// workgroup's k range instead, so nothing is summed across waves:
//   * every byte of the workgroup's B window (SPW steps of 64 rows x 128
//     columns) and of its A window (16 MB rows x SPW 64 k) moves global ->
//     LDS by DMA (no registers), all issued at once, then one wait;
//   * a wave's B operands (its 16 columns x 16 k per lane) come from LDS with
//     gfx950 transpose reads (ds_read_b64_tr_b8: lane t of each 16-lane group
//     gathers byte t % 8 of the 8-byte vectors addressed by lanes t / 8 + 2 j,
//     j = 0..7, i.e. one column for 8 consecutive k rows), its A operands with
//     ds_read_b128, one v_mfma_i32_16x16x64_i8 per 16-row block and step;
//   * each wave then adds its 16 MB x 16 block into C (atomic adds when k is
//     sliced across workgroups, else read-add-write).
// B's rows past k lie beyond its buffer resource and read as zeros, so the
// elements of A past k (the next row's, or zeros past A's end) meet zeros; rows
// of A past m read as zeros and their outputs are not written; columns past
// n are multiplied and not written.
// LDS rows: B 128 bytes per k row, 16-byte chunk c of row r at c ^ (r & 7)
// (the 8 rows of one transpose read hit 8 distinct bank groups); A 64 bytes
// per row, chunk q of row r at q ^ swz(r).
template <int MB, int SPW, bool SPLIT>
__global__ void __launch_bounds__(512)
igemm_stream_lds(const int8_t *__restrict__ A, int64_t lda, const int8_t *__restrict__ B,
                 int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int k,
                 int colblocks, int rowblocks) {
    constexpr int BST = 64 * 128;      // B bytes per step
    constexpr int AST = MB * 16 * 64;  // A bytes per step
    static_assert(SPW == 4 || SPW == 8 || SPW == 16, "steps per workgroup");
    // One LDS array per step of B, so that the compiler tells the DMA into
    // each apart and a step's reads wait only for that step's data.
#define IGEMM_SB(i) __shared__ __attribute__((aligned(16))) char sB##i[SPW > i ? BST : 16]
    IGEMM_SB(0); IGEMM_SB(1); IGEMM_SB(2); IGEMM_SB(3); IGEMM_SB(4); IGEMM_SB(5);
    IGEMM_SB(6); IGEMM_SB(7); IGEMM_SB(8); IGEMM_SB(9); IGEMM_SB(10); IGEMM_SB(11);
    IGEMM_SB(12); IGEMM_SB(13); IGEMM_SB(14); IGEMM_SB(15);
#undef IGEMM_SB
    auto sb = [&](auto sc) -> char * {
        constexpr int S = decltype(sc)::value;
        if constexpr (S == 0) return sB0;
        else if constexpr (S == 1) return sB1;
        else if constexpr (S == 2) return sB2;
        else if constexpr (S == 3) return sB3;
        else if constexpr (S == 4) return sB4;
        else if constexpr (S == 5) return sB5;
        else if constexpr (S == 6) return sB6;
        else if constexpr (S == 7) return sB7;
        else if constexpr (S == 8) return sB8;
        else if constexpr (S == 9) return sB9;
        else if constexpr (S == 10) return sB10;
        else if constexpr (S == 11) return sB11;
        else if constexpr (S == 12) return sB12;
        else if constexpr (S == 13) return sB13;
        else if constexpr (S == 14) return sB14;
        else return sB15;
    };
    __shared__ __attribute__((aligned(16))) char sA[SPW * AST];
    asm volatile("" ::"s"(A), "s"(lda), "s"(B), "s"(ldb), "s"(C), "s"(ldc), "s"(m), "s"(n),
                 "s"(k), "s"(colblocks), "s"(rowblocks));
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const unsigned t = blockIdx.x / (unsigned)colblocks;
    const int cb = (int)(blockIdx.x - t * (unsigned)colblocks);
    const int rb = (int)(t % (unsigned)rowblocks);
    const int ks = (int)(t / (unsigned)rowblocks);
    const int j0 = cb * 128, i0 = rb * 16 * MB, kbeg = ks * SPW * 64;
    const int mrows = min(m - i0, 16 * MB);

    const int8_t *bw = B + (int64_t)kbeg * ldb + j0;
    const int64_t b_ext = (int64_t)(k - 1 - kbeg) * ldb + (n - j0);
    const __amdgpu_buffer_rsrc_t Brs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)bw, 0, (int)min((b_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0), 0x00020000);
    const int8_t *aw = A + (int64_t)i0 * lda + kbeg;
    const int64_t a_ext = (int64_t)(mrows - 1) * lda + (k - kbeg);
    const __amdgpu_buffer_rsrc_t Ars = __builtin_amdgcn_make_buffer_rsrc(
        (void *)aw, 0, (int)min((a_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0), 0x00020000);

    // ---- every load of the workgroup, by DMA -------------------------------
    // A first (every step reads it), then B step by step, so that step s can
    // start once A and B's steps up to s have landed.
    // A: SPW * MB blocks of 16 rows x 64 bytes, dealt to the waves in turn
    // (lane i: row i / 4, physical chunk i % 4, logical (i % 4) ^ swz(row)).
    {
        const int rr = lane / 4;
        const u32 off = 16u * (u32)((lane % 4) ^ swz(rr));
#pragma unroll
        for (int b0 = 0; b0 < SPW * MB; b0 += 8) {
            const int b = b0 + wave;
            if (b < SPW * MB) {
                const int s = b / MB, mb = b % MB;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    Ars, (lds_void *)(sA + s * AST + mb * 1024), 16,
                    (int)((u32)(16 * mb + rr) * (u32)lda + (u32)(64 * s) + off), 0, 0, 0);
            }
        }
    }
    // B: wave w moves rows 8 w .. 8 w + 7 of each step (lane i: row 8 w + i / 8,
    // physical chunk i % 8, which holds logical chunk (i % 8) ^ (row & 7)).
    {
        const int rr = 8 * wave + lane / 8;
        const u32 off = (u32)rr * (u32)ldb + 16u * (u32)((lane % 8) ^ (rr & 7));
        auto dma_step = [&](auto sc) {
            constexpr int S = decltype(sc)::value;
            if constexpr (S < SPW)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    Brs, (lds_void *)(sb(sc) + wave * 1024), 16,
                    (int)(off + (u32)(64 * S) * (u32)ldb), 0, 0, 0);
        };
        dma_step(ic<0>{}); dma_step(ic<1>{}); dma_step(ic<2>{}); dma_step(ic<3>{});
        dma_step(ic<4>{}); dma_step(ic<5>{}); dma_step(ic<6>{}); dma_step(ic<7>{});
        dma_step(ic<8>{}); dma_step(ic<9>{}); dma_step(ic<10>{}); dma_step(ic<11>{});
        dma_step(ic<12>{}); dma_step(ic<13>{}); dma_step(ic<14>{}); dma_step(ic<15>{});
    }

    // ---- multiply -------------------------------------------------------------
    // B: lane u of each 16-lane group q addresses k row 16 q + 8 h + u / 2 of the
    // step at the 8-byte half u % 2 of the wave's logical chunk; A: row
    // lane % 16 of each 16-row block, k chunk q.
    const int q = lane >> 4, u = lane & 15;
    int b_rd[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int row = 16 * q + 8 * h + u / 2;
        b_rd[h] = row * 128 + 16 * (wave ^ (row & 7)) + 8 * (u % 2);
    }
    const int a_rd = u * 64 + 16 * (q ^ swz(u));
    v4i acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = v4i{0, 0, 0, 0};
    // Step s: wait until this wave's DMA of A and of B's steps up to s has
    // landed (the SPW - 1 - s later steps may stay in flight), then for the
    // other waves' (barrier), then multiply.
    auto mul_step = [&](auto sc) {
        constexpr int S = decltype(sc)::value;
        if constexpr (S < SPW) {
            // s_waitcnt: vmcnt[3:0] = SPW - 1 - S, expcnt and lgkmcnt not waited on
            __builtin_amdgcn_s_waitcnt((SPW - 1 - S) | (0x7 << 4) | (0xf << 8));
            __builtin_amdgcn_s_barrier();
            const char *bs = sb(sc);
            const v2i_t b0 = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) v2i_t *)(lds_void *)(bs + b_rd[0]));
            const v2i_t b1 = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) v2i_t *)(lds_void *)(bs + b_rd[1]));
            const v4i b = v4i{b0.x, b0.y, b1.x, b1.y};
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const v4i a = *(const v4i *)(sA + S * AST + mb * 1024 + a_rd);
                acc[mb] = Mfma<16>::mma(a, b, acc[mb]);
            }
        }
    };
    mul_step(ic<0>{}); mul_step(ic<1>{}); mul_step(ic<2>{}); mul_step(ic<3>{});
    mul_step(ic<4>{}); mul_step(ic<5>{}); mul_step(ic<6>{}); mul_step(ic<7>{});
    mul_step(ic<8>{}); mul_step(ic<9>{}); mul_step(ic<10>{}); mul_step(ic<11>{});
    mul_step(ic<12>{}); mul_step(ic<13>{}); mul_step(ic<14>{}); mul_step(ic<15>{});

    // ---- into C ---------------------------------------------------------------
    const int col = j0 + 16 * wave + Mfma<16>::out_col(lane);
    if (col < n) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * mb + Mfma<16>::out_row(lane, r);
                if (row < mrows) {
                    int32_t *dst = C + (int64_t)(i0 + row) * ldc + col;
                    if constexpr (SPLIT)
                        atomicAdd(dst, acc[mb][r]);
                    else
                        *dst = (int)((u32)*dst + (u32)acc[mb][r]);
                }
            }
        }
    }
}

template <int MB, int SPW>
const void *pick_lds(bool split) {
    return split ? (const void *)igemm_stream_lds<MB, SPW, true>
                 : (const void *)igemm_stream_lds<MB, SPW, false>;
}

template <int MB>
const void *pick_lds_spw(int spw, bool split) {
    if (spw == 4) return pick_lds<MB, 4>(split);
    if (spw == 8) return pick_lds<MB, 8>(split);
    if (spw == 16) return pick_lds<MB, 16>(split);
    return nullptr;
}


// ---------------------------------------------------------------------------
// Ring variant of the column-per-wave kernel for long k ranges per workgroup
// (few k slices, so that C receives few atomic adds): the same LDS rows,
// swizzles, transpose reads and per-wave columns, but B and A move through
// a ring of R stages (one LDS array per stage, so that the compiler tells the
// DMA into each apart) instead of all being resident at once:
//   * R - 1 steps are in flight ahead of the one being multiplied; at step s
//     a wave waits for its own DMA of step s, the barrier then also covers
//     the other waves' and their reads of step s - 1, whose stage then takes
//     step s + R - 1;
//   * every wave moves one 1 KB block of B (8 rows) and 128 MB bytes of A
//     (2 MB rows, 8 MB lanes) per step, both by DMA;
//   * the workgroup's k range is `spw` steps (any count); steps past k read
//     zeros from B as in the kernel above.
template <int MB, int R, bool SPLIT>
__global__ void __launch_bounds__(512)
igemm_stream_ring(const int8_t *__restrict__ A, int64_t lda, const int8_t *__restrict__ B,
                  int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int k,
                  int colblocks, int rowblocks, int spw) {
    constexpr int BST = 64 * 128;      // B bytes per step
    constexpr int AST = MB * 16 * 64;  // A bytes per step
    static_assert(R == 4 || R == 8, "ring stages");
    // (one array per stage, B then A: the compiler tracks a limited number of
    // DMA destinations, and loses the per-stage waits beyond that)
#define IGEMM_RS(i) __shared__ __attribute__((aligned(16))) char rS##i[R > i ? BST + AST : 16]
    IGEMM_RS(0); IGEMM_RS(1); IGEMM_RS(2); IGEMM_RS(3);
    IGEMM_RS(4); IGEMM_RS(5); IGEMM_RS(6); IGEMM_RS(7);
#undef IGEMM_RS
    auto sb = [&](auto sc) -> char * {
        constexpr int S = decltype(sc)::value;
        if constexpr (S == 0) return rS0;
        else if constexpr (S == 1) return rS1;
        else if constexpr (S == 2) return rS2;
        else if constexpr (S == 3) return rS3;
        else if constexpr (S == 4) return rS4;
        else if constexpr (S == 5) return rS5;
        else if constexpr (S == 6) return rS6;
        else return rS7;
    };
    auto sa = [&](auto sc) -> char * { return sb(sc) + BST; };
    asm volatile("" ::"s"(A), "s"(lda), "s"(B), "s"(ldb), "s"(C), "s"(ldc), "s"(m), "s"(n),
                 "s"(k), "s"(colblocks), "s"(rowblocks), "s"(spw));
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const unsigned t = blockIdx.x / (unsigned)colblocks;
    const int cb = (int)(blockIdx.x - t * (unsigned)colblocks);
    const int rb = (int)(t % (unsigned)rowblocks);
    const int ks = (int)(t / (unsigned)rowblocks);
    const int j0 = cb * 128, i0 = rb * 16 * MB, kbeg = ks * spw * 64;
    const int mrows = min(m - i0, 16 * MB);
    const int nsteps = min(spw, (k - kbeg + 63) / 64);  // >= 1 (grid)

    const int8_t *bw = B + (int64_t)kbeg * ldb + j0;
    const int64_t b_ext = (int64_t)(k - 1 - kbeg) * ldb + (n - j0);
    const __amdgpu_buffer_rsrc_t Brs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)bw, 0, (int)min((b_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0), 0x00020000);
    const int8_t *aw = A + (int64_t)i0 * lda + kbeg;
    const int64_t a_ext = (int64_t)(mrows - 1) * lda + (k - kbeg);
    const __amdgpu_buffer_rsrc_t Ars = __builtin_amdgcn_make_buffer_rsrc(
        (void *)aw, 0, (int)min((a_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0), 0x00020000);

    // B: wave w moves rows 8 w .. 8 w + 7 of a step (lane i: row 8 w + i / 8,
    // physical chunk i % 8, logical (i % 8) ^ (row & 7)). A: wave w moves rows
    // 2 MB w .. 2 MB w + 2 MB - 1 (lane i < 8 MB: row 2 MB w + i / 4, physical
    // chunk i % 4, logical (i % 4) ^ swz(row)). Both by DMA written as inline
    // assembly: the compiler's own wait placement does not follow loads whose
    // data is used a loop iteration later and adds early waits before the LDS
    // reads, so the kernel keeps the count itself -- each wave issues exactly
    // two DMAs per step (the A one with its first 8 MB lanes active), and a
    // step waits until at most the later steps' are outstanding. Steps past
    // the workgroup's range are issued too, at an offset beyond both
    // resources (zeros, no memory traffic). The kernel makes no other use of
    // M0, which holds each DMA's LDS address.
    const int brow = 8 * wave + lane / 8;
    const u32 boff = (u32)brow * (u32)ldb + 16u * (u32)((lane % 8) ^ (brow & 7));
    const int arow = 2 * MB * wave + lane / 4;
    const u32 aoff = (u32)arow * (u32)lda + 16u * (u32)((lane % 4) ^ swz(arow));
    auto lds_addr = [](const char *p) -> u32 {
        return (u32)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
    };
    auto dma = [&](auto sc, int s) {
        const bool in = s < nsteps;
        const u32 bo = in ? boff + (u32)(64 * s) * (u32)ldb : 0x80000000u;
        const u32 bl = lds_addr(sb(sc) + wave * 1024);
        const __amdgpu_buffer_rsrc_t br = Brs;
        asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                     ::"v"(bo), "s"(br), "s"(bl)
                     : "memory");
        const u32 ao = in ? aoff + (u32)(64 * s) : 0x80000000u;
        const u32 al = lds_addr(sa(sc) + wave * 128 * MB);
        const __amdgpu_buffer_rsrc_t ar = Ars;
        if (lane < 8 * MB)
            asm volatile(
                "s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                ::"v"(ao), "s"(ar), "s"(al)
                : "memory");
    };

    const int q = lane >> 4, u = lane & 15;
    int b_rd[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int row = 16 * q + 8 * h + u / 2;
        b_rd[h] = row * 128 + 16 * (wave ^ (row & 7)) + 8 * (u % 2);
    }
    const int a_rd = u * 64 + 16 * (q ^ swz(u));
    v4i acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = v4i{0, 0, 0, 0};

    // prologue: steps 0 .. R - 2 into stages 0 .. R - 2
    dma(ic<0>{}, 0);
    dma(ic<1>{}, 1);
    dma(ic<2>{}, 2);
    if constexpr (R == 8) {
        dma(ic<3>{}, 3);
        dma(ic<4>{}, 4);
        dma(ic<5>{}, 5);
        dma(ic<6>{}, 6);
    }
    // step s (stage S = s % R): the R - 2 later steps' DMAs may stay in
    // flight; the barrier then covers every wave's DMAs of step s and their
    // reads of step s - 1, whose stage takes step s + R - 1.
    auto step = [&](auto sc, int s) {
        constexpr int S = decltype(sc)::value;
        constexpr int W = 2 * (R - 2);
        __builtin_amdgcn_s_waitcnt((W & 0xf) | ((W >> 4) << 14) | (0x7 << 4) | (0xf << 8));
        __builtin_amdgcn_s_barrier();
        dma(ic<(S + R - 1) % R>{}, s + R - 1);
        const char *bs = sb(sc);
        const v2i_t b0 = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
            (__attribute__((address_space(3))) v2i_t *)(lds_void *)(bs + b_rd[0]));
        const v2i_t b1 = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
            (__attribute__((address_space(3))) v2i_t *)(lds_void *)(bs + b_rd[1]));
        const v4i b = v4i{b0.x, b0.y, b1.x, b1.y};
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const v4i a = *(const v4i *)(sa(sc) + mb * 1024 + a_rd);
            acc[mb] = Mfma<16>::mma(a, b, acc[mb]);
        }
    };
    for (int s0 = 0; s0 < nsteps; s0 += R) {
        step(ic<0>{}, s0);
        if (s0 + 1 < nsteps) step(ic<1>{}, s0 + 1);
        if (s0 + 2 < nsteps) step(ic<2>{}, s0 + 2);
        if (s0 + 3 < nsteps) step(ic<3>{}, s0 + 3);
        if constexpr (R == 8) {
            if (s0 + 4 < nsteps) step(ic<4>{}, s0 + 4);
            if (s0 + 5 < nsteps) step(ic<5>{}, s0 + 5);
            if (s0 + 6 < nsteps) step(ic<6>{}, s0 + 6);
            if (s0 + 7 < nsteps) step(ic<7>{}, s0 + 7);
        }
    }

    const int col = j0 + 16 * wave + Mfma<16>::out_col(lane);
    if (col < n) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * mb + Mfma<16>::out_row(lane, r);
                if (row < mrows) {
                    int32_t *dst = C + (int64_t)(i0 + row) * ldc + col;
                    if constexpr (SPLIT)
                        atomicAdd(dst, acc[mb][r]);
                    else
                        *dst = (int)((u32)*dst + (u32)acc[mb][r]);
                }
            }
        }
    }
}

template <int MB>
const void *pick_ring(bool split) {
    return split ? (const void *)igemm_stream_ring<MB, 8, true>
                 : (const void *)igemm_stream_ring<MB, 8, false>;
}


// ---------------------------------------------------------------------------
// int16 column-per-wave variant (few-row int16 products whose B, the weights,
// dominates the traffic). As in the int8 kernel above, B moves to LDS once by
// DMA and each wave owns 16 columns for the workgroup's whole k range; here
// four waves cover 64 int16 columns (B rows of 128 bytes: the same LDS rows
// and swizzle), and every element is split into its high and offset-low int8
// limbs in registers (the int16 limb identity, Sec. 4.1 definition):
//   * A fragments (16 int16 of one row per lane) by two ds_read_b128, B
//     fragments (16 int16 of one column per lane) by four transpose reads
//     ds_read_b64_tr_b16, then the limb bytes by v_perm;
//   * four v_mfma_i32_16x16x64_i8 per 16-row block and step (hh, hl', l'h,
//     l'l') into three accumulators, and the exact row sums of A and column
//     sums of B (v_dot2 with ones) on the raw fragments;
//   * C += 65536 S_hh + 256 S_x + S_ll + 128 (row sum + column sum) - 16384 K
//     modulo 2^32 over the workgroup's K = 64 (steps) elements of k (atomic
//     adds when k is sliced).
// Preconditions (planner): A and B 16-byte aligned with rows of whole 16
// bytes, k a multiple of 64, n a multiple of 8. Steps past k (a short last
// slice) are loaded (reads past the resources' ranges return zeros) and not
// multiplied. Rows of A past m and columns past n are multiplied and not
// written.
template <int MB, int SPW, bool SPLIT>
__global__ void __launch_bounds__(256)
igemm_stream_lds16(const int16_t *__restrict__ A, int64_t lda, const int16_t *__restrict__ B,
                   int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int k,
                   int colblocks, int rowblocks) {
    using lds::hi4;
    using lds::lo4;
    using lds::sum2;
    using lds::v4;
    constexpr int BST = 64 * 128;       // B bytes per step: 64 k rows x 64 int16
    constexpr int AST = MB * 16 * 128;  // A bytes per step: 16 MB rows x 64 int16
    static_assert(SPW == 4 || SPW == 8, "steps per workgroup");
#define IGEMM_SB(i) __shared__ __attribute__((aligned(16))) char sB##i[SPW > i ? BST : 16]
    IGEMM_SB(0); IGEMM_SB(1); IGEMM_SB(2); IGEMM_SB(3);
    IGEMM_SB(4); IGEMM_SB(5); IGEMM_SB(6); IGEMM_SB(7);
#undef IGEMM_SB
    auto sb = [&](auto sc) -> char * {
        constexpr int S = decltype(sc)::value;
        if constexpr (S == 0) return sB0;
        else if constexpr (S == 1) return sB1;
        else if constexpr (S == 2) return sB2;
        else if constexpr (S == 3) return sB3;
        else if constexpr (S == 4) return sB4;
        else if constexpr (S == 5) return sB5;
        else if constexpr (S == 6) return sB6;
        else return sB7;
    };
    __shared__ __attribute__((aligned(16))) char sA[SPW * AST];
    asm volatile("" ::"s"(A), "s"(lda), "s"(B), "s"(ldb), "s"(C), "s"(ldc), "s"(m), "s"(n),
                 "s"(k), "s"(colblocks), "s"(rowblocks));
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const unsigned t = blockIdx.x / (unsigned)colblocks;
    const int cb = (int)(blockIdx.x - t * (unsigned)colblocks);
    const int rb = (int)(t % (unsigned)rowblocks);
    const int ks = (int)(t / (unsigned)rowblocks);
    const int j0 = cb * 64, i0 = rb * 16 * MB, kbeg = ks * SPW * 64;
    const int mrows = min(m - i0, 16 * MB);
    const int nsteps = min(SPW, (k - kbeg) / 64);  // >= 1 (grid)

    const char *bw = (const char *)B + ((int64_t)kbeg * ldb + j0) * 2;
    const int64_t b_ext = ((int64_t)(k - 1 - kbeg) * ldb + (n - j0)) * 2;
    const __amdgpu_buffer_rsrc_t Brs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)bw, 0, (int)min((b_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0), 0x00020000);
    const char *aw = (const char *)A + ((int64_t)i0 * lda + kbeg) * 2;
    const int64_t a_ext = ((int64_t)(mrows - 1) * lda + (k - kbeg)) * 2;
    const __amdgpu_buffer_rsrc_t Ars = __builtin_amdgcn_make_buffer_rsrc(
        (void *)aw, 0, (int)min((a_ext + 3) & ~(int64_t)3, (int64_t)0x7ffffff0), 0x00020000);

    // ---- every load, by DMA: A first, then B step by step --------------------
    // 1 KB blocks of 8 rows x 128 bytes; lane i writes row i / 8 of its block,
    // physical chunk i % 8, which holds logical chunk (i % 8) ^ (row & 7).
    // A: SPW * 2 MB blocks (step s, rows 8 h .. 8 h + 7), dealt to the waves.
    {
        const int rr = lane / 8;
#pragma unroll
        for (int b0 = 0; b0 < SPW * 2 * MB; b0 += 4) {
            const int b = b0 + wave;
            if (b < SPW * 2 * MB) {
                const int s = b / (2 * MB), h = b % (2 * MB);
                const int row = 8 * h + rr;
                const u32 off = (u32)row * (u32)lda * 2u + (u32)(128 * s) +
                                16u * (u32)((lane % 8) ^ (row & 7));
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    Ars, (lds_void *)(sA + s * AST + h * 1024), 16, (int)off, 0, 0, 0);
            }
        }
    }
    // B: wave w moves k rows 16 w .. 16 w + 15 of each step (two blocks).
    {
        auto dma_step = [&](auto sc) {
            constexpr int S = decltype(sc)::value;
            if constexpr (S < SPW) {
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const int rr = 16 * wave + 8 * e + lane / 8;
                    const u32 off = (u32)(64 * S + rr) * (u32)ldb * 2u +
                                    16u * (u32)((lane % 8) ^ (rr & 7));
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        Brs, (lds_void *)(sb(sc) + (2 * wave + e) * 1024), 16, (int)off, 0, 0,
                        0);
                }
            }
        };
        dma_step(ic<0>{}); dma_step(ic<1>{}); dma_step(ic<2>{}); dma_step(ic<3>{});
        dma_step(ic<4>{}); dma_step(ic<5>{}); dma_step(ic<6>{}); dma_step(ic<7>{});
    }

    // ---- multiply -------------------------------------------------------------
    // Lane (q, u) = (lane / 16, lane % 16): A row u of each 16-row block and B
    // column u of the wave's 16, k chunk q (16 elements) of the step.
    const int q = lane >> 4, u = lane & 15;
    int a_rd[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) a_rd[c] = u * 128 + 16 * ((2 * q + c) ^ (u & 7));
    // transpose reads: lane u of group q addresses k row 16 q + 4 r + u / 4 at
    // the 8-byte column group u % 4 of the wave's columns
    int b_rd[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int row = 16 * q + 4 * r + u / 4;
        const int byte = 32 * wave + 8 * (u % 4);
        b_rd[r] = row * 128 + 16 * ((byte / 16) ^ (row & 7)) + (byte % 16);
    }
    v4i acc_hh[MB], acc_x[MB], acc_ll[MB];
    int rsum[MB], csum = 0;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        acc_hh[mb] = v4i{0, 0, 0, 0};
        acc_x[mb] = v4i{0, 0, 0, 0};
        acc_ll[mb] = v4i{0, 0, 0, 0};
        rsum[mb] = 0;
    }
    // Step s: wait until this wave's A and B steps up to s have landed (two
    // DMAs per later step may stay in flight), then for the other waves'.
    auto mul_step = [&](auto sc) {
        constexpr int S = decltype(sc)::value;
        if constexpr (S < SPW) {
            constexpr int W = 2 * (SPW - 1 - S);
            __builtin_amdgcn_s_waitcnt((W & 0xf) | ((W >> 4) << 14) | (0x7 << 4) | (0xf << 8));
            __builtin_amdgcn_s_barrier();
            if (S < nsteps) {
                const char *bs = sb(sc);
                u32 wb[8];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const lds::v2i d = lds::tr16(bs + b_rd[r]);
                    wb[2 * r] = (u32)d.x;
                    wb[2 * r + 1] = (u32)d.y;
                }
                const v4i bh = v4(hi4(wb[1], wb[0]), hi4(wb[3], wb[2]), hi4(wb[5], wb[4]),
                                  hi4(wb[7], wb[6]));
                const v4i bl = v4(lo4(wb[1], wb[0]), lo4(wb[3], wb[2]), lo4(wb[5], wb[4]),
                                  lo4(wb[7], wb[6]));
#pragma unroll
                for (int x = 0; x < 8; ++x) csum = sum2(wb[x], csum);
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const char *as = sA + S * AST + mb * 2048;
                    const v4i a0 = *(const v4i *)(as + a_rd[0]);
                    const v4i a1 = *(const v4i *)(as + a_rd[1]);
                    const u32 wa[8] = {(u32)a0.x, (u32)a0.y, (u32)a0.z, (u32)a0.w,
                                       (u32)a1.x, (u32)a1.y, (u32)a1.z, (u32)a1.w};
                    const v4i ah = v4(hi4(wa[1], wa[0]), hi4(wa[3], wa[2]), hi4(wa[5], wa[4]),
                                      hi4(wa[7], wa[6]));
                    const v4i al = v4(lo4(wa[1], wa[0]), lo4(wa[3], wa[2]), lo4(wa[5], wa[4]),
                                      lo4(wa[7], wa[6]));
#pragma unroll
                    for (int x = 0; x < 8; ++x) rsum[mb] = sum2(wa[x], rsum[mb]);
                    acc_hh[mb] = Mfma<16>::mma(ah, bh, acc_hh[mb]);
                    acc_x[mb] = Mfma<16>::mma(ah, bl, acc_x[mb]);
                    acc_ll[mb] = Mfma<16>::mma(al, bl, acc_ll[mb]);
                    acc_x[mb] = Mfma<16>::mma(al, bh, acc_x[mb]);
                }
            }
        }
    };
    mul_step(ic<0>{}); mul_step(ic<1>{}); mul_step(ic<2>{}); mul_step(ic<3>{});
    mul_step(ic<4>{}); mul_step(ic<5>{}); mul_step(ic<6>{}); mul_step(ic<7>{});

    // ---- into C ---------------------------------------------------------------
    // Sums over the four k chunks (lanes u, u + 16, u + 32, u + 48).
    csum += __shfl_xor(csum, 16);
    csum += __shfl_xor(csum, 32);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        rsum[mb] += __shfl_xor(rsum[mb], 16);
        rsum[mb] += __shfl_xor(rsum[mb], 32);
    }
    const u32 kconst = 0u - 16384u * (u32)(64 * nsteps);
    const int col = j0 + 16 * wave + Mfma<16>::out_col(lane);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * mb + Mfma<16>::out_row(lane, r);
            // the row's sum sits in lane (row % 16)
            const int rs = __shfl(rsum[mb], Mfma<16>::out_row(lane, r));
            const u32 v = 65536u * (u32)acc_hh[mb][r] + 256u * (u32)acc_x[mb][r] +
                          (u32)acc_ll[mb][r] + 128u * ((u32)rs + (u32)csum) + kconst;
            if (col < n && row < mrows) {
                int32_t *dst = C + (int64_t)(i0 + row) * ldc + col;
                if constexpr (SPLIT)
                    atomicAdd(dst, (int)v);
                else
                    *dst = (int)((u32)*dst + v);
            }
        }
    }
}

template <int MB, int SPW>
const void *pick_lds16(bool split) {
    return split ? (const void *)igemm_stream_lds16<MB, SPW, true>
                 : (const void *)igemm_stream_lds16<MB, SPW, false>;
}

}  // namespace stream

int launch_stream(const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                  void *stream) {
    const int waves = p.threads / 64;
    const int spw = (int)(p.k_chunk / kBK);
    const bool va = p.vec_a != 0, vb = p.vec_b != 0, split = p.split > 1;
    const void *fn;
    if (p.kernel == K_I16_STREAM) {
        // int16: 64 columns per workgroup of four waves
        fn = p.bm == 16 ? (spw == 8 ? stream::pick_lds16<1, 8>(split)
                                    : spw == 4 ? stream::pick_lds16<1, 4>(split) : nullptr)
                        : (spw == 8 ? stream::pick_lds16<2, 8>(split)
                                    : spw == 4 ? stream::pick_lds16<2, 4>(split) : nullptr);
        if (fn == nullptr) return IGEMM_EINVAL;
        int mi = (int)m, ni = (int)n, ki = (int)k;
        int cbs = (int)((n + 63) / 64), rbs = (int)((m + p.bm - 1) / p.bm);
        void *args[] = {(void *)&A, (void *)&lda, (void *)&B, (void *)&ldb, (void *)&C,
                        (void *)&ldc, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&cbs,
                        (void *)&rbs};
        hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3(256), args, 0,
                                       (hipStream_t)stream);
        return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
    }
    if (va && vb && spw > 16) {
        // the column-per-wave kernel's ring variant (more than 16 steps)
        fn = p.bm == 16 ? stream::pick_ring<1>(split) : stream::pick_ring<2>(split);
        int mi = (int)m, ni = (int)n, ki = (int)k, si = spw;
        int cbs = (int)((n + 127) / 128), rbs = (int)((m + p.bm - 1) / p.bm);
        void *args[] = {(void *)&A, (void *)&lda, (void *)&B, (void *)&ldb, (void *)&C,
                        (void *)&ldc, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&cbs,
                        (void *)&rbs, (void *)&si};
        hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3(512), args, 0,
                                       (hipStream_t)stream);
        return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
    }
    if (va && vb) {
        // the column-per-wave kernel (operands of whole 16-byte rows)
        fn = p.bm == 16 ? stream::pick_lds_spw<1>(spw, split)
                        : stream::pick_lds_spw<2>(spw, split);
    } else {
        // the register kernel; 8-byte loads of B where its rows allow
        const bool vb8 = (uintptr_t)B % 8 == 0 && ldb % 8 == 0;
        const int s = spw / waves;
        fn = p.bm == 16 ? stream::pick<1>(waves, s, va, vb8, split)
                        : stream::pick<2>(waves, s, va, vb8, split);
    }
    if (fn == nullptr) return IGEMM_EINVAL;
    int mi = (int)m, ni = (int)n, ki = (int)k;
    int cbs = (int)((n + 127) / 128), rbs = (int)((m + p.bm - 1) / p.bm);
    void *args[] = {(void *)&A, (void *)&lda, (void *)&B, (void *)&ldb, (void *)&C,
                    (void *)&ldc, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&cbs,
                    (void *)&rbs};
    hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3((unsigned)p.threads), args, 0,
                                   (hipStream_t)stream);
    return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

}  // namespace igemm
