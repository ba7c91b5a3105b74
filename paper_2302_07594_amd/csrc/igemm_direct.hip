// Direct multiply for large GEMMs: no packing pass, no workspace.
//
// The packed path (igemm_packed.hip) first rewrites A and B into limb planes
// with k-contiguous rows, so that its multiply kernel only streams bytes.
// On gfx950 that rewrite is not needed: row-major A is already k-contiguous,
// and the LDS transpose reads (ds_read_b64_tr_b16 / _tr_b8) turn a row-major
// tile of B in LDS into k-contiguous matrix-core operands. So this kernel
//   * moves the caller's A and B tiles global -> LDS unchanged with the DMA
//     loads (global_load_lds_dwordx4), four stages ahead as the packed kernel;
//   * reads A fragments with ds_read_b128 and B fragments with transpose
//     reads, and for int16 splits every element into its high and offset-low
//     int8 limbs in registers (v_perm_b32, one xor) right before the MFMAs;
//   * accumulates the exact row sums of A and column sums of B from the raw
//     int16 fragments (v_dot2 with ones; each row and column by one wave), so
//     that the epilogue adds the limb corrections of its own k range;
//   * updates C modulo 2^32 with the branch-free buffer-resource epilogue.
// Exactness (Sec. 4.1 definition, int16 limb identity): for x = 256 h + l
// with h = x >> 8 and l = x & 255, write l' = l - 128 in [-128, 127]; then
//   sum_p x_p y_p = 65536 S_hh + 256 (S_hl' + S_l'h) + S_l'l'
//                   + 128 sum_p x_p + 128 sum_p y_p - 16384 k     (mod 2^32)
// with every int8 partial sum below 2^31 for k <= 32768 per launch.
//
// Preconditions (checked by the planner): A and B 16-byte aligned, rows of
// A and B a multiple of 16 bytes, k a multiple of 64 (no k tail), n a
// multiple of 8 (int16) or 16 (int8) columns, and the tile-offset bounds
// below; m and n need not be multiples of the tile.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm.h"
#include "igemm_device.h"
#include "igemm_internal.h"
#include "igemm_lds.h"

namespace igemm {
namespace direct {

using namespace lds;

// Swizzles of the raw tiles in LDS. A rows hold the 64 k of one row of A
// (128 bytes int16, 64 bytes int8), B rows the BN columns of one k (256
// bytes); 16-byte chunk c of row r sits at c ^ swz(r). They keep the
// fragment reads (16 or 32 rows at one chunk) and the transpose reads (4 or
// 8 k rows at 32 or 16 contiguous bytes, two groups side by side) spread
// over all 64 banks.
template <int ES>
__device__ __forceinline__ int swz_a(int row) {
    if constexpr (ES == 2) return (row >> 1) & 7;
    else return ((row >> 1) ^ (row >> 2)) & 3;
}
template <int ES>
__device__ __forceinline__ int swz_b(int row) {
    if constexpr (ES == 2) return 4 * (row & 3);
    else return 2 * (row & 7);
}

// C += A B on one BM x BN tile per workgroup over k range [0, 64 ktiles)
// of the given bases (the host offsets A and B to the launch's k chunk).
// ktiles is a multiple of four.
template <int ES, int BM, int BN, int WM, int WN, int NST>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64, 1)
igemm_direct(const char *__restrict__ A, int64_t lda, const char *__restrict__ B, int64_t ldb,
             int32_t *__restrict__ C, int64_t ldc, int m, int n, int ktiles, int tiles_m,
             int tiles_n) {
    constexpr int MF = 32;
    typedef Mfma<MF> M;
    typedef typename M::acc_t acc_t;
    constexpr int NACC = ES == 2 ? 3 : 1;
    constexpr int TM = WM / MF, TN = WN / MF;
    constexpr int WGN = BN / WN;
    constexpr int NW = (BM / WM) * WGN;
    static_assert(NW == 4 || NW == 8, "four or eight waves per workgroup");
    static_assert(NST == 4, "four LDS stages");
    constexpr int RA = 64 * ES;            // bytes of one A row per k-tile
    constexpr int RB = BN * ES;            // bytes of one B row (one k)
    static_assert(RB == 256, "B rows of 256 bytes");
    constexpr int APL = BM * RA, BPL = 64 * RB;
    constexpr int STAGE = APL + BPL;
    static_assert(NST * STAGE + 1024 <= 160 * 1024, "gfx950 LDS");
    constexpr int ROWS_A = 1024 / RA;      // A rows per 1 KB DMA block
    constexpr int NBA = APL / 1024, NBB = BPL / 1024;
    static_assert(NBA % NW == 0 && NBB % NW == 0, "DMA blocks per wave");
    constexpr int DPA = NBA / NW, DPB = NBB / NW, DPW = DPA + DPB;
    static_assert(DPW <= 15, "outstanding DMA count fits s_waitcnt");

    __shared__ __attribute__((aligned(16))) char st0[STAGE];
    __shared__ __attribute__((aligned(16))) char st1[STAGE];
    __shared__ __attribute__((aligned(16))) char st2[STAGE];
    __shared__ __attribute__((aligned(16))) char st3[STAGE];
    __shared__ u32 sums[ES == 2 ? BM + BN : 1];
    auto stage = [&](auto s) -> char * {
        constexpr int S = decltype(s)::value;
        if constexpr (S == 0) return st0;
        else if constexpr (S == 1) return st1;
        else if constexpr (S == 2) return st2;
        else return st3;
    };

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;

    int bid = blockIdx.x;
    const int G = gridDim.x;
    if ((G & 7) == 0) bid = (bid & 7) * (G >> 3) + (bid >> 3);
    constexpr int GROUP = 8;
    const int span = GROUP * tiles_n;
    const int first_m = (bid / span) * GROUP;
    const int gsize = min(tiles_m - first_m, GROUP);
    const int tm = first_m + (bid % span) % gsize;
    const int tn = (bid % span) / gsize;
    const int m0 = tm * BM, n0 = tn * BN;

    // DMA: lane i of a 1 KB block writes LDS bytes [16 i, 16 i + 16): for A
    // row rb + i / (RA / 16), physical chunk i % (RA / 16); for B row
    // 4 b + i / 16, physical chunk i % 16. The lane fetches the logical chunk
    // that the swizzle puts there. Rows of A beyond m read row m - 1 and
    // column chunks of B beyond n read the last chunk (their products only
    // reach elements of C that are never stored). Offsets are 32-bit byte
    // offsets from the operand bases (the planner keeps them below 2^31); the
    // k-tile's position is added as a wave-uniform 64-bit base.
    u32 off[DPW];
    int ldsoff[DPW];
#pragma unroll
    for (int d = 0; d < DPW; ++d) {
        if (d < DPA) {
            const int b = wave * DPA + d;
            const int row = b * ROWS_A + lane / (RA / 16);
            const int pc = lane % (RA / 16);
            const int lc = pc ^ swz_a<ES>(row);
            const int grow = min(m0 + row, m - 1);
            off[d] = (u32)grow * (u32)(lda * ES) + 16u * (u32)lc;
            ldsoff[d] = b * 1024;
        } else {
            const int b = wave * DPB + (d - DPA);
            const int row = 4 * b + (lane >> 4);
            const int lc = (lane & 15) ^ swz_b<ES>(row);
            const int col = min(n0 + lc * (16 / ES), n - 16 / ES);
            off[d] = (u32)row * (u32)(ldb * ES) + (u32)(col * ES);
            ldsoff[d] = APL + b * 1024;
        }
    }
    const int64_t a_step = 64 * ES, b_step = 64 * ldb * ES;
    auto dma_range = [&](auto s, int kt, auto d0, auto d1) {
        constexpr int D0 = decltype(d0)::value, D1 = decltype(d1)::value;
        char *dst = stage(s);
        // The k-tile bases are made opaque scalars, so that the optimiser
        // cannot re-associate base + lane offset into 64-bit vector adds: the
        // loads then take a scalar base and a 32-bit lane offset.
        const char *ak = A + (int64_t)kt * a_step;
        const char *bk = B + (int64_t)kt * b_step;
        asm volatile("" : "+s"(ak), "+s"(bk));
#pragma unroll
        for (int d = D0; d < D1; ++d) {
            u32 o = off[d];
            asm volatile("" : "+v"(o));
            dma16((d < DPA ? ak : bk) + o, (lds_void *)(dst + ldsoff[d]));
        }
    };

    // Fragment addresses. A: lane row fr = lane % 32 of each 32-row block,
    // k chunk q = 2 ks + lane / 32 of 16 elements (32 bytes int16: two
    // ds_read_b128; 16 bytes int8: one). B: transpose reads, group g =
    // lane / 16 covers columns 16 (g % 2) + [0, 16) of a 32-column block
    // and k chunk q = 2 ks + g / 2; lane u = lane % 16 addresses k row
    // 16 q + (4 r + u / 4) (int16, reads r < 4) or (8 r + u / 2) (int8,
    // r < 2) at columns 4 (u % 4) (int16) or 8 (u % 2) (int8) of the group.
    const int fr = lane & 31, g = lane >> 4, u = lane & 15;
    int a_rd[2][2], b_rd[2][TN];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int q = 2 * ks + (lane >> 5);
        const int row = wm0 + fr;   // swz_a depends on row mod 16 only
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int lc = ES == 2 ? 2 * q + h : q;
            a_rd[ks][h] = row * RA + 16 * (lc ^ swz_a<ES>(row));
        }
        const int qb = 2 * ks + (g >> 1);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wn0 + 32 * j + 16 * (g & 1) + (ES == 2 ? 4 * (u & 3) : 8 * (u & 1));
            const int krow = 16 * qb + (ES == 2 ? (u >> 2) : (u >> 1));
            const int lc = col * ES / 16, inner = (col * ES) % 16;
            b_rd[ks][j] = APL + krow * RB + 16 * (lc ^ swz_b<ES>(krow)) + inner;
        }
    }
    // Raw fragments: int16 A: TM x 8 dwords, B: TN x 8 dwords (four tr16
    // reads); int8 A: TM x 4, B: TN x 4 (two tr8 reads). int8 keeps two
    // slots of raw fragments, which are its MFMA operands; int16 keeps one
    // slot of raw fragments and two slots of split operands (see below).
    constexpr int RW = ES == 2 ? 8 : 4;
    constexpr int RS = ES == 2 ? 1 : 2;
    u32 ra[RS][TM][RW], rb[RS][TN][RW];
    auto read_frags = [&](auto slot, auto s, auto ks) {
        constexpr int SL = decltype(slot)::value;
        constexpr int KS = decltype(ks)::value;
        const char *base = stage(s);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
            for (int r = 0; r < RW / 2; ++r) {
                const v2i x = ES == 2 ? tr16(base + b_rd[KS][j] + r * 4 * RB)
                                      : tr8(base + b_rd[KS][j] + r * 8 * RB);
                rb[SL][j][2 * r] = (u32)x.x;
                rb[SL][j][2 * r + 1] = (u32)x.y;
            }
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int h = 0; h < (ES == 2 ? 2 : 1); ++h) {
                const v4i x = *(const v4i *)(base + a_rd[KS][h] + i * MF * RA);
                ra[SL][i][4 * h] = (u32)x.x;
                ra[SL][i][4 * h + 1] = (u32)x.y;
                ra[SL][i][4 * h + 2] = (u32)x.z;
                ra[SL][i][4 * h + 3] = (u32)x.w;
            }
        }
    };

    acc_t acc[NACC][TM][TN];
#pragma unroll
    for (int a = 0; a < NACC; ++a)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < M::REGS; ++r) acc[a][i][j][r] = 0;
    // Exact sums of this wave's share: rows (waves 0 and 3) or columns
    // (waves 1 and 2) of its tile, int16 only.
    constexpr int NPS = ES == 2 ? (TM > TN ? TM : TN) : 1;
    int psum[NPS];
#pragma unroll
    for (int i = 0; i < NPS; ++i) psum[i] = 0;

    // int16 operands of one sub-step: high and offset-low limbs of the TM A
    // and TN B fragments, split from the raw slot one sub-step ahead.
    v4i ah[2][TM], al[2][TM], bh[2][TN], bl[2][TN];
    auto split = [&](auto slot, auto sums_kind) {
        constexpr int SL = decltype(slot)::value;
        constexpr int SK = decltype(sums_kind)::value;
        if constexpr (ES == 2) {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const u32 *w = ra[0][i];
                ah[SL][i] = v4(hi4(w[1], w[0]), hi4(w[3], w[2]), hi4(w[5], w[4]), hi4(w[7], w[6]));
                al[SL][i] = v4(lo4(w[1], w[0]), lo4(w[3], w[2]), lo4(w[5], w[4]), lo4(w[7], w[6]));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const u32 *w = rb[0][j];
                bh[SL][j] = v4(hi4(w[1], w[0]), hi4(w[3], w[2]), hi4(w[5], w[4]), hi4(w[7], w[6]));
                bl[SL][j] = v4(lo4(w[1], w[0]), lo4(w[3], w[2]), lo4(w[5], w[4]), lo4(w[7], w[6]));
            }
            if constexpr (SK == 1) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int x = 0; x < 8; ++x) psum[i] = sum2(ra[0][i][x], psum[i]);
            } else if constexpr (SK == 2) {
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int x = 0; x < 8; ++x) psum[j] = sum2(rb[0][j][x], psum[j]);
            }
        }
    };
    auto mfmas = [&](auto slot) {
        constexpr int SL = decltype(slot)::value;
        if constexpr (ES == 1) {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const v4i a = v4(ra[SL][i][0], ra[SL][i][1], ra[SL][i][2], ra[SL][i][3]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] = M::mma(a, v4(rb[SL][j][0], rb[SL][j][1], rb[SL][j][2],
                                                rb[SL][j][3]), acc[0][i][j]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[0][i][j] = M::mma(ah[SL][i], bh[SL][j], acc[0][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[1][i][j] = M::mma(ah[SL][i], bl[SL][j], acc[1][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[2][i][j] = M::mma(al[SL][i], bl[SL][j], acc[2][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[1][i][j] = M::mma(al[SL][i], bh[SL][j], acc[1][i][j]);
            }
        }
    };

    constexpr int WAIT_NEWEST = (DPW & 0xf) | (0x7 << 4) | (0xf << 8);
    constexpr int WAIT_ALL = (0x7 << 4) | (0xf << 8);
    constexpr int NM = TM * TN * (ES == 2 ? 4 : 1);
    constexpr int NR = TN * (RW / 2) + TM * (ES == 2 ? 2 : 1);
    constexpr int D_SUB0 = DPW / 2;
    // VALU instructions of one split: 8 v_perm_b32 and 4 xors per fragment,
    // plus 8 v_dot2 for the sums of two fragments.
    constexpr int NV = ES == 2 ? 12 * (TM + TN) + 16 : 0;
    // MFMA slots that carry the split, and LDS reads per slot after them
    // (a sweep of 8, 10, 11 and 12 split slots with 2-4 reads per slot put
    // all within 2 % of each other on int16 4096^3; this one was fastest).
    constexpr int VSLOTS = 12;
    constexpr int VPS = VSLOTS > 0 ? (NV + VSLOTS - 1) / VSLOTS : 0;
    constexpr int RPS = 4;

    // One sub-step's MFMAs with, between them, the DMA share `dma`, the
    // split of the raw slot into operand slot NXT (int16, if SPLIT) in the
    // first half of the slots, then the LDS reads of the raw slot for a later
    // sub-step (if READ) in the second half.
    auto sub16 = [&](auto cur, auto nxt, auto split_flag, auto read_flag, auto sums_kind,
                     auto rd_stage, auto rd_ks, auto dma) {
        constexpr int CUR = decltype(cur)::value, NXT = decltype(nxt)::value;
        constexpr bool SPLIT = decltype(split_flag)::value != 0;
        constexpr bool READ = decltype(read_flag)::value != 0;
        constexpr int ND = decltype(dma)::value;
        mfmas(ic<CUR>{});
        if constexpr (SPLIT) split(ic<NXT>{}, sums_kind);
        if constexpr (READ) read_frags(ic<0>{}, rd_stage, rd_ks);
        // Slot layout: the split runs in slots [1, 1 + VSLOTS) (slot 0 leaves
        // the previous sub-step's reads time to land), the reads, which
        // overwrite the raw slot the split consumes, in the slots after it,
        // RPS per slot.
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (SPLIT && i >= 1 && i < 1 + VSLOTS)
                __builtin_amdgcn_sched_group_barrier(0x002, VPS, 0);
            if (READ && i >= 1 + VSLOTS && i < 1 + VSLOTS + (NR + RPS - 1) / RPS)
                __builtin_amdgcn_sched_group_barrier(0x100, RPS, 0);
            if (ND > 0 && (i * ND) / NM != ((i + 1) * ND) / NM)
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    // The k loop. Step kt computes tile kt from stage kt % 4 while the DMA
    // of tile kt + 3 runs.
    //   int16: the raw slot holds sub-step (kt, 1) and operand slot 0 the split
    //   (kt, 0) on entry; sub-step 0 multiplies slot 0, splits the raw slot
    //   into slot 1 and reads (kt + 1, 0); sub-step 1 multiplies slot 1,
    //   splits into slot 0 and reads (kt + 1, 1). Reads run one tile ahead.
    //   int8: read the next sub-step's fragments under the MFMAs of this one.
    auto run = [&](auto sums_kind) {
        auto step = [&](auto s, int kt, auto do_dma, auto do_pref) {
            constexpr int S = decltype(s)::value;
            constexpr int SD = (S + NST - 1) % NST;
            constexpr bool DMA = decltype(do_dma)::value != 0;
            constexpr bool PREF = decltype(do_pref)::value != 0;
            if constexpr (ES == 2) {
                if constexpr (DMA) dma_range(ic<SD>{}, kt + NST - 1, ic<0>{}, ic<D_SUB0>{});
                sub16(ic<0>{}, ic<1>{}, ic<1>{}, ic<PREF>{}, sums_kind, ic<(S + 1) % NST>{},
                      ic<0>{}, ic<DMA ? D_SUB0 : 0>{});
                if constexpr (DMA) dma_range(ic<SD>{}, kt + NST - 1, ic<D_SUB0>{}, ic<DPW>{});
                sub16(ic<1>{}, ic<0>{}, ic<PREF>{}, ic<PREF>{}, sums_kind, ic<(S + 1) % NST>{},
                      ic<1>{}, ic<DMA ? DPW - D_SUB0 : 0>{});
            } else {
                if constexpr (DMA) dma_range(ic<SD>{}, kt + NST - 1, ic<0>{}, ic<D_SUB0>{});
                read_frags(ic<1>{}, ic<S>{}, ic<1>{});
                mfmas(ic<0>{});
#pragma unroll
                for (int i = 0; i < NM; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    if (i < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    if (DMA && (i * D_SUB0) / NM != ((i + 1) * D_SUB0) / NM)
                        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (DMA) dma_range(ic<SD>{}, kt + NST - 1, ic<D_SUB0>{}, ic<DPW>{});
                if constexpr (PREF) read_frags(ic<0>{}, ic<(S + 1) % NST>{}, ic<0>{});
                mfmas(ic<1>{});
#pragma unroll
                for (int i = 0; i < NM; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    if (PREF && i < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    if (DMA && (i * (DPW - D_SUB0)) / NM != ((i + 1) * (DPW - D_SUB0)) / NM)
                        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (PREF) {
                __builtin_amdgcn_s_waitcnt(DMA ? WAIT_NEWEST : WAIT_ALL);
                __builtin_amdgcn_s_barrier();
            }
        };
        auto tail_step = [&](auto jc, auto tc, int kt0) {
            constexpr int J = decltype(jc)::value, T = decltype(tc)::value;
            if constexpr (J < T)
                step(ic<J % NST>{}, kt0 + J, ic<(J + NST - 1 < T)>{}, ic<(J + 1 < T)>{});
        };
        dma_range(ic<0>{}, 0, ic<0>{}, ic<DPW>{});
        dma_range(ic<1>{}, 1, ic<0>{}, ic<DPW>{});
        dma_range(ic<2>{}, 2, ic<0>{}, ic<DPW>{});
        __builtin_amdgcn_s_waitcnt(WAIT_NEWEST);
        __builtin_amdgcn_s_barrier();
        read_frags(ic<0>{}, ic<0>{}, ic<0>{});
        if constexpr (ES == 2) {
            split(ic<0>{}, sums_kind);
            read_frags(ic<0>{}, ic<0>{}, ic<1>{});
        }
        int kt = 0;
        for (; kt <= ktiles - 2 * NST + 1; kt += NST) {
            step(ic<0>{}, kt, ic<1>{}, ic<1>{});
            step(ic<1>{}, kt + 1, ic<1>{}, ic<1>{});
            step(ic<2>{}, kt + 2, ic<1>{}, ic<1>{});
            step(ic<3>{}, kt + 3, ic<1>{}, ic<1>{});
        }
        // The last four tiles (ktiles is a multiple of four).
        tail_step(ic<0>{}, ic<4>{}, kt);
        tail_step(ic<1>{}, ic<4>{}, kt);
        tail_step(ic<2>{}, ic<4>{}, kt);
        tail_step(ic<3>{}, ic<4>{}, kt);
    };
    // Which sums this wave takes (uniform per wave, so each runs its own copy
    // of the loop with the same barriers): four waves (2 x 2 grid of 64 x 64)
    // -- waves 0 and 3 the row sums of their 64 rows, waves 1 and 2 the column
    // sums of their 64 columns; eight waves (2 x 4 grid of 64 x 32) -- waves 0
    // and 5 the rows, waves 1 to 4 the columns (every row and column once).
    const int skind = NW == 4 ? (wave == 0 || wave == 3 ? 1 : 2)
                              : (wave == 0 || wave == 5 ? 1 : (wave <= 4 ? 2 : 0));
    if constexpr (ES == 2) {
        if (skind == 1) run(ic<1>{});
        else if (skind == 2) run(ic<2>{});
        else run(ic<0>{});
    } else {
        run(ic<0>{});
    }

    // ---- epilogue -----------------------------------------------------------
    u32 colt[TN], rowt[TM][M::REGS];
#pragma unroll
    for (int j = 0; j < TN; ++j) colt[j] = 0;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < M::REGS; ++r) rowt[i][r] = 0;
    if constexpr (ES == 2) {
        // Lanes l and l + 32 hold complementary k chunks of the same row or
        // column: add them, scale by 128 and publish through LDS.
        const bool rows = skind == 1;
#pragma unroll
        for (int i = 0; i < (TM > TN ? TM : TN); ++i) {
            const u32 s = 128u * (u32)(psum[i] + __shfl_xor(psum[i], 32));
            if (lane < 32 && skind != 0 && i < (rows ? TM : TN))
                sums[rows ? wm0 + 32 * i + lane : BM + wn0 + 32 * i + lane] = s;
        }
        __syncthreads();
        const u32 kconst = 0u - 16384u * (u32)(64 * ktiles);
#pragma unroll
        for (int j = 0; j < TN; ++j) colt[j] = kconst + sums[BM + wn0 + MF * j + M::out_col(lane)];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < M::REGS; ++r)
                rowt[i][r] = sums[wm0 + MF * i + M::out_row(lane, r)];
    }
    const __amdgpu_buffer_rsrc_t Crs = __builtin_amdgcn_make_buffer_rsrc(
        (char *)C + ((int64_t)m0 * ldc + n0) * 4, 0, 0x7fffffff, 0x00020000);
    const int ldc32 = (int)ldc;
    auto c_off = [&](int lr, int lc) -> u32 {
        return (m0 + lr < m && n0 + lc < n) ? (u32)(lr * ldc32 + lc) * 4u : 0x80000000u;
    };
    constexpr int NOUT = TM * TN;
    constexpr int NB = NW == 8 ? 1 : (NOUT <= 4 ? NOUT : 2);
    constexpr int NBATCH = NOUT / NB;
    static_assert(NOUT % NB == 0 && NBATCH <= 8, "epilogue batches");
    int32_t cv[2][NB][M::REGS];
    auto load_batch = [&](auto buf, auto batch) {
        constexpr int BF = decltype(buf)::value, B0 = decltype(batch)::value * NB;
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) {
            const int i = (B0 + bb) / TN, j = (B0 + bb) % TN;
            const int lc = wn0 + MF * j + M::out_col(lane);
#pragma unroll
            for (int r = 0; r < M::REGS; ++r) {
                const int lr = wm0 + MF * i + M::out_row(lane, r);
                cv[BF][bb][r] = __builtin_amdgcn_raw_buffer_load_b32(Crs, c_off(lr, lc), 0, 0);
            }
        }
    };
    auto finish_batch = [&](auto buf, auto batch) {
        constexpr int BF = decltype(buf)::value, B0 = decltype(batch)::value * NB;
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) {
            const int i = (B0 + bb) / TN, j = (B0 + bb) % TN;
            const int lc = wn0 + MF * j + M::out_col(lane);
#pragma unroll
            for (int r = 0; r < M::REGS; ++r) {
                const int lr = wm0 + MF * i + M::out_row(lane, r);
                u32 v;
                if constexpr (ES == 1) {
                    v = (u32)acc[0][i][j][r];
                } else {
                    v = 65536u * (u32)acc[0][i][j][r] + 256u * (u32)acc[1][i][j][r] +
                        (u32)acc[2][i][j][r] + colt[j] + rowt[i][r];
                }
                __builtin_amdgcn_raw_buffer_store_b32((int)((u32)cv[BF][bb][r] + v), Crs,
                                                      c_off(lr, lc), 0, 0);
            }
        }
    };
    load_batch(ic<0>{}, ic<0>{});
    auto epi_step = [&](auto batch) {
        constexpr int BT = decltype(batch)::value;
        if constexpr (BT + 1 < NBATCH) load_batch(ic<(BT + 1) & 1>{}, ic<BT + 1>{});
        finish_batch(ic<BT & 1>{}, ic<BT>{});
        __builtin_amdgcn_sched_barrier(0);
    };
    epi_step(ic<0>{});
    if constexpr (NBATCH > 1) epi_step(ic<1>{});
    if constexpr (NBATCH > 2) epi_step(ic<2>{});
    if constexpr (NBATCH > 3) epi_step(ic<3>{});
    if constexpr (NBATCH > 4) epi_step(ic<4>{});
    if constexpr (NBATCH > 5) epi_step(ic<5>{});
    if constexpr (NBATCH > 6) epi_step(ic<6>{});
    if constexpr (NBATCH > 7) epi_step(ic<7>{});
}

}  // namespace direct

using namespace direct;

// One launch per k chunk of at most kMaxKChunk elements (a multiple of 256);
// each adds its own exact contribution, corrections included.
int launch_direct(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, const void *B, int64_t ldb, int32_t *C, int64_t ldc,
                  void *stream_) {
    hipStream_t stream = (hipStream_t)stream_;
    const KernelDesc &d = kKernels[p.kernel];
    const int tm = (int)((m + d.bm - 1) / d.bm), tn = (int)((n + d.bn - 1) / d.bn);
    const dim3 grid((unsigned)p.grid);
    const int mi = (int)m, ni = (int)n;
    for (int64_t k0 = 0; k0 < k; k0 += p.k_chunk) {
        const int64_t kc = k - k0 < p.k_chunk ? k - k0 : p.k_chunk;
        const int ktiles = (int)(kc / 64);
        const char *Ak = (const char *)A + k0 * es;
        const char *Bk = (const char *)B + k0 * ldb * es;
        if (ktiles % 4 != 0 || ktiles < 4) return IGEMM_EINVAL;   // the planner prevents it
        // int16 with at most eight k-tiles per launch: eight waves of 64 x 32
        // (one wave's limb split beside the other's matrix-core work; 4096 x
        // 4096 x 256 in 55.3 us against 58.7 us), else four waves of 64 x 64
        // (k = 4096: 276.6 us against 302.2 us with eight waves).
        if (es == 2 && ktiles <= 8)
            igemm_direct<2, 128, 128, 64, 32, 4><<<grid, 512, 0, stream>>>(
                Ak, lda, Bk, ldb, C, ldc, mi, ni, ktiles, tm, tn);
        else if (es == 2)
            igemm_direct<2, 128, 128, 64, 64, 4><<<grid, 256, 0, stream>>>(
                Ak, lda, Bk, ldb, C, ldc, mi, ni, ktiles, tm, tn);
        else
            igemm_direct<1, 256, 256, 64, 128, 4><<<grid, 512, 0, stream>>>(
                Ak, lda, Bk, ldb, C, ldc, mi, ni, ktiles, tm, tn);
        if (hipGetLastError() != hipSuccess) return IGEMM_EHIP;
    }
    return IGEMM_OK;
}

}  // namespace igemm
