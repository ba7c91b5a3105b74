// Pack-then-multiply path for large GEMMs.
//
// The paper's GEMM packs panels of A and B into buffers whose layout lets the
// micro-kernel stream them with unit stride (Sec. 4.1, the packing routines
// around the micro-kernel; Sec. 5.1 pre-packs A_c once for DL inference). On
// the GPU this is done for the whole operands, once per call, by two small
// memory-bound kernels:
//   * pack A: int16 rows are split into a high and an offset-low int8 limb
//     plane (k-contiguous, zero-padded to m_pad x k_pad) and the row limb sums
//     are reduced into one 32-bit correction per row; int8 A is only copied
//     when its rows are not 16-byte aligned or not tile multiples;
//   * pack B: B is transposed to k-contiguous columns (and split into limb
//     planes for int16), zero-padded to n_pad x k_pad, with per-column limb
//     sums reduced per k slice.
// The main kernel then reads both operands with global-to-LDS DMA loads
// (global_load_lds_dwordx4: no VGPRs, no staging instructions) into a
// four-stage LDS ring, three k-tiles ahead of the matrix cores, and runs the
// same MFMA micro-tiles as the fused kernels. All padding is zero, so the
// main loop has no bounds checks and every partial limb product of padding is
// zero; only the C update is bounded.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm.h"
#include "igemm_device.h"
#include "igemm_internal.h"

namespace igemm {
namespace packed {

typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from global memory straight into LDS: lane i writes
// [lds + 16 i, lds + 16 i + 16) (global_load_lds_dwordx4; lds must be wave
// uniform). Kept out of the kernel templates: the builtin exists only for
// the device, and inside a template it would suppress the host launch stub.
__device__ __forceinline__ void dma16(const void *g, lds_void *lds) {
    __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// ---- clear n 32-bit words (a fill kernel: graph captures record no memset) --
__global__ void __launch_bounds__(256) clear_u32(uint32_t *__restrict__ p, int n) {
    for (int j = blockIdx.x * 256 + threadIdx.x; j < n; j += gridDim.x * 256) p[j] = 0u;
}

// ---- pack A, int16: one workgroup per padded row ---------------------------
// Writes Ah/Al[i][0, k_pad) and corrA[i] = 32768*sum(h) + 128*sum(l) mod 2^32,
// and, if corrB is given, zeroes corrB[0, n_pad).
// For the int16-output update (bsA given): also the exact per-block limb
// sums of the row, block b = [b bspan, (b + 1) bspan) of the planes (bspan a
// multiple of 256, at most 64 blocks), at bsA[2 (b m_pad + i)] (high limbs)
// and + 1 (offset low limbs), m_pad = gridDim.x; and zeroes clr[0, nclr)
// (B's block sums, which pack_b adds into).
template <bool VEC>
__global__ void __launch_bounds__(256)
pack_a_i16(const int16_t *__restrict__ A, int64_t lda, int m, int k, int k_pad,
           int8_t *__restrict__ Ah, int8_t *__restrict__ Al, uint32_t *__restrict__ corrA,
           uint32_t *__restrict__ corrB, int n_pad, uint32_t *__restrict__ bsA, int bspan,
           int nblocks, uint32_t *__restrict__ clr, int nclr) {
    const int i = blockIdx.x, tid = threadIdx.x;
    // Clear the column corrections that pack_b (next on the stream) adds into.
    if (corrB != nullptr)
        for (int j = i * 256 + tid; j < n_pad; j += gridDim.x * 256) corrB[j] = 0u;
    if (clr != nullptr)
        for (int j = i * 256 + tid; j < nclr; j += gridDim.x * 256) clr[j] = 0u;
    __shared__ int bsum[64][2];
    if (bsA != nullptr) {
        if (tid < 128) (&bsum[0][0])[tid] = 0;
        __syncthreads();
    }
    const int len = i < m ? k : 0;
    const int16_t *arow = A + (int64_t)(i < m ? i : 0) * lda;
    int8_t *hrow = Ah + (int64_t)i * k_pad;
    int8_t *lrow = Al + (int64_t)i * k_pad;
    int sh = 0, sl = 0;
    for (int e0 = tid * 8; e0 < k_pad; e0 += 256 * 8) {
        const v4i raw = load16<2, VEC>(arow, e0, len);
        const u32 y0 = raw.x, y1 = raw.y, y2 = raw.z, y3 = raw.w;
        const int v = len - e0;
        const u32 m0 = byte_mask(v), m1 = byte_mask(v - 4);
        const u32 h0 = perm(y1, y0, 0x07050301u) & m0, h1 = perm(y3, y2, 0x07050301u) & m1;
        const u32 l0 = (perm(y1, y0, 0x06040200u) ^ 0x80808080u) & m0;
        const u32 l1 = (perm(y3, y2, 0x06040200u) ^ 0x80808080u) & m1;
        sh = sum4(h1, sum4(h0, sh));
        sl = sum4(l1, sum4(l0, sl));
        if (bsA != nullptr) {
            // the 32 lanes of a half-wave cover 256 elements of one block:
            // their sums, then one LDS add per half-wave
            int bh = sum4(h1, sum4(h0, 0)), bl = sum4(l1, sum4(l0, 0));
#pragma unroll
            for (int o = 16; o > 0; o >>= 1) {
                bh += __shfl_xor(bh, o);
                bl += __shfl_xor(bl, o);
            }
            if ((tid & 31) == 0) {
                atomicAdd(&bsum[e0 / bspan][0], bh);
                atomicAdd(&bsum[e0 / bspan][1], bl);
            }
        }
        *(uint2 *)(hrow + e0) = make_uint2(h0, h1);
        *(uint2 *)(lrow + e0) = make_uint2(l0, l1);
    }
    if (bsA != nullptr) {
        __syncthreads();
        for (int b = tid; b < nblocks; b += 256) {
            bsA[((int64_t)b * gridDim.x + i) * 2] = (u32)bsum[b][0];
            bsA[((int64_t)b * gridDim.x + i) * 2 + 1] = (u32)bsum[b][1];
        }
    }
    __shared__ int red[2][4];
    sh = wave_sum(sh);
    sl = wave_sum(sl);
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = sh;
        red[1][tid >> 6] = sl;
    }
    __syncthreads();
    if (tid == 0) {
        const u32 h = (u32)red[0][0] + (u32)red[0][1] + (u32)red[0][2] + (u32)red[0][3];
        const u32 l = (u32)red[1][0] + (u32)red[1][1] + (u32)red[1][2] + (u32)red[1][3];
        corrA[i] = 32768u * h + 128u * l;
    }
}

// ---- pack A, int16, short rows (k_pad <= 512): one wave per padded row -----
// The same outputs as pack_a_i16 (four rows per workgroup, so that no wave
// idles when a row is shorter than a workgroup's 2048 elements): lane t
// takes elements [8 t, 8 t + 8); the row's sums are wave sums; with blocks of
// 256 each half-wave's sums are one block's.
template <bool VEC>
__global__ void __launch_bounds__(256)
pack_a_i16_rows(const int16_t *__restrict__ A, int64_t lda, int m, int k, int k_pad,
                int8_t *__restrict__ Ah, int8_t *__restrict__ Al, uint32_t *__restrict__ corrA,
                uint32_t *__restrict__ corrB, int n_pad, uint32_t *__restrict__ bsA, int bspan,
                int m_pad, uint32_t *__restrict__ clr, int nclr) {
    const int tid = threadIdx.x, lane = tid & 63;
    if (corrB != nullptr)
        for (int j = blockIdx.x * 256 + tid; j < n_pad; j += gridDim.x * 256) corrB[j] = 0u;
    if (clr != nullptr)
        for (int j = blockIdx.x * 256 + tid; j < nclr; j += gridDim.x * 256) clr[j] = 0u;
    const int i = blockIdx.x * 4 + (tid >> 6);
    const int len = i < m ? k : 0;
    const int16_t *arow = A + (int64_t)(i < m ? i : 0) * lda;
    const int e0 = lane * 8;
    u32 h0 = 0, h1 = 0, l0 = 0, l1 = 0;
    if (e0 < k_pad) {
        const v4i raw = load16<2, VEC>(arow, e0, len);
        const u32 y0 = raw.x, y1 = raw.y, y2 = raw.z, y3 = raw.w;
        const int v = len - e0;
        const u32 m0 = byte_mask(v), m1 = byte_mask(v - 4);
        h0 = perm(y1, y0, 0x07050301u) & m0;
        h1 = perm(y3, y2, 0x07050301u) & m1;
        l0 = (perm(y1, y0, 0x06040200u) ^ 0x80808080u) & m0;
        l1 = (perm(y3, y2, 0x06040200u) ^ 0x80808080u) & m1;
        *(uint2 *)(Ah + (int64_t)i * k_pad + e0) = make_uint2(h0, h1);
        *(uint2 *)(Al + (int64_t)i * k_pad + e0) = make_uint2(l0, l1);
    }
    // half-wave sums (32 lanes, 256 elements), then the row's
    int sh = sum4(h1, sum4(h0, 0)), sl = sum4(l1, sum4(l0, 0));
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
        sh += __shfl_xor(sh, o);
        sl += __shfl_xor(sl, o);
    }
    const int th = sh + __shfl_xor(sh, 32), tl = sl + __shfl_xor(sl, 32);
    if (bsA != nullptr) {
        if (bspan >= 512) {
            // the whole row is block 0
            if (lane == 0) {
                bsA[(int64_t)i * 2] = (u32)th;
                bsA[(int64_t)i * 2 + 1] = (u32)tl;
            }
        } else if ((lane & 31) == 0 && e0 < k_pad) {
            // bspan = 256: one block per half-wave
            const int b = e0 / 256;
            bsA[((int64_t)b * m_pad + i) * 2] = (u32)sh;
            bsA[((int64_t)b * m_pad + i) * 2 + 1] = (u32)sl;
        }
    }
    if (lane == 0) corrA[i] = 32768u * (u32)th + 128u * (u32)tl;
}

// ---- pack A, int8: copy into a zero-padded m_pad x k_pad buffer ------------
template <bool VEC>
__global__ void __launch_bounds__(256)
pack_a_i8(const int8_t *__restrict__ A, int64_t lda, int m, int k, int k_pad,
          int8_t *__restrict__ Ap) {
    const int i = blockIdx.x, tid = threadIdx.x;
    const int len = i < m ? k : 0;
    const int8_t *arow = A + (int64_t)(i < m ? i : 0) * lda;
    int8_t *prow = Ap + (int64_t)i * k_pad;
    for (int e0 = tid * 16; e0 < k_pad; e0 += 256 * 16)
        *(v4i *)(prow + e0) = load16<1, VEC>(arow, e0, len);
}

// ---- pack B: transpose to k-contiguous columns ----------------------------
// Workgroup (blockIdx.x, blockIdx.y) covers columns [64x, 64x + 64) and the
// k slice [kspan*y, kspan*(y+1)). Per pass, thread (rg, cc) loads 4 rows x 16
// bytes, transposes 4x4 byte blocks in registers (and for int16 separates the
// limb planes), parks the per-column dwords in LDS, and the workgroup writes
// each column's k run out contiguously. For int16 the per-column limb sums of
// the slice are added into corrB[col] (zeroed by pack_a_i16, which runs first),
// and, for the int16-output update (bsB given), the exact per-block limb sums
// of the slice into bsB[2 (b n_pad + col)] and + 1 (zeroed by pack_a_i16;
// blocks of bspan rows, a multiple of 128, so that each pass of 128 rows lies
// in one block).
template <int ES, bool VEC>
__global__ void __launch_bounds__(256)
pack_b(const void *__restrict__ Bv, int64_t ldb, int k, int n, int k_pad, int kspan, int n_pad,
       int8_t *__restrict__ Bp0, int8_t *__restrict__ Bp1, uint32_t *__restrict__ corrB,
       uint32_t *__restrict__ bsB = nullptr, int bspan = 0) {
    constexpr int P = ES;                 // output planes
    constexpr int CC = ES == 2 ? 8 : 4;   // 16-byte column chunks per workgroup (64 columns)
    constexpr int RG = 256 / CC;          // row groups of 4 rows
    constexpr int ROWS = 4 * RG;          // k rows per pass
    constexpr int DW = ROWS / 4;          // dwords per column per pass
    constexpr int CPU = 16 / ES;          // columns per chunk
    __shared__ u32 T[P][64][DW + 1];
    __shared__ int cs[64];
    const int8_t *B8 = (const int8_t *)Bv;
    const int tid = threadIdx.x, cc = tid % CC, rg = tid / CC;
    const int j0 = blockIdx.x * 64;
    const int kb = blockIdx.y * kspan, ke = min(k_pad, kb + kspan);
    const int nlen = n - j0;
    int shh[8] = {0, 0, 0, 0, 0, 0, 0, 0}, sll[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    // this thread's column sums of the current block (bsB)
    int bh[8] = {0, 0, 0, 0, 0, 0, 0, 0}, bl[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    __shared__ int bcs[64][2];
    // Adds the current block's column sums into bsB (uniform: every thread
    // calls it at the same pass).
    auto flush = [&](int b) {
        if (tid < 128) (&bcs[0][0])[tid] = 0;
        __syncthreads();
        // the 8 lanes of a wave with one chunk cc (lanes cc + 8 j) first
#pragma unroll
        for (int c = 0; c < 8; ++c) {
#pragma unroll
            for (int o = 8; o < 64; o <<= 1) {
                bh[c] += __shfl_xor(bh[c], o);
                bl[c] += __shfl_xor(bl[c], o);
            }
        }
        if ((tid & 63) < 8) {
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                atomicAdd(&bcs[cc * 8 + c][0], bh[c]);
                atomicAdd(&bcs[cc * 8 + c][1], bl[c]);
            }
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            bh[c] = 0;
            bl[c] = 0;
        }
        __syncthreads();
        if (tid < 64) {
            atomicAdd(&bsB[((int64_t)b * n_pad + j0 + tid) * 2], (u32)bcs[tid][0]);
            atomicAdd(&bsB[((int64_t)b * n_pad + j0 + tid) * 2 + 1], (u32)bcs[tid][1]);
        }
        __syncthreads();
    };
    if (tid < 64) cs[tid] = 0;
    for (int p0 = kb; p0 < ke; p0 += ROWS) {
        if constexpr (ES == 2)
            if (bsB != nullptr && p0 > kb && p0 % bspan == 0) flush(p0 / bspan - 1);
        v4i x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int p = p0 + 4 * rg + r;
            const int len = p < k ? nlen : 0;
            const void *rowp = B8 + ((int64_t)(p < k ? p : 0) * ldb + j0) * ES;
            x[r] = load16<ES, VEC>(rowp, cc * CPU, len);
        }
        const u32 rmask = ES == 2 ? byte_mask(k - (p0 + 4 * rg)) : 0xffffffffu;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            u32 y[4];
            transpose4x4((u32)x[0][d], (u32)x[1][d], (u32)x[2][d], (u32)x[3][d], y[0], y[1],
                         y[2], y[3]);
            if constexpr (ES == 1) {
#pragma unroll
                for (int t = 0; t < 4; ++t) T[0][cc * 16 + 4 * d + t][rg] = y[t];
            } else {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const u32 lo = (y[2 * h] ^ 0x80808080u) & rmask;
                    const u32 hi = y[2 * h + 1] & rmask;
                    const int c = 2 * d + h;
                    shh[c] = sum4(hi, shh[c]);
                    sll[c] = sum4(lo, sll[c]);
                    if (bsB != nullptr) {
                        bh[c] = sum4(hi, bh[c]);
                        bl[c] = sum4(lo, bl[c]);
                    }
                    T[0][cc * 8 + c][rg] = hi;
                    T[1][cc * 8 + c][rg] = lo;
                }
            }
        }
        __syncthreads();
        // P planes x 64 columns x ROWS bytes, in 16-byte chunks.
        constexpr int CH = ROWS / 16;
        for (int idx = tid; idx < P * 64 * CH; idx += 256) {
            const int plane = idx / (64 * CH), rem = idx % (64 * CH);
            const int col = rem / CH, ch = rem % CH;
            const u32 *src = &T[plane][col][4 * ch];
            v4i v;
            v.x = (int)src[0];
            v.y = (int)src[1];
            v.z = (int)src[2];
            v.w = (int)src[3];
            int8_t *dst = (plane ? Bp1 : Bp0) + (int64_t)(j0 + col) * k_pad + p0 + ch * 16;
            *(v4i *)dst = v;
        }
        __syncthreads();
    }
    if constexpr (ES == 2) {
        if (bsB != nullptr && ke > kb) flush((ke - 1) / bspan);
#pragma unroll
        for (int c = 0; c < 8; ++c) atomicAdd(&cs[cc * 8 + c], (int)(32768u * (u32)shh[c] + 128u * (u32)sll[c]));
        __syncthreads();
        if (tid < 64) atomicAdd(&corrB[j0 + tid], (u32)cs[tid]);
    }
}

// ---- the packed-operand GEMM ---------------------------------------------
// A planes: P x m_pad x k_pad (row stride lda_p, plane stride a_plane), B
// planes: P x n_pad x k_pad; ktiles k-tiles of 64 from the given origin. NST is
// the number of LDS stages of the DMA ring (4, or 3 for tiles whose stage
// is too large for four).
// EPI 1 (int16 only): C is int16 (passed through the int32 pointer) and
// gets srs(A B) of this launch's k range added modulo 2^16, the product
// converted by an arithmetic shift right by (epi & 0xff) bits (half a unit
// added first when bit 8 is set) and saturation; corrA / corrB then hold the
// exact (high, low) limb sums of the range per row / column, and kconst is
// 16384 times the range's length.
// EPI 2-5 (int16 only): the int16-output update of every k block in one
// launch (the form of the conversion by shift range, below). The k range is
// kcb-tile blocks (kcb a multiple of 4 and at most 32, i.e. k_c <= 2048;
// ktiles = nblocks kcb, at most 16 blocks; shift <= 16); corrA / corrB hold
// the exact (high, low) limb sums of every block (block q at
// 2 (q m_pad + row), as the pack kernels write them), staged in LDS at the
// start; kconst is 16384 kcb 64. At the end of each block the lane converts
// its accumulators into the block's int16 contribution (the conversion of
// EPI 1) and adds it to running sums kept in registers; the accumulators
// restart at zero; C is read and written once.
// RAGGED: ktiles need not be a multiple of four (at least three), so that the
// zero padding of k to a multiple of 256 is not multiplied; otherwise it is.
// SKIPZ (short k, one k range): kcb counts the k-tiles that hold data, and the
// MFMAs of the zero-padding tiles past them are skipped (RAGGED's run-time
// tail needs more registers than eight waves have).
template <int ES, int BM, int BN, int WM, int WN, int NST, int EPI = 0, bool RAGGED = false,
          bool SKIPZ = false>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64, 1)
igemm_packed(const int8_t *__restrict__ Ap, int64_t lda_p, int64_t a_plane,
             const int8_t *__restrict__ Bp, int64_t ldb_p, int64_t b_plane,
             const uint32_t *__restrict__ corrA, const uint32_t *__restrict__ corrB,
             uint32_t kconst, int32_t *__restrict__ C, int64_t ldc,
             int m, int n, int ktiles, int tiles_m, int tiles_n, int epi, int kcb = 0,
             int m_pad = 0, int n_pad = 0) {
    constexpr int MF = 32;
    typedef Mfma<MF> M;
    typedef typename M::acc_t acc_t;
    constexpr int P = ES;
    constexpr int NACC = ES == 2 ? 3 : 1;
    constexpr int TM = WM / MF, TN = WN / MF;
    constexpr int WGN = BN / WN;
    // Four waves (one per SIMD), or eight (two per SIMD, at most 256
    // registers each, so that one wave's waits are covered by the other).
    constexpr int NW = (BM / WM) * WGN;
    static_assert(NW == 4 || NW == 8, "four or eight waves per workgroup");
    static_assert(NST == 3 || NST == 4, "three or four LDS stages");
    constexpr int APL = BM * 64, BPL = BN * 64;
    constexpr int STAGE = P * (APL + BPL);
    static_assert(NST * STAGE <= 160 * 1024, "gfx950 LDS");
    // 1 KB DMA blocks per stage: NBA hold the A planes, NBB the B planes;
    // each wave moves DPA of the A blocks and DPB of the B blocks.
    constexpr int NBA = P * BM / 16, NBB = P * BN / 16;
    static_assert(NBA % NW == 0 && NBB % NW == 0, "DMA blocks per wave");
    constexpr int DPA = NBA / NW, DPB = NBB / NW, DPW = DPA + DPB;
    static_assert(DPW <= 15, "outstanding DMA count fits s_waitcnt");
    static_assert(EPI == 0 || ES == 2, "the int16-output update is for int16 operands");
    // EPI 2-5: the multi-block update; its shift range selects the form of the
    // conversion (2: shift 0, 3: shift 1-7, 4: shift 8-16, 5: shift 0 with
    // blocks of 256).
    constexpr bool MULTI = EPI >= 2;
    constexpr int SMODE = EPI - 2;
    static_assert(!MULTI || !RAGGED, "blocks of whole groups of four k-tiles");
    static_assert(!SKIPZ || (!MULTI && !RAGGED), "zero tiles skipped in one k range");
    constexpr int MAXB = 16;  // blocks of one multi-block launch

    // The LDS stages as separate objects, so that the compiler can tell the
    // DMA writes of one stage from the fragment reads of another.
    __shared__ __attribute__((aligned(16))) char st0[STAGE];
    __shared__ __attribute__((aligned(16))) char st1[STAGE];
    __shared__ __attribute__((aligned(16))) char st2[STAGE];
    __shared__ __attribute__((aligned(16))) char st3[NST == 4 ? STAGE : 16];
    auto stage = [&](auto s) -> char * {
        constexpr int S = decltype(s)::value;
        static_assert(S < NST, "stage index");
        if constexpr (S == 0) return st0;
        else if constexpr (S == 1) return st1;
        else if constexpr (S == 2) return st2;
        else return st3;
    };

    const int tid = threadIdx.x, lane = tid & 63;
    // wave-uniform, so that DMA sources and destinations are scalar values
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

    // EPI 2-5: every block's limb sums of this tile's rows and columns, in LDS,
    // moved by DMA (1 KB per block and operand, spread over the waves) ahead
    // of the prologue's tiles, whose wait and barrier cover them.
    __shared__ __attribute__((aligned(16))) uint2 bsA[MULTI ? MAXB * BM : 1];
    __shared__ __attribute__((aligned(16))) uint2 bsB[MULTI ? MAXB * BN : 1];
    if constexpr (MULTI) {
        static_assert(BM * 8 == 1024 && BN * 8 == 1024, "one DMA block per block's sums");
        const int nblocks = ktiles / kcb;
        for (int x = wave; x < 2 * nblocks; x += NW) {
            const bool on_a = x < nblocks;
            const int q = on_a ? x : x - nblocks;
            const char *g = on_a ? (const char *)corrA + ((int64_t)q * m_pad + m0) * 8
                                 : (const char *)corrB + ((int64_t)q * n_pad + n0) * 8;
            char *d = on_a ? (char *)bsA + q * 1024 : (char *)bsB + q * 1024;
            dma16(g + 16 * lane, (lds_void *)d);
        }
    }

    // DMA: lane i of a 1 KB block writes LDS bytes [16i, 16i+16), i.e. row
    // r0 + i/4 of the block, physical chunk i%4, which holds logical chunk
    // (i%4) ^ swz(row); r0 is a multiple of 16, so swz(row) = swz(i/4). The
    // source is a wave-uniform block base plus a per-lane 32-bit offset that
    // is the same for every block of an operand (the planner keeps 16 rows
    // of a plane below 2^32 bytes).
    const u32 lrow = (u32)(lane >> 2);
    const u32 lq = (u32)((lane & 3) ^ swz(lane >> 2));
    const u32 a_loff = lrow * (u32)lda_p + 16u * lq;
    const u32 b_loff = lrow * (u32)ldb_p + 16u * lq;
    const int8_t *src[DPW];
    int ldsoff[DPW];
#pragma unroll
    for (int d = 0; d < DPW; ++d) {
        if (d < DPA) {
            const int b = wave * DPA + d;
            const int plane = b / (BM / 16), r0 = (b % (BM / 16)) * 16;
            src[d] = Ap + plane * a_plane + (int64_t)(m0 + r0) * lda_p;
            ldsoff[d] = b * 1024;
        } else {
            const int bb = wave * DPB + (d - DPA);
            const int plane = bb / (BN / 16), r0 = (bb % (BN / 16)) * 16;
            src[d] = Bp + plane * b_plane + (int64_t)(n0 + r0) * ldb_p;
            ldsoff[d] = (NBA + bb) * 1024;
        }
    }
    // DMA blocks [D0, D1) of k-tile kt into stage s.
    auto dma_range = [&](auto s, int kt, auto d0, auto d1) {
        constexpr int D0 = decltype(d0)::value, D1 = decltype(d1)::value;
        char *dst = stage(s);
        const int64_t koff = (int64_t)kt * 64;
#pragma unroll
        for (int d = D0; d < D1; ++d)
            dma16(src[d] + koff + (d < DPA ? a_loff : b_loff), (lds_void *)(dst + ldsoff[d]));
    };

    // Fragment reads (same LDS layout as the fused kernels).
    const int fr = M::frag_row(lane);
    int a_rbase[2], b_rbase[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int cq = (M::frag_chunk(lane, ks) ^ swz(fr)) << 4;
        a_rbase[ks] = (wm0 + fr) * 64 + cq;
        b_rbase[ks] = (wn0 + fr) * 64 + cq;
    }
    v4i fa[2][P][TM], fb[2][P][TN];
    auto read_frags = [&](auto slot, auto s, auto ks) {
        constexpr int SL = decltype(slot)::value;
        constexpr int KS = decltype(ks)::value;
        const char *As = stage(s);
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

    acc_t acc[NACC][TM][TN];
#pragma unroll
    for (int a = 0; a < NACC; ++a)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < M::REGS; ++r) acc[a][i][j][r] = 0;
    // FRESH: the first products of a k block start from zero (a zero
    // accumulator operand) instead of adding to the accumulators.
    auto mfmas = [&](auto slot, auto fresh) {
        constexpr int SL = decltype(slot)::value;
        constexpr bool FRESH = decltype(fresh)::value != 0;
        const acc_t zero = {};
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if constexpr (ES == 1) {
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] = M::mma(fa[SL][0][i], fb[SL][0][j], acc[0][i][j]);
            } else {
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] =
                        M::mma(fa[SL][0][i], fb[SL][0][j], FRESH ? zero : acc[0][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[1][i][j] =
                        M::mma(fa[SL][0][i], fb[SL][1][j], FRESH ? zero : acc[1][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[2][i][j] =
                        M::mma(fa[SL][1][i], fb[SL][1][j], FRESH ? zero : acc[2][i][j]);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[1][i][j] = M::mma(fa[SL][1][i], fb[SL][0][j], acc[1][i][j]);
            }
        }
    };

    // s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14.
    constexpr int WAIT_NEWEST = (DPW & 0xf) | (0x7 << 4) | (0xf << 8);
    constexpr int WAIT_ALL = (0x7 << 4) | (0xf << 8);

    constexpr int NM = TM * TN * (ES == 2 ? 4 : 1);  // MFMAs per sub-step
    constexpr int NR = P * (TM + TN);                // fragment reads per sub-step
    // DMA issue: with four stages the next tile's loads are spread over both
    // sub-steps, with three (less slack) over the first sub-step only.
    constexpr int D_SUB0 = NST == 4 ? DPW / 2 : DPW;
    // Step kt (S = kt mod NST): stages S and S+1 hold tiles kt and kt+1, slot
    // 0 holds sub-step 0 of tile kt. Start the DMA of tile kt+NST-1 (if there
    // is one) into the stage that held tile kt-1, run both sub-steps while
    // reading the next fragments, then wait until tile kt+2 has landed (with
    // four stages tile kt+3 may stay in flight) and synchronise. The last
    // steps start no DMA and the last one prefetches nothing, so no copy is
    // in flight when the epilogue starts (the compiler then tracks the C
    // loads' completion precisely instead of waiting for every load before a
    // store). Each sub-step opens with an MFMA, and its fragment reads follow
    // MFMAs: the compiler cannot tell the DMA loads' LDS writes apart from
    // other LDS traffic, so any wait for a fragment is a full lgkmcnt(0), and
    // this order makes that wait cover only reads issued a sub-step earlier.
    auto step = [&](auto s, int kt, auto do_dma, auto do_pref, auto fresh) {
        constexpr int S = decltype(s)::value;
        constexpr int SD = (S + NST - 1) % NST;  // stage receiving the DMA
        constexpr bool DMA = decltype(do_dma)::value != 0;
        constexpr bool PREF = decltype(do_pref)::value != 0;
        if constexpr (DMA) dma_range(ic<SD>{}, kt + NST - 1, ic<0>{}, ic<D_SUB0>{});
        read_frags(ic<1>{}, ic<S>{}, ic<1>{});
        if (!SKIPZ || kt < kcb) mfmas(ic<0>{}, fresh);
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if (DMA && (i * D_SUB0) / NM != ((i + 1) * D_SUB0) / NM)
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (DMA && D_SUB0 < DPW)
            dma_range(ic<SD>{}, kt + NST - 1, ic<D_SUB0>{}, ic<DPW>{});
        if constexpr (PREF) read_frags(ic<0>{}, ic<(S + 1) % NST>{}, ic<0>{});
        if (!SKIPZ || kt < kcb) mfmas(ic<1>{}, ic<0>{});
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (PREF && i < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if (DMA && D_SUB0 < DPW &&
                (i * (DPW - D_SUB0)) / NM != ((i + 1) * (DPW - D_SUB0)) / NM)
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (PREF) {
            __builtin_amdgcn_s_waitcnt(DMA && NST == 4 ? WAIT_NEWEST : WAIT_ALL);
            __builtin_amdgcn_s_barrier();
        }
    };
    // The last T steps from a stage-0 step at kt0: step j starts a DMA only if
    // tile j+NST-1 exists and prefetches only if tile j+1 exists.
    // (FRESH: the first of them opens a k block.)
    auto tail_step = [&](auto jc, auto tc, int kt0, auto fresh) {
        constexpr int J = decltype(jc)::value, T = decltype(tc)::value;
        if constexpr (J < T)
            step(ic<J % NST>{}, kt0 + J, ic<(J + NST - 1 < T)>{}, ic<(J + 1 < T)>{},
                 ic<(J == 0 && decltype(fresh)::value != 0)>{});
    };
    auto tail = [&](auto tc, int kt0, auto fresh) {
        tail_step(ic<0>{}, tc, kt0, fresh);
        tail_step(ic<1>{}, tc, kt0, fresh);
        tail_step(ic<2>{}, tc, kt0, fresh);
        tail_step(ic<3>{}, tc, kt0, fresh);
        tail_step(ic<4>{}, tc, kt0, fresh);
        tail_step(ic<5>{}, tc, kt0, fresh);
    };

    // Prologue: tiles 0 .. NST-2 into stages 0 .. NST-2; tiles 0 and 1 must
    // have landed (with four stages tile 2 may stay in flight).
    dma_range(ic<0>{}, 0, ic<0>{}, ic<DPW>{});
    dma_range(ic<1>{}, 1, ic<0>{}, ic<DPW>{});
    if constexpr (NST == 4) dma_range(ic<2>{}, 2, ic<0>{}, ic<DPW>{});
    __builtin_amdgcn_s_waitcnt(NST == 4 ? WAIT_NEWEST : WAIT_ALL);
    __builtin_amdgcn_s_barrier();
    read_frags(ic<0>{}, ic<0>{}, ic<0>{});
    // Groups of NST steps in which every step starts a DMA and prefetches,
    // then the remaining T = ktiles - kt steps (T in [NST-1, 2*NST-2];
    // ktiles >= NST - 1, a multiple of four unless RAGGED). The planes are
    // zero-padded to a multiple of four k-tiles, so the prologue's loads stay
    // inside them.
    // EPI 2-5: this lane's running int16 sums, two per register (16-bit lanes
    // that wrap modulo 2^16, as the update of C does), and the conversion of
    // block q's accumulators into them.
    typedef short s2 __attribute__((ext_vector_type(2)));
    constexpr int RT = MULTI ? TM : 1, RN = MULTI ? TN : 1;
    constexpr int RR = MULTI ? M::REGS / 2 : 1;
    s2 run16[RT][RN][RR];
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j)
#pragma unroll
            for (int r = 0; r < RR; ++r) run16[i][j][r] = s2{0, 0};
    // The conversion runs in 32-bit integer arithmetic; the host takes this
    // launch only for blocks of k_c <= 2048 elements and shifts <= 16. With
    //   X = S_x + 128 (hA + hB),  L = S_ll + 128 (l'A + l'B) + 16384 k_c
    // (hA, l'A: the row's limb sums over the block; hB, l'B: the column's),
    // the block's exact product is v = 65536 S_hh + 256 X + L, where
    // |S_hh| <= 2^14 k_c <= 2^25 and |X|, |L| <= 2^16 k_c <= 2^27. Then
    //   y = floor(v / 256) = 256 S_hh + X + (L >> 8),  v = 256 y + (L & 255).
    // S_hh is clamped to [-2^21, 2^21] first: inside, y is exact and
    // |y| < 2^30; outside, |v| > 2^36 and the clamped y (|y| > 2^28, same
    // sign) saturates the same way for every shift <= 16. The shift then
    // takes one of two forms:
    //   shift >= 8: floor((v + half) / 2^s) = (y + ((L & 255) + half) >> 8) >> (s - 8)
    //   shift <  8: y is clamped to [-2^22, 2^22] (beyond it |v| >= 2^30 - 255
    //               saturates for every shift < 8) and v = 256 y + (L & 255)
    //               is formed exactly, then (v + half) >> s.
    // Arithmetic shifts right are floors; half = 2^(s-1) with rounding, else 0;
    // the saturation to int16 is that of v_cvt_pk_i16_i32.
    // Shift 0 (the paper's case) takes a shorter form: y is saturated to int16
    // (a pair at a time), v' = 256 sat16(y) + (L & 255) is formed exactly from
    // its bytes (sign-extended), and sat16(v') = sat16(v): v' = v when y fits,
    // and otherwise both lie beyond the int16 range on the same side. With
    // blocks of 256 (EPI 5) |S_hh| <= 2^22, so y = 256 S_hh + X + (L >> 8) fits
    // in 32 bits (|y| < 2^30 + 2^25) without the clamp of S_hh.
    auto convert = [&](int q) {
        if constexpr (MULTI) {
            const int sh = epi & 0xff;
            const int half = ((epi >> 8) & 1) != 0 && sh > 0 ? 1 << (sh - 1) : 0;
            int colM[TN], colL[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const uint2 v = bsB[q * BN + wn0 + MF * j + M::out_col(lane)];
                colM[j] = (int)(v.x << 7);
                colL[j] = (int)((v.y << 7) + kconst);
            }
            // One output block at a time, so that few accumulators are live
            // outside the AGPRs (the next block's first products overwrite
            // them: FRESH steps).
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                int rowM[M::REGS], rowL[M::REGS];
#pragma unroll
                for (int r = 0; r < M::REGS; ++r) {
                    const uint2 v = bsA[q * BM + wm0 + MF * i + M::out_row(lane, r)];
                    rowM[r] = (int)(v.x << 7);
                    rowL[r] = (int)(v.y << 7);
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
#pragma unroll
                    for (int r2 = 0; r2 < M::REGS / 2; ++r2) {
                        if constexpr (SMODE == 0 || SMODE == 3) {
                            int y2[2], L2[2];
#pragma unroll
                            for (int h = 0; h < 2; ++h) {
                                const int r = 2 * r2 + h;
                                const int hh =
                                    SMODE == 3 ? acc[0][i][j][r]
                                               : min(max(acc[0][i][j][r], -(1 << 21)), 1 << 21);
                                L2[h] = acc[2][i][j][r] + rowL[r] + colL[j];
                                y2[h] = (int)((u32)hh << 8) + acc[1][i][j][r] + rowM[r] +
                                        colM[j] + (L2[h] >> 8);
                            }
                            const u32 yp =
                                __builtin_bit_cast(u32, __builtin_amdgcn_cvt_pk_i16(y2[0], y2[1]));
                            // bytes: the lowest of L, the two of sat16(y), its sign
                            const int v0 = (int)perm(yp, (u32)L2[0], 0x0A050400u);
                            const int v1 = (int)perm(yp, (u32)L2[1], 0x0B070600u);
                            run16[i][j][r2] += __builtin_amdgcn_cvt_pk_i16(v0, v1);
                            continue;
                        }
                        int t32[2];
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            const int r = 2 * r2 + h;
                            const int hh = min(max(acc[0][i][j][r], -(1 << 21)), 1 << 21);
                            const int L = acc[2][i][j][r] + rowL[r] + colL[j];
                            const int y = (int)((u32)hh << 8) + acc[1][i][j][r] + rowM[r] +
                                          colM[j] + (L >> 8);
                            int t;
                            if constexpr (SMODE == 2) {
                                t = (y + (((L & 255) + half) >> 8)) >> (sh - 8);
                            } else {
                                const int yc = min(max(y, -(1 << 22)), 1 << 22);
                                // bytes: the lowest of L, then the lower three of yc
                                t = (int)perm((u32)yc, (u32)L, 0x06050400u);
                                if constexpr (SMODE == 1) t = (t + half) >> sh;
                            }
                            t32[h] = t;
                        }
                        // v_cvt_pk_i16_i32 saturates each to int16 (checked on the
                        // device); the running sums wrap modulo 2^16
                        run16[i][j][r2] += __builtin_amdgcn_cvt_pk_i16(t32[0], t32[1]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };
    int kt = 0;
    for (; kt <= ktiles - 2 * NST + 1; kt += NST) {
        // (k blocks of the multi-block update start at multiples of kcb, a
        // multiple of NST = 4, so only the first step of a group opens one)
        if (MULTI && kt % kcb == 0)
            step(ic<0>{}, kt, ic<1>{}, ic<1>{}, ic<1>{});
        else
            step(ic<0>{}, kt, ic<1>{}, ic<1>{}, ic<0>{});
        step(ic<1>{}, kt + 1, ic<1>{}, ic<1>{}, ic<0>{});
        step(ic<2>{}, kt + 2, ic<1>{}, ic<1>{}, ic<0>{});
        if constexpr (NST == 4) step(ic<3>{}, kt + 3, ic<1>{}, ic<1>{}, ic<0>{});
        if constexpr (MULTI)
            if ((kt + NST) % kcb == 0) convert((kt + NST) / kcb - 1);
    }
    if constexpr (NST == 4 && !RAGGED) {
        // the last group of four opens a block only when blocks are four tiles
        if (MULTI && kcb == 4)
            tail(ic<4>{}, kt, ic<1>{});
        else
            tail(ic<4>{}, kt, ic<0>{});
        if constexpr (MULTI) convert(ktiles / kcb - 1);
    } else if constexpr (NST == 4) {
        // T = ktiles - kt lies in [3, 6] (the host passes ktiles >= 3).
        const int T = ktiles - kt;
        if (T == 4)
            tail(ic<4>{}, kt, ic<0>{});
        else if (T == 3)
            tail(ic<3>{}, kt, ic<0>{});
        else if (T == 5)
            tail(ic<5>{}, kt, ic<0>{});
        else
            tail(ic<6>{}, kt, ic<0>{});
    } else {
        const int T = ktiles - kt;
        if (T == 2)
            tail(ic<2>{}, kt, ic<0>{});
        else if (T == 3)
            tail(ic<3>{}, kt, ic<0>{});
        else
            tail(ic<4>{}, kt, ic<0>{});
    }
    // ---- epilogue -----------------------------------------------------------
    // int16 corrections (first k chunk only): the column term of each output
    // column and the row term of each output row of this lane.
    u32 colt[TN], rowt[TM][M::REGS];
#pragma unroll
    for (int j = 0; j < TN; ++j) colt[j] = 0;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < M::REGS; ++r) rowt[i][r] = 0;
    if constexpr (ES == 2 && EPI == 0) {
        if (corrA != nullptr) {
#pragma unroll
            for (int j = 0; j < TN; ++j)
                colt[j] = kconst + corrB[n0 + wn0 + MF * j + M::out_col(lane)];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int r = 0; r < M::REGS; ++r)
                    rowt[i][r] = corrA[m0 + wm0 + MF * i + M::out_row(lane, r)];
        }
    }
    // C is accessed through a buffer resource based at the tile's corner,
    // with 32-bit byte offsets (the planner keeps bm * ldc * 4 below 2^31).
    // Elements outside m x n get an offset beyond the resource's range: the
    // hardware returns 0 for such loads and drops such stores, so the
    // epilogue has no branches and the compiler can count the outstanding
    // loads exactly (with a branch per element it waits for all of them
    // before every store).
    constexpr u32 CE = EPI != 0 ? 2u : 4u;  // bytes per C element
    const __amdgpu_buffer_rsrc_t Crs = __builtin_amdgcn_make_buffer_rsrc(
        (char *)C + ((int64_t)m0 * ldc + n0) * CE, 0, 0x7fffffff, 0x00020000);
    const int ldc32 = (int)ldc;
    auto c_off = [&](int lr, int lc) -> u32 {
        return (m0 + lr < m && n0 + lc < n) ? (u32)(lr * ldc32 + lc) * CE : 0x80000000u;
    };
    // EPI 1: exact (high, low) limb sums of this lane's columns; the rows'
    // are loaded with each batch.
    int colh[EPI == 1 ? TN : 1], coll[EPI == 1 ? TN : 1];
    if constexpr (EPI == 1) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const uint2 q = *(const uint2 *)(corrB + 2 * (n0 + wn0 + MF * j + M::out_col(lane)));
            colh[j] = (int)q.x;
            coll[j] = (int)q.y;
        }
    }
    const int srs_shift = epi & 0xff;
    const int64_t srs_half =
        ((epi >> 8) & 1) != 0 && srs_shift > 0 ? (int64_t)1 << (srs_shift - 1) : 0;
    // C is read, added to and written back in batches of NB output blocks,
    // software-pipelined: the loads of batch b+1 are issued before batch b is
    // added and stored, so a wave keeps up to 2 * NB * REGS loads in flight.
    // (All workgroups of a round reach this point together; one round trip
    // per block would leave the matrix cores idle for many microseconds.)
    constexpr int NOUT = TM * TN;
    // Eight waves (256 registers each) keep one block per batch.
    constexpr int NB = NW == 8 ? 1 : (NOUT <= 4 ? NOUT : 2);
    constexpr int NBATCH = NOUT / NB;
    static_assert(NOUT % NB == 0 && NBATCH <= 8, "epilogue batches");
    int32_t cv[2][NB][M::REGS];
    uint2 rv[EPI == 1 ? 2 : 1][EPI == 1 ? NB : 1][EPI == 1 ? M::REGS : 1];
    auto load_batch = [&](auto buf, auto batch) {
        constexpr int BF = decltype(buf)::value, B0 = decltype(batch)::value * NB;
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) {
            const int i = (B0 + bb) / TN, j = (B0 + bb) % TN;
            const int lc = wn0 + MF * j + M::out_col(lane);
#pragma unroll
            for (int r = 0; r < M::REGS; ++r) {
                const int lr = wm0 + MF * i + M::out_row(lane, r);
                if constexpr (EPI == 1) {
                    cv[BF][bb][r] = (int32_t)(int16_t)__builtin_amdgcn_raw_buffer_load_b16(
                        Crs, c_off(lr, lc), 0, 0);
                    rv[BF][bb][r] = *(const uint2 *)(corrA + 2 * (m0 + lr));
                } else if constexpr (MULTI) {
                    cv[BF][bb][r] = (int32_t)(int16_t)__builtin_amdgcn_raw_buffer_load_b16(
                        Crs, c_off(lr, lc), 0, 0);
                } else {
                    cv[BF][bb][r] =
                        __builtin_amdgcn_raw_buffer_load_b32(Crs, c_off(lr, lc), 0, 0);
                }
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
                if constexpr (EPI == 1) {
                    // exact product of this k range, converted and added mod 2^16
                    const int64_t a64 =
                        (int64_t)acc[0][i][j][r] * 65536 + (int64_t)acc[1][i][j][r] * 256 +
                        (int64_t)acc[2][i][j][r] +
                        (int64_t)((int)rv[BF][bb][r].x + colh[j]) * 32768 +
                        (int64_t)((int)rv[BF][bb][r].y + coll[j]) * 128 + (int64_t)kconst;
                    int64_t t = (a64 + srs_half) >> srs_shift;
                    t = t > 32767 ? 32767 : (t < -32768 ? -32768 : t);
                    __builtin_amdgcn_raw_buffer_store_b16(
                        (unsigned short)(u32)(cv[BF][bb][r] + (int32_t)t), Crs, c_off(lr, lc), 0,
                        0);
                    continue;
                }
                if constexpr (MULTI) {
                    // the sum of every block's conversion, added modulo 2^16
                    __builtin_amdgcn_raw_buffer_store_b16(
                        (unsigned short)(u32)(cv[BF][bb][r] + (int)run16[i][j][r / 2][r & 1]),
                        Crs, c_off(lr, lc), 0, 0);
                    continue;
                }
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

}  // namespace packed

using namespace packed;

// ---------------------------------------------------------------------------
// Host side of the packed path.

int launch_pack_a(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, void *a_part, void *b_part_to_clear, void *stream_,
                  uint32_t *sums, int64_t kc, int64_t nblocks) {
    hipStream_t stream = (hipStream_t)stream_;
    PackedLayout L;
    packed_layout(es, m, n, k, p.kernel, A, lda, &L);
    if (!L.pack_a) return IGEMM_OK;
    int8_t *wa = (int8_t *)a_part;
    const bool va = p.vec_a != 0;
    const int mi = (int)m, ki = (int)k, kp = (int)L.k_pad, np = (int)L.n_pad;
    int8_t *Apk = wa + L.off_a;
    uint32_t *corrA = (uint32_t *)(wa + L.off_corr_a);
    uint32_t *corrB = b_part_to_clear != nullptr
                          ? (uint32_t *)((int8_t *)b_part_to_clear + L.off_corr_b)
                          : nullptr;
    const int64_t a_plane = L.m_pad * L.k_pad;
    const dim3 g((unsigned)L.m_pad);
    if (es == 2) {
        int8_t *Al = Apk + a_plane;
        const int16_t *A16 = (const int16_t *)A;
        // int16-output update: A's block sums, and B's cleared for pack_b
        const int bspan = sums != nullptr ? (int)(nblocks == 1 ? L.k_pad : kc) : 0;
        const int nb = sums != nullptr ? (int)nblocks : 0;
        uint32_t *clr = sums != nullptr ? sums + 2 * nblocks * L.m_pad : nullptr;
        const int nclr = sums != nullptr ? (int)(2 * nblocks * L.n_pad) : 0;
        const int mp = (int)L.m_pad;
        if (kp <= 512) {
            // short rows: one wave per row (m_pad is a multiple of 128)
            const dim3 g4((unsigned)(L.m_pad / 4));
            if (va)
                pack_a_i16_rows<true><<<g4, 256, 0, stream>>>(A16, lda, mi, ki, kp, Apk, Al, corrA,
                                                              corrB, np, sums, bspan, mp, clr, nclr);
            else
                pack_a_i16_rows<false><<<g4, 256, 0, stream>>>(A16, lda, mi, ki, kp, Apk, Al,
                                                               corrA, corrB, np, sums, bspan, mp,
                                                               clr, nclr);
        } else if (va)
            pack_a_i16<true><<<g, 256, 0, stream>>>(A16, lda, mi, ki, kp, Apk, Al, corrA, corrB, np,
                                                    sums, bspan, nb, clr, nclr);
        else
            pack_a_i16<false><<<g, 256, 0, stream>>>(A16, lda, mi, ki, kp, Apk, Al, corrA, corrB,
                                                     np, sums, bspan, nb, clr, nclr);
    } else {
        const int8_t *A8 = (const int8_t *)A;
        if (va)
            pack_a_i8<true><<<g, 256, 0, stream>>>(A8, lda, mi, ki, kp, Apk);
        else
            pack_a_i8<false><<<g, 256, 0, stream>>>(A8, lda, mi, ki, kp, Apk);
    }
    return hipGetLastError() == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

int launch_pack_b(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                  int64_t lda, const void *B, int64_t ldb, void *b_part, bool clear_corr,
                  void *stream_, uint32_t *sums, int64_t kc, int64_t nblocks) {
    hipStream_t stream = (hipStream_t)stream_;
    PackedLayout L;
    packed_layout(es, m, n, k, p.kernel, A, lda, &L);
    int8_t *wb = (int8_t *)b_part;
    const bool vb = p.vec_b != 0;
    const int ni = (int)n, ki = (int)k, kp = (int)L.k_pad, np = (int)L.n_pad;
    int8_t *Bpk = wb + L.off_b;
    uint32_t *corrB = (uint32_t *)(wb + L.off_corr_b);
    const int64_t b_plane = L.n_pad * L.k_pad;
    if (es == 2 && clear_corr) {
        clear_u32<<<dim3((unsigned)((np + 255) / 256)), 256, 0, stream>>>(corrB, np);
        if (hipGetLastError() != hipSuccess) return IGEMM_EHIP;
    }
    const dim3 g((unsigned)(L.n_pad / 64), (unsigned)L.b_slices);
    const int ks = (int)L.kspan;
    if (es == 2) {
        int8_t *Bl = Bpk + b_plane;
        // int16-output update: B's block sums (after A's; cleared by pack_a_i16)
        uint32_t *sb = sums != nullptr ? sums + 2 * nblocks * L.m_pad : nullptr;
        const int bspan = sums != nullptr ? (int)(nblocks == 1 ? L.k_pad : kc) : 0;
        if (vb)
            pack_b<2, true><<<g, 256, 0, stream>>>(B, ldb, ki, ni, kp, ks, np, Bpk, Bl, corrB, sb,
                                                   bspan);
        else
            pack_b<2, false><<<g, 256, 0, stream>>>(B, ldb, ki, ni, kp, ks, np, Bpk, Bl, corrB, sb,
                                                    bspan);
    } else {
        if (vb)
            pack_b<1, true><<<g, 256, 0, stream>>>(B, ldb, ki, ni, kp, ks, np, Bpk, Bpk, corrB);
        else
            pack_b<1, false><<<g, 256, 0, stream>>>(B, ldb, ki, ni, kp, ks, np, Bpk, Bpk, corrB);
    }
    return hipGetLastError() == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

int64_t srs_sums_bytes(const igemm_plan &p, int64_t m, int64_t n, int64_t k, int64_t nblocks,
                       const void *A, int64_t lda) {
    PackedLayout L;
    packed_layout(2, m, n, k, p.kernel, A, lda, &L);
    return 8 * nblocks * (L.m_pad + L.n_pad);
}

int launch_srs_packed(const igemm_plan &p, int64_t m, int64_t n, int64_t k, int64_t kc,
                      int64_t nblocks, const void *A, int64_t lda, int16_t *C, int64_t ldc,
                      const void *a_part, const void *b_part, uint32_t *sums, int shift,
                      int round_half_up, void *stream_) {
    hipStream_t stream = (hipStream_t)stream_;
    PackedLayout L;
    packed_layout(2, m, n, k, p.kernel, A, lda, &L);
    if (nblocks < 1 || nblocks > 64 || (nblocks > 1 && kc % 256 != 0)) return IGEMM_EINVAL;
    const int8_t *wa = (const int8_t *)a_part, *wb = (const int8_t *)b_part;
    const int8_t *Apk = wa + L.off_a, *Bpk = wb + L.off_b;
    const int64_t a_plane = L.m_pad * L.k_pad, b_plane = L.n_pad * L.k_pad;
    const int kb = nblocks == 1 ? (int)L.k_pad : (int)kc;  // block span in the planes
    // the block sums, written by the pack kernels
    uint32_t *sa = sums, *sb = sums + 2 * nblocks * L.m_pad;
    const KernelDesc &d = kKernels[p.kernel];
    const int tm = (int)(L.m_pad / d.bm), tn = (int)(L.n_pad / d.bn);
    const int mi = (int)m, ni = (int)n;
    const int epi = (shift & 0xff) | (round_half_up ? 0x100 : 0);
    const dim3 grid((unsigned)(tm * tn));
    // Two to sixteen whole blocks (k a multiple of kc) of at most 2048, shift
    // at most 16: one launch that converts each block in registers (32-bit
    // integer arithmetic, exact within these bounds) and updates C once.
    // Eight waves of 64 x 32 (two per SIMD), so that one wave's matrix-core
    // work covers the other's conversions: 4096^3 with k_c = 256 in 364-392
    // us against 402-434 us with four waves of 64 x 64 (k_c = 512: 335
    // against 369; 1024: 314 against 346).
    if (nblocks >= 2 && nblocks <= 16 && k % kc == 0 && L.k_pad == k && kc <= 2048 &&
        shift <= 16) {
        const int kcb = (int)(kc / 64), ktl = (int)(k / 64);
        const uint32_t kcon = 16384u * (uint32_t)kc;
#define IGEMM_SRS_MULTI(E)                                                                 \
    igemm_packed<2, 128, 128, 64, 32, 4, E><<<grid, 512, 0, stream>>>(                    \
        Apk, L.k_pad, a_plane, Bpk, L.k_pad, b_plane, sa, sb, kcon, (int32_t *)C, ldc, mi, \
        ni, ktl, tm, tn, epi, kcb, (int)L.m_pad, (int)L.n_pad)
        if (shift == 0 && kc == 256)
            IGEMM_SRS_MULTI(5);
        else if (shift == 0)
            IGEMM_SRS_MULTI(2);
        else if (shift < 8)
            IGEMM_SRS_MULTI(3);
        else
            IGEMM_SRS_MULTI(4);
#undef IGEMM_SRS_MULTI
        return hipGetLastError() == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
    }
    // Otherwise one launch per block, in order (the update modulo 2^16 makes
    // the order immaterial); block q spans [q kb, q kb + kb) of the planes.
    for (int64_t q = 0; q < nblocks; ++q) {
        const int64_t k0 = q * kb;
        const int64_t span = L.k_pad - k0 < kb ? L.k_pad - k0 : kb;   // a multiple of 256
        const int64_t real = (k - k0 < kb ? k - k0 : kb);              // elements inside k
        // k-tiles holding data, at least 3 (covered by the zero padding);
        // a multiple of four takes the variant with the tail fixed at build
        // time
        int ktiles = (int)((real + 63) / 64);
        if (ktiles < 3) ktiles = 3;
        if (ktiles > (int)(span / 64)) ktiles = (int)(span / 64);
        if (span <= 512) {
            // short blocks: eight waves, the zero tiles' MFMAs skipped
            igemm_packed<2, 128, 128, 64, 32, 4, 1, false, true><<<grid, 512, 0, stream>>>(
                Apk + k0, L.k_pad, a_plane, Bpk + k0, L.k_pad, b_plane, sa + 2 * q * L.m_pad,
                sb + 2 * q * L.n_pad, 16384u * (uint32_t)real, (int32_t *)C, ldc, mi, ni,
                (int)(span / 64), tm, tn, epi, (int)((real + 63) / 64));
        } else if (ktiles % 4 == 0)
            igemm_packed<2, 128, 128, 64, 64, 4, 1><<<grid, 256, 0, stream>>>(
                Apk + k0, L.k_pad, a_plane, Bpk + k0, L.k_pad, b_plane, sa + 2 * q * L.m_pad,
                sb + 2 * q * L.n_pad, 16384u * (uint32_t)real, (int32_t *)C, ldc, mi, ni, ktiles,
                tm, tn, epi);
        else
            igemm_packed<2, 128, 128, 64, 64, 4, 1, true><<<grid, 256, 0, stream>>>(
                Apk + k0, L.k_pad, a_plane, Bpk + k0, L.k_pad, b_plane, sa + 2 * q * L.m_pad,
                sb + 2 * q * L.n_pad, 16384u * (uint32_t)real, (int32_t *)C, ldc, mi, ni, ktiles,
                tm, tn, epi);
        if (hipGetLastError() != hipSuccess) return IGEMM_EHIP;
    }
    return IGEMM_OK;
}

int launch_multiply(int es, const igemm_plan &p, int64_t m, int64_t n, int64_t k, const void *A,
                    int64_t lda, int32_t *C, int64_t ldc, const void *a_part, const void *b_part,
                    void *stream_) {
    hipStream_t stream = (hipStream_t)stream_;
    PackedLayout L;
    packed_layout(es, m, n, k, p.kernel, A, lda, &L);
    const int8_t *wa = (const int8_t *)a_part, *wb = (const int8_t *)b_part;
    const int mi = (int)m, ni = (int)n;
    const int8_t *Bpk = wb + L.off_b;
    const uint32_t *corrA = (const uint32_t *)(wa + L.off_corr_a);
    const uint32_t *corrB = (const uint32_t *)(wb + L.off_corr_b);
    const int64_t a_plane = L.m_pad * L.k_pad, b_plane = L.n_pad * L.k_pad;
    const KernelDesc &d = kKernels[p.kernel];
    const int tm = (int)(L.m_pad / d.bm), tn = (int)(L.n_pad / d.bn);
    const int8_t *Asrc = L.pack_a ? wa + L.off_a : (const int8_t *)A;
    const int64_t lda_p = L.pack_a ? L.k_pad : lda;
    const dim3 grid((unsigned)p.grid);
    if (es == 2 && L.k_pad <= 512) {
        // Short k (one chunk of four or eight k-tiles): eight waves of 64 x 32,
        // the MFMAs of the zero tiles skipped. (4096, 4096, k) one call, us,
        // against four waves (RAGGED where it applied): k = 64 52.8 / 58.8,
        // 256 58.9 / 61.9, 290 68.3 / 71.5, 512 75.0 / 77.8.
        const int kr = (int)((k + kBK - 1) / kBK);
        igemm_packed<2, 128, 128, 64, 32, 4, 0, false, true><<<grid, 512, 0, stream>>>(
            Asrc, lda_p, a_plane, Bpk, L.k_pad, b_plane, corrA, corrB, 16384u * (uint32_t)k, C,
            ldc, mi, ni, (int)(L.k_pad / kBK), tm, tn, 0, kr);
        return hipGetLastError() == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
    }
    // One launch per k chunk; the row and column corrections and the
    // 16384 k constant are added by the first launch only.
    for (int64_t k0 = 0; k0 < L.k_pad; k0 += p.k_chunk) {
        const int64_t kc = L.k_pad - k0 < p.k_chunk ? L.k_pad - k0 : p.k_chunk;
        // int16: when the zero padding of k to a multiple of 256 spans three
        // k-tiles of 64, only the tiles holding data are multiplied, through
        // the RAGGED variant (the paper's k = 290: 5 k-tiles instead of 8).
        // Saving one or two tiles does not pay: on m = n = 4096 the RAGGED
        // kernel took 48.9 us for 3 tiles against 46.0 for 4, and 61.3 us
        // for 7 against 56.6 for 8 (54.0 us for 5).
        const int64_t real = k - k0 < kc ? k - k0 : kc;
        int ktiles = (int)(kc / 64);
        const int kr = (int)((real + 63) / 64);
        const bool ragged = es == 2 && kr % 4 == 1 && kr > 4 && kr < ktiles;
        if (ragged) ktiles = kr;
        const bool first = k0 == 0;
        const uint32_t *cA = first ? corrA : nullptr;
        const uint32_t kc16 = first ? 16384u * (uint32_t)k : 0u;
        if (es == 2 && ragged)
            igemm_packed<2, 128, 128, 64, 64, 4, 0, true><<<grid, 256, 0, stream>>>(
                Asrc + k0, lda_p, a_plane, Bpk + k0, L.k_pad, b_plane, cA, corrB, kc16, C, ldc,
                mi, ni, ktiles, tm, tn, 0);
        else if (es == 2)
            igemm_packed<2, 128, 128, 64, 64, 4><<<grid, 256, 0, stream>>>(
                Asrc + k0, lda_p, a_plane, Bpk + k0, L.k_pad, b_plane, cA, corrB, kc16, C, ldc,
                mi, ni, ktiles, tm, tn, 0);
        else
            igemm_packed<1, 256, 256, 64, 128, 4><<<grid, 512, 0, stream>>>(
                Asrc + k0, lda_p, 0, Bpk + k0, L.k_pad, 0, nullptr, nullptr, 0u, C, ldc, mi, ni,
                ktiles, tm, tn, 0);
        if (hipGetLastError() != hipSuccess) return IGEMM_EHIP;
    }
    return IGEMM_OK;
}

}  // namespace igemm
