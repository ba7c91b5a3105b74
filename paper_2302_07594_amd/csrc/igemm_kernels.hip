// Integer GEMM C += A B on gfx950 (CDNA4) int8 matrix cores.
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
//   * each wave keeps its C tile in accumulator registers and runs
//     v_mfma_i32_16x16x64_i8 over the k-tile (loop L6: rank-64 updates
//     instead of rank-1);
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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm.h"
#include "igemm_internal.h"

namespace igemm {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned int u32;

// ---------------------------------------------------------------------------
// LDS layout. Every operand plane is stored as rows of 64 bytes (the 64
// k-elements of one row of A or one column of B), split into four 16-byte
// chunks. The chunk index is XORed with bits 1-2 of the row, and for B the
// row parity is flipped by bit 4 of the row, so that (i) eight consecutive
// rows read at the same chunk -- one MFMA fragment load phase -- hit distinct
// banks, and (ii) the B staging writes of one wave spread over both halves of
// the banks.
__device__ __forceinline__ int lds_off_a(int row, int q) {
    return row * 64 + ((q ^ ((row >> 1) & 3)) << 4);
}
__device__ __forceinline__ int lds_off_b(int row, int q) {
    const int r = row ^ ((row >> 4) & 1);
    return r * 64 + ((q ^ ((r >> 1) & 3)) << 4);
}

__device__ __forceinline__ u32 perm(u32 hi, u32 lo, u32 sel) {
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// 4x4 byte transpose: x_r holds bytes (r, c = 0..3); y_c receives bytes
// (r = 0..3, c).
__device__ __forceinline__ void transpose4x4(u32 x0, u32 x1, u32 x2, u32 x3, u32 &y0,
                                             u32 &y1, u32 &y2, u32 &y3) {
    const u32 t0 = perm(x1, x0, 0x05010400u);
    const u32 t1 = perm(x1, x0, 0x07030602u);
    const u32 t2 = perm(x3, x2, 0x05010400u);
    const u32 t3 = perm(x3, x2, 0x07030602u);
    y0 = perm(t2, t0, 0x05040100u);
    y1 = perm(t2, t0, 0x07060302u);
    y2 = perm(t3, t1, 0x05040100u);
    y3 = perm(t3, t1, 0x07060302u);
}

__device__ __forceinline__ int sum4(u32 x, int acc) {
    return __builtin_amdgcn_sdot4((int)x, 0x01010101, acc, false);
}

// Byte mask keeping the first `v` bytes of a dword (v clamped to 0..4).
__device__ __forceinline__ u32 byte_mask(int v) {
    return v >= 4 ? 0xffffffffu : (v <= 0 ? 0u : ((1u << (8 * v)) - 1u));
}

// Element-wise load of 16 bytes (16 int8 or 8 int16 elements) starting at
// element e0 of a row with `len` valid elements; invalid elements are zero.
template <int ES>
__device__ __forceinline__ v4i load_elems(const void *rowp, int e0, int len) {
    u32 w[4] = {0u, 0u, 0u, 0u};
    if (ES == 1) {
        const uint8_t *p = (const uint8_t *)rowp;
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (e0 + i < len) w[i >> 2] |= (u32)p[e0 + i] << (8 * (i & 3));
    } else {
        const uint16_t *p = (const uint16_t *)rowp;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (e0 + i < len) w[i >> 1] |= (u32)p[e0 + i] << (16 * (i & 1));
    }
    v4i r;
    r.x = (int)w[0];
    r.y = (int)w[1];
    r.z = (int)w[2];
    r.w = (int)w[3];
    return r;
}

template <int ES, bool VEC>
__device__ __forceinline__ v4i load16(const void *rowp, int e0, int len) {
    constexpr int E = 16 / ES;
    if (VEC && e0 + E <= len)
        return *(const v4i *)((const char *)rowp + (size_t)e0 * ES);
    return load_elems<ES>(rowp, e0, len);
}

// ---------------------------------------------------------------------------
template <int ES, int BM, int BN, int WM, int WN, bool VA, bool VB, bool SPLIT>
__global__ void __launch_bounds__(256, 1)
igemm_tiled(const void *__restrict__ Ap, int64_t lda, const void *__restrict__ Bp,
            int64_t ldb, int32_t *__restrict__ C, int64_t ldc, int m, int n, int k,
            int kchunk, int tiles_m, int tiles_n) {
    constexpr int P = ES;                // limb planes per operand
    constexpr int NACC = ES == 2 ? 3 : 1;  // accumulator sets
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int WGN = BN / WN;
    static_assert((BM / WM) * WGN == 4, "four waves per workgroup");
    constexpr int APL = BM * 64, BPL = BN * 64;  // bytes per LDS plane
    constexpr int STAGE = P * (APL + BPL);
    constexpr int ACH = BM * 4 * ES;  // 16-byte A chunks per k-tile
    constexpr int ACT = (ACH + 255) / 256;
    constexpr int BUN = BN * ES;  // B units (4 rows x 16 bytes) per k-tile
    constexpr int BUT = (BUN + 255) / 256;
    constexpr int CPU = 16 / ES;  // columns per B unit
    static_assert(2 * STAGE >= 4 * 2 * (BM + BN), "LDS reuse for the limb sums");

    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

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
    const int ktiles = (kend - kbeg + 63) >> 6;

    const int8_t *A8 = (const int8_t *)Ap;
    const int8_t *B8 = (const int8_t *)Bp;

    v4i ra[ACT];
    v4i rb[BUT][4];
    int sah[ACT], sal[ACT];
    int sbh[BUT][8], sbl[BUT][8];
#pragma unroll
    for (int s = 0; s < ACT; ++s) sah[s] = sal[s] = 0;
#pragma unroll
    for (int s = 0; s < BUT; ++s)
#pragma unroll
        for (int c = 0; c < 8; ++c) sbh[s][c] = sbl[s][c] = 0;

    v4i acc[NACC][TM][TN];
#pragma unroll
    for (int a = 0; a < NACC; ++a)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[a][i][j] = v4i{0, 0, 0, 0};

    // ---- global -> registers ------------------------------------------------
    auto load_tile = [&](int k0) {
        const int klen = kend - k0;
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            const int c = tid + 256 * s;
            if (ACH % 256 == 0 || c < ACH) {
                const int row = c / (4 * ES), q = c % (4 * ES);
                const int gi = m0 + row;
                const int len = gi < m ? klen : 0;
                const int gic = gi < m ? gi : m - 1;
                const void *rowp = A8 + ((int64_t)gic * lda + k0) * ES;
                ra[s] = load16<ES, VA>(rowp, q * (16 / ES), len);
            }
        }
        const int nlen = n - n0;
#pragma unroll
        for (int s = 0; s < BUT; ++s) {
            const int u = tid + 256 * s;
            if (BUN % 256 == 0 || u < BUN) {
                const int rg = u & 15, cc = u >> 4;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int p = k0 + 4 * rg + r;
                    const int len = p < kend ? nlen : 0;
                    const int pc = p < kend ? p : kend - 1;
                    const void *rowp = B8 + ((int64_t)pc * ldb + n0) * ES;
                    rb[s][r] = load16<ES, VB>(rowp, cc * CPU, len);
                }
            }
        }
    };

    // ---- registers -> LDS (limb split, B transpose, limb sums) ------------
    auto store_tile = [&](int buf, int k0) {
        char *As = smem + buf * STAGE;
        char *Bs = As + P * APL;
        const bool ktail = k0 + 64 > kend;
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            const int c = tid + 256 * s;
            if (ACH % 256 == 0 || c < ACH) {
                const int row = c / (4 * ES), q = c % (4 * ES);
                if (ES == 1) {
                    *(v4i *)(As + lds_off_a(row, q)) = ra[s];
                } else {
                    const u32 y0 = ra[s].x, y1 = ra[s].y, y2 = ra[s].z, y3 = ra[s].w;
                    u32 h0 = perm(y1, y0, 0x07050301u), h1 = perm(y3, y2, 0x07050301u);
                    u32 l0 = perm(y1, y0, 0x06040200u) ^ 0x80808080u;
                    u32 l1 = perm(y3, y2, 0x06040200u) ^ 0x80808080u;
                    if (ktail) {
                        const int v = kend - k0 - q * 8;
                        const u32 m0k = byte_mask(v), m1k = byte_mask(v - 4);
                        h0 &= m0k;
                        l0 &= m0k;
                        h1 &= m1k;
                        l1 &= m1k;
                    }
                    sah[s] = sum4(h1, sum4(h0, sah[s]));
                    sal[s] = sum4(l1, sum4(l0, sal[s]));
                    const int off = lds_off_a(row, q >> 1) + ((q & 1) << 3);
                    *(uint2 *)(As + off) = make_uint2(h0, h1);
                    *(uint2 *)(As + APL + off) = make_uint2(l0, l1);
                }
            }
        }
#pragma unroll
        for (int s = 0; s < BUT; ++s) {
            const int u = tid + 256 * s;
            if (BUN % 256 == 0 || u < BUN) {
                const int rg = u & 15, cc = u >> 4;
                const int q = rg >> 2, sub = (rg & 3) << 2;
                u32 rmask = 0xffffffffu;
                if (ES == 2 && ktail) rmask = byte_mask(kend - (k0 + 4 * rg));
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    u32 y0, y1, y2, y3;
                    transpose4x4((u32)rb[s][0][d], (u32)rb[s][1][d], (u32)rb[s][2][d],
                                 (u32)rb[s][3][d], y0, y1, y2, y3);
                    if (ES == 1) {
                        const int col = cc * 16 + 4 * d;
                        *(u32 *)(Bs + lds_off_b(col + 0, q) + sub) = y0;
                        *(u32 *)(Bs + lds_off_b(col + 1, q) + sub) = y1;
                        *(u32 *)(Bs + lds_off_b(col + 2, q) + sub) = y2;
                        *(u32 *)(Bs + lds_off_b(col + 3, q) + sub) = y3;
                    } else {
                        // y0/y2: low bytes of columns 2d, 2d+1; y1/y3: high bytes.
                        const u32 la = (y0 ^ 0x80808080u) & rmask, ha = y1 & rmask;
                        const u32 lb = (y2 ^ 0x80808080u) & rmask, hb = y3 & rmask;
                        sbh[s][2 * d] = sum4(ha, sbh[s][2 * d]);
                        sbl[s][2 * d] = sum4(la, sbl[s][2 * d]);
                        sbh[s][2 * d + 1] = sum4(hb, sbh[s][2 * d + 1]);
                        sbl[s][2 * d + 1] = sum4(lb, sbl[s][2 * d + 1]);
                        const int col = cc * 8 + 2 * d;
                        const int oa = lds_off_b(col, q) + sub, ob = lds_off_b(col + 1, q) + sub;
                        *(u32 *)(Bs + oa) = ha;
                        *(u32 *)(Bs + BPL + oa) = la;
                        *(u32 *)(Bs + ob) = hb;
                        *(u32 *)(Bs + BPL + ob) = lb;
                    }
                }
            }
        }
    };

    // ---- MFMA over one k-tile ----------------------------------------------
    auto compute = [&](int buf) {
        const char *As = smem + buf * STAGE;
        const char *Bs = As + P * APL;
        const int fr = lane & 15, fq = lane >> 4;
        v4i af[P][TM], bf[P][TN];
#pragma unroll
        for (int p = 0; p < P; ++p) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[p][i] = *(const v4i *)(As + p * APL + lds_off_a(wm0 + 16 * i + fr, fq));
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bf[p][j] = *(const v4i *)(Bs + p * BPL + lds_off_b(wn0 + 16 * j + fr, fq));
        }
        if (ES == 1) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[0][i], bf[0][j],
                                                                         acc[0][i][j], 0, 0, 0);
        } else {
            // plane 0 = high limbs, plane 1 = offset low limbs
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[0][i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[0][i], bf[0][j],
                                                                         acc[0][i][j], 0, 0, 0);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[1][i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[0][i], bf[1][j],
                                                                         acc[1][i][j], 0, 0, 0);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[2][i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[1][i], bf[1][j],
                                                                         acc[2][i][j], 0, 0, 0);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[1][i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[1][i], bf[0][j],
                                                                         acc[1][i][j], 0, 0, 0);
        }
    };

    // ---- main loop: double-buffered LDS, next tile's loads in flight -------
    load_tile(kbeg);
    store_tile(0, kbeg);
    __syncthreads();
    for (int kt = 0; kt < ktiles; ++kt) {
        const bool more = kt + 1 < ktiles;
        const int knext = kbeg + (kt + 1) * 64;
        if (more) load_tile(knext);
        compute(kt & 1);
        if (more) store_tile((kt + 1) & 1, knext);
        __syncthreads();
    }

    // ---- epilogue -------------------------------------------------------------
    int *sRH = (int *)smem;
    int *sRL = sRH + BM;
    int *sKH = sRL + BM;
    int *sKL = sKH + BN;
    if (ES == 2) {
        for (int i = tid; i < 2 * (BM + BN); i += 256) sRH[i] = 0;
        __syncthreads();
#pragma unroll
        for (int s = 0; s < ACT; ++s) {
            const int c = tid + 256 * s;
            if (ACH % 256 == 0 || c < ACH) {
                const int row = c / 8;
                atomicAdd(&sRH[row], sah[s]);
                atomicAdd(&sRL[row], sal[s]);
            }
        }
#pragma unroll
        for (int s = 0; s < BUT; ++s) {
            const int u = tid + 256 * s;
            if (BUN % 256 == 0 || u < BUN) {
                const int cc = u >> 4;
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    atomicAdd(&sKH[cc * 8 + c], sbh[s][c]);
                    atomicAdd(&sKL[cc * 8 + c], sbl[s][c]);
                }
            }
        }
        __syncthreads();
    }
    const u32 kconst = 16384u * (u32)(kend - kbeg);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int lc = wn0 + 16 * j + (lane & 15);
            const int gc = n0 + lc;
            u32 colterm = 0;
            if (ES == 2) colterm = 32768u * (u32)sKH[lc] + 128u * (u32)sKL[lc] + kconst;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int lr = wm0 + 16 * i + 4 * (lane >> 4) + r;
                const int gr = m0 + lr;
                u32 v;
                if (ES == 1) {
                    v = (u32)acc[0][i][j][r];
                } else {
                    v = 65536u * (u32)acc[0][i][j][r] + 256u * (u32)acc[1][i][j][r] +
                        (u32)acc[2][i][j][r] + 32768u * (u32)sRH[lr] + 128u * (u32)sRL[lr] +
                        colterm;
                }
                if (gr < m && gc < n) {
                    int32_t *cp = C + (int64_t)gr * ldc + gc;
                    if (SPLIT)
                        atomicAdd(cp, (int)v);
                    else
                        *cp = (int32_t)((u32)*cp + v);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
template <int ES, int BM, int BN, int WM, int WN>
const void *pick(bool va, bool vb, bool split) {
#define IGEMM_K(a, b, s) (const void *)&igemm_tiled<ES, BM, BN, WM, WN, a, b, s>
    if (split) {
        if (va) return vb ? IGEMM_K(true, true, true) : IGEMM_K(true, false, true);
        return vb ? IGEMM_K(false, true, true) : IGEMM_K(false, false, true);
    }
    if (va) return vb ? IGEMM_K(true, true, false) : IGEMM_K(true, false, false);
    return vb ? IGEMM_K(false, true, false) : IGEMM_K(false, false, false);
#undef IGEMM_K
}

const void *kernel_fn(int id, bool va, bool vb, bool split) {
    switch (id) {
        case K_I8_256x256: return pick<1, 256, 256, 128, 128>(va, vb, split);
        case K_I8_128x128: return pick<1, 128, 128, 64, 64>(va, vb, split);
        case K_I8_32x256: return pick<1, 32, 256, 32, 64>(va, vb, split);
        case K_I8_16x256: return pick<1, 16, 256, 16, 64>(va, vb, split);
        case K_I16_128x128: return pick<2, 128, 128, 64, 64>(va, vb, split);
        case K_I16_64x64: return pick<2, 64, 64, 32, 32>(va, vb, split);
        case K_I16_32x128: return pick<2, 32, 128, 32, 32>(va, vb, split);
        case K_I16_16x128: return pick<2, 16, 128, 16, 32>(va, vb, split);
        default: return nullptr;
    }
}

int num_cu_of_current_device() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev >= 0 && dev < 64 && cached[dev] > 0) return cached[dev];
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cu <= 0)
        cu = 256;
    if (dev >= 0 && dev < 64) cached[dev] = cu;
    return cu;
}

int run(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda, const void *B,
        int64_t ldb, int32_t *C, int64_t ldc, void *stream, int kernel, int split) {
    int st = validate(es, m, n, k, A, lda, B, ldb, C, ldc);
    if (st != IGEMM_OK) return st;
    if (m == 0 || n == 0 || k == 0) return IGEMM_OK;
    if (kernel < -1 || kernel >= K_COUNT || split < -1 || split == 0) return IGEMM_EINVAL;
    if (kernel >= 0 && kKernels[kernel].es != es) return IGEMM_EINVAL;
    igemm_plan p;
    st = make_plan(es, m, n, k, A, lda, B, ldb, num_cu_of_current_device(), kernel, split, &p);
    if (st != IGEMM_OK) return st;
    const void *fn = kernel_fn(p.kernel, p.vec_a != 0, p.vec_b != 0, p.split > 1);
    if (fn == nullptr) return IGEMM_EINVAL;
    int mi = (int)m, ni = (int)n, ki = (int)k, kc = (int)p.k_chunk;
    int tm = (int)((m + p.bm - 1) / p.bm), tn = (int)((n + p.bn - 1) / p.bn);
    void *args[] = {(void *)&A, (void *)&lda, (void *)&B, (void *)&ldb, (void *)&C,
                    (void *)&ldc, (void *)&mi, (void *)&ni, (void *)&ki, (void *)&kc,
                    (void *)&tm, (void *)&tn};
    hipError_t e = hipLaunchKernel(fn, dim3((unsigned)p.grid), dim3(kThreads), args, 0,
                                   (hipStream_t)stream);
    return e == hipSuccess ? IGEMM_OK : IGEMM_EHIP;
}

}  // namespace
}  // namespace igemm

extern "C" {

int igemm_i16(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
              const int16_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream) {
    return igemm::run(2, m, n, k, A, lda, B, ldb, C, ldc, stream, -1, -1);
}

int igemm_i8(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda, const int8_t *B,
             int64_t ldb, int32_t *C, int64_t ldc, void *stream) {
    return igemm::run(1, m, n, k, A, lda, B, ldb, C, ldc, stream, -1, -1);
}

int igemm_i16_ex(int64_t m, int64_t n, int64_t k, const int16_t *A, int64_t lda,
                 const int16_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                 int kernel, int split) {
    return igemm::run(2, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split);
}

int igemm_i8_ex(int64_t m, int64_t n, int64_t k, const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb, int32_t *C, int64_t ldc, void *stream,
                int kernel, int split) {
    return igemm::run(1, m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split);
}

}  // extern "C"
