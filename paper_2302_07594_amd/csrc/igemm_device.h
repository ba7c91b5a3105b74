// Device helpers shared by the fused tiled kernels, the packing kernels and
// the packed-operand kernel: vector types, the two gfx950 int8 matrix-core
// instruction shapes, the LDS swizzle, byte permutes and masks, the MFMA
// interleave pattern and element-wise bounded loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace igemm {


typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned int u32;

// The two gfx950 int8 matrix-core instructions, described by their tile
// shape. Both take 16 bytes of A and 16 bytes of B per lane (one row of A /
// one column of B, k-contiguous); the k range a lane holds is chunk
// `2*ks + lane/32` (32x32x32) or `lane/16` (16x16x64) of the 64-byte k-tile.
// 32x32x32 is the default: the compiler accumulates it in place, whereas it
// rotates the 16x16x64 accumulators through copies, so 16x16x64 is kept for
// 16-row tiles only.
template <int MF>
struct Mfma;
template <>
struct Mfma<16> {
    typedef v4i acc_t;
    static constexpr int REGS = 4, KSTEPS = 1;
    static __device__ __forceinline__ acc_t mma(v4i a, v4i b, acc_t c) {
        return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int frag_row(int lane) { return lane & 15; }
    static __device__ __forceinline__ int frag_chunk(int lane, int ks) { return lane >> 4; }
    // output register r of `lane` holds C[row][col] of the 16x16 tile
    static __device__ __forceinline__ int out_row(int lane, int r) { return 4 * (lane >> 4) + r; }
    static __device__ __forceinline__ int out_col(int lane) { return lane & 15; }
};
template <>
struct Mfma<32> {
    typedef v16i acc_t;
    static constexpr int REGS = 16, KSTEPS = 2;
    static __device__ __forceinline__ acc_t mma(v4i a, v4i b, acc_t c) {
        return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int frag_row(int lane) { return lane & 31; }
    static __device__ __forceinline__ int frag_chunk(int lane, int ks) { return 2 * ks + (lane >> 5); }
    static __device__ __forceinline__ int out_row(int lane, int r) {
        return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    }
    static __device__ __forceinline__ int out_col(int lane) { return lane & 31; }
};

// ---------------------------------------------------------------------------
// LDS layout. Every operand plane is stored as rows of 64 bytes (the 64
// k-elements of one row of A or one column of B), split into four 16-byte
// chunks; chunk q of row r sits at position q ^ swz(r). With
// swz(r) = ((r >> 1) ^ (r >> 2)) & 3 the fragment reads of both MFMA shapes
// (16 or 32 consecutive rows at one chunk) are free of bank conflicts on
// gfx950's 64-bank LDS (measured: ~200 B/clk/CU, against ~110 for the
// 2-way-conflicted (r >> 1) & 3).
__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 2)) & 3; }
__device__ __forceinline__ int lds_off(int row, int q) { return row * 64 + ((q ^ swz(row)) << 4); }

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

// Instruction interleaving for one pipelined k sub-step (a scheduling
// region). With one wave per SIMD the matrix core only stays busy if every
// other instruction is issued between MFMAs, so the region is laid out as
// NM slots, each one MFMA preceded by a fragment read (first NR slots) and
// followed by global loads, VALU work and LDS writes.
// Group masks: 0x008 MFMA, 0x100 LDS read, 0x200 LDS write, 0x020 global
// read, 0x002 VALU.
template <int NM, int NR, int NV, int VALU_PER, int DSW_PER>
__device__ __forceinline__ void interleave() {
#pragma unroll
    for (int i = 0; i < NM; ++i) {
        if (i < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        if (VALU_PER > 0) __builtin_amdgcn_sched_group_barrier(0x002, VALU_PER, 0);
        if (DSW_PER > 0) __builtin_amdgcn_sched_group_barrier(0x200, DSW_PER, 0);
    }
}

// Element-wise load of 16 bytes (16 int8 or 8 int16 elements) starting at
// element e0 of a row with `len` valid elements; invalid elements are zero.
template <int ES>
__device__ __forceinline__ v4i load_elems(const void *rowp, int e0, int len) {
    u32 w[4] = {0u, 0u, 0u, 0u};
    if constexpr (ES == 1) {
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

template <int V>
using ic = std::integral_constant<int, V>;

}  // namespace igemm
