// Device helpers of the kernels that move raw row-major operand tiles into
// LDS unchanged (the direct and the small-output kernels): the global -> LDS
// DMA load, the gfx950 transpose reads that turn row-major B in LDS into
// k-contiguous matrix-core operands, and the int16 limb split in registers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "igemm_device.h"

namespace igemm {
namespace lds {

typedef __attribute__((address_space(3))) void lds_void;
typedef short v2s __attribute__((ext_vector_type(2)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) v2i lds_v2i;

// 16 bytes per lane from global memory straight into LDS
// (global_load_lds_dwordx4): lane i of the wave writes bytes [16 i, 16 i + 16)
// after the wave-uniform LDS address.
__device__ __forceinline__ void dma16(const void *g, lds_void *lds) {
    __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}

// Transpose reads (gfx950). Within each group of 16 lanes, lane t receives
// element t % 4 (tr16) or byte t % 8 (tr8) of the 8-byte vectors that lanes
// t / 4 + 4 j (tr16, j < 4) or t / 8 + 2 j (tr8, j < 8) of its group address,
// in order of j (measured on the device).
__device__ __forceinline__ v2i tr16(const char *p) {
    const v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(lds_void *)p);
    return __builtin_bit_cast(v2i, r);
}
__device__ __forceinline__ v2i tr8(const char *p) {
    return __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i *)(lds_void *)p);
}

// acc + the two int16 halves of x (v_dot2 with ones).
__device__ __forceinline__ int sum2(u32 x, int acc) {
    return __builtin_amdgcn_sdot2(__builtin_bit_cast(v2s, x), v2s{1, 1}, acc, false);
}

// Four int16 pairs (w0 holds elements 0, 1; w1 elements 2, 3) -> the high
// limbs and the offset low limbs of the four elements, one byte each.
__device__ __forceinline__ u32 hi4(u32 w1, u32 w0) { return perm(w1, w0, 0x07050301u); }
__device__ __forceinline__ u32 lo4(u32 w1, u32 w0) {
    return perm(w1, w0, 0x06040200u) ^ 0x80808080u;
}

__device__ __forceinline__ v4i v4(u32 a, u32 b, u32 c, u32 d) {
    v4i r;
    r.x = (int)a;
    r.y = (int)b;
    r.z = (int)c;
    r.w = (int)d;
    return r;
}

}  // namespace lds
}  // namespace igemm
