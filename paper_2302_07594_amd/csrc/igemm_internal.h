// Internal declarations shared by the host planner and the kernel launcher.
#pragma once

#include <stdint.h>

#include "igemm.h"

namespace igemm {

// One tiled kernel family: operand size, workgroup tile of C and the tile of
// C each of the four waves owns.
struct KernelDesc {
    const char *name;
    int es;      // operand bytes: 2 = int16 (two int8 limb planes), 1 = int8
    int bm, bn;  // workgroup tile of C
    int wm, wn;  // wave tile of C
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
    K_COUNT
};

constexpr int kBK = 64;        // k elements per k-tile (one 16x16x64 MFMA step)
constexpr int kThreads = 256;  // four waves of 64
// Largest k range one workgroup accumulates in int32 MFMA accumulators. Each
// int16 limb sum is bounded by 2^15 per k element (2^14 for int8), so partial
// sums stay below 2^31 and never depend on how the hardware treats overflow.
constexpr int64_t kMaxKChunk = 32768;

extern const KernelDesc kKernels[K_COUNT];

// Validation and planning; pure host code, no HIP calls.
int validate(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
             const void *B, int64_t ldb, const void *C, int64_t ldc);
int make_plan(int es, int64_t m, int64_t n, int64_t k, const void *A, int64_t lda,
              const void *B, int64_t ldb, int num_cu, int kernel, int split,
              igemm_plan *out);

}  // namespace igemm
