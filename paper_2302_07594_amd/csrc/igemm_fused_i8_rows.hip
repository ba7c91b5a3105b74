// Instantiations of the fused kernel: GEMM, int8 operands, 32- and 16-row tiles.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_i8_rows(int id, bool va, bool vb, bool split) {
    switch (id) {
        case K_I8_32x256: return pick<1, 32, 256, 32, 64, 32>(va, vb, split);
        case K_I8_16x256: return pick<1, 16, 256, 16, 64, 16>(va, vb, split);
        default: return nullptr;
    }
}

}  // namespace igemm
