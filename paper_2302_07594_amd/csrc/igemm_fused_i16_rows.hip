// Instantiations of the fused kernel: GEMM, int16 operands, 32- and 16-row tiles.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_i16_rows(int id, bool va, bool vb, bool split) {
    switch (id) {
        case K_I16_32x128: return pick<2, 32, 128, 32, 32, 32>(va, vb, split);
        case K_I16_16x128: return pick<2, 16, 128, 16, 32, 16>(va, vb, split);
        default: return nullptr;
    }
}

}  // namespace igemm
