// Instantiations of the fused kernel: GEMM, int16 operands, 128x128 and 64x64 tiles.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_i16_wide(int id, bool va, bool vb, bool split) {
    switch (id) {
        case K_I16_128x128: return pick<2, 128, 128, 64, 64, 32>(va, vb, split);
        case K_I16_64x64: return pick<2, 64, 64, 32, 32, 32>(va, vb, split);
        default: return nullptr;
    }
}

}  // namespace igemm
