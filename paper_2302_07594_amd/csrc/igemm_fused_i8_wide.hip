// Instantiations of the fused kernel: GEMM, int8 operands, 256x256 and 128x128 tiles.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_i8_wide(int id, bool va, bool vb, bool split) {
    switch (id) {
        case K_I8_256x256: return pick<1, 256, 256, 128, 128, 32>(va, vb, split);
        case K_I8_128x128: return pick<1, 128, 128, 64, 64, 32>(va, vb, split);
        default: return nullptr;
    }
}

}  // namespace igemm
