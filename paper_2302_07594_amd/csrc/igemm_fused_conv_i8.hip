// Instantiations of the fused kernel: convolution (IM2ROW gather), int8 operands, 32x256 and
// 16x256 tiles.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_conv_i8(int id, int gather, bool vb, bool split) {
    switch (id) {
        case K_I8_32x256: return pick_conv<1, 32, 256, 32, 64, 32>(gather, vb, split);
        case K_I8_16x256: return pick_conv<1, 16, 256, 16, 64, 16>(gather, vb, split);
        default: return nullptr;
    }
}

}  // namespace igemm
