// Instantiations of the fused kernel: convolution (IM2ROW gather), int16 operands, 64x64, 32x128
// and 16x128 tiles.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_conv_i16(int id, int gather, bool vb, bool split) {
    switch (id) {
        case K_I16_128x128: return pick_conv<2, 128, 128, 64, 64, 32>(gather, vb, split);
        case K_I16_64x64: return pick_conv<2, 64, 64, 32, 32, 32>(gather, vb, split);
        case K_I16_32x128: return pick_conv<2, 32, 128, 32, 32, 32>(gather, vb, split);
        case K_I16_16x128: return pick_conv<2, 16, 128, 16, 32, 16>(gather, vb, split);
        default: return nullptr;
    }
}

}  // namespace igemm
