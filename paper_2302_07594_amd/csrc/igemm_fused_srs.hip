// Instantiations of the fused kernel: int16-output update (shift-round-saturate
// conversion of Sec. 5.2), int16 and int8 operands, the small-tile shapes.
#include "igemm_tiled.h"

namespace igemm {

const void *fused_srs(int id, bool va, bool vb) {
    switch (id) {
        case K_I16_128x128: return pick_srs<2, 128, 128, 64, 64, 32>(va, vb);
        case K_I16_64x64: return pick_srs<2, 64, 64, 32, 32, 32>(va, vb);
        case K_I16_32x128: return pick_srs<2, 32, 128, 32, 32, 32>(va, vb);
        case K_I16_16x128: return pick_srs<2, 16, 128, 16, 32, 16>(va, vb);
        case K_I8_32x256: return pick_srs<1, 32, 256, 32, 64, 32>(va, vb);
        case K_I8_16x256: return pick_srs<1, 16, 256, 16, 64, 16>(va, vb);
        default: return nullptr;
    }
}

}  // namespace igemm
