// Kernel T instantiations: fp32, variant kGeneral (stacked tiles, sheared B runs, 64-bit offsets).
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_general(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, kGeneral>(mode, hints, va, vb, block);
}

}  // namespace hptt
