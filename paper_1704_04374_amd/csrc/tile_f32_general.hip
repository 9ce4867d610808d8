// Kernel T instantiations: fp32, general variant (shifted runs, stacked tiles).
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_general(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, true>(mode, hints, va, vb, block);
}

}  // namespace hptt
