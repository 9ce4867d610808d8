// Kernel T instantiations: fp32, variant kShifted (runs shifted onto the vector grid).
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_shifted(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, kShifted>(mode, hints, va, vb, block);
}

}  // namespace hptt
