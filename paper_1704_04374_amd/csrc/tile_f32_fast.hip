// Kernel T instantiations: fp32, specialised variant (runs on the vector grid, no stacking).
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_fast(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, false>(mode, hints, va, vb, block);
}

}  // namespace hptt
