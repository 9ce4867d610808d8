// Kernel T instantiations: fp32, variant kFast (runs on the vector grid).
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_fast(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, kFast>(mode, hints, va, vb, block);
}

}  // namespace hptt
