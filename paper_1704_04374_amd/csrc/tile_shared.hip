// Kernel T instantiations: variant kShared (runs that share indices), fp32
// and fp64.
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_shared(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, kShared>(mode, hints, va, vb, block);
}

const void* tile_kernel_f64_shared(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<double, kShared>(mode, hints, va, vb, block);
}

}  // namespace hptt
