// Kernel T instantiations: variant kDirect (A fetched straight into LDS),
// fp32 and fp64.
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_direct(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<float, kDirect>(mode, hints, va, vb, block);
}

const void* tile_kernel_f64_direct(int mode, int hints, int va, int vb, int block) {
    return tile_kernel_address<double, kDirect>(mode, hints, va, vb, block);
}

}  // namespace hptt
