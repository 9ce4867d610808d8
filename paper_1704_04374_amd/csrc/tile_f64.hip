// Kernel T instantiations: fp64, both variants, and the fp32 dispatcher
// over tile_f32_fast.hip and tile_f32_general.hip.
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_fast(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_general(int mode, int hints, int va, int vb, int block);

const void* tile_kernel_f32(bool general, int mode, int hints, int va, int vb, int block) {
    return general ? tile_kernel_f32_general(mode, hints, va, vb, block)
                   : tile_kernel_f32_fast(mode, hints, va, vb, block);
}

const void* tile_kernel_f64(bool general, int mode, int hints, int va, int vb, int block) {
    return general ? tile_kernel_address<double, true>(mode, hints, va, vb, block)
                   : tile_kernel_address<double, false>(mode, hints, va, vb, block);
}

}  // namespace hptt
