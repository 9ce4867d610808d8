// Kernel T instantiations: fp64, all three variants, and the fp32
// dispatcher over tile_f32_fast.hip, tile_f32_shifted.hip and
// tile_f32_general.hip.
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_fast(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_shifted(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_general(int mode, int hints, int va, int vb, int block);

const void* tile_kernel_f32(int variant, int mode, int hints, int va, int vb, int block) {
    switch (variant) {
        case kFast: return tile_kernel_f32_fast(mode, hints, va, vb, block);
        case kShifted: return tile_kernel_f32_shifted(mode, hints, va, vb, block);
        default: return tile_kernel_f32_general(mode, hints, va, vb, block);
    }
}

const void* tile_kernel_f64(int variant, int mode, int hints, int va, int vb, int block) {
    switch (variant) {
        case kFast: return tile_kernel_address<double, kFast>(mode, hints, va, vb, block);
        case kShifted: return tile_kernel_address<double, kShifted>(mode, hints, va, vb, block);
        default: return tile_kernel_address<double, kGeneral>(mode, hints, va, vb, block);
    }
}

}  // namespace hptt
