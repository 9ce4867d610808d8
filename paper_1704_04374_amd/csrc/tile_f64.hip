// Kernel T instantiations: fp64 in variants kFast, kShifted and kGeneral,
// and the dispatchers over them, tile_f32_fast.hip, tile_f32_shifted.hip,
// tile_f32_general.hip, tile_shared.hip and tile_direct.hip.
#include "tile_kernel.h"

namespace hptt {

const void* tile_kernel_f32_fast(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_shifted(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_general(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_shared(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f64_shared(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f32_direct(int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f64_direct(int mode, int hints, int va, int vb, int block);

const void* tile_kernel_f32(int variant, int mode, int hints, int va, int vb, int block) {
    switch (variant) {
        case kFast: return tile_kernel_f32_fast(mode, hints, va, vb, block);
        case kShifted: return tile_kernel_f32_shifted(mode, hints, va, vb, block);
        case kShared: return tile_kernel_f32_shared(mode, hints, va, vb, block);
        case kDirect: return tile_kernel_f32_direct(mode, hints, va, vb, block);
        default: return tile_kernel_f32_general(mode, hints, va, vb, block);
    }
}

const void* tile_kernel_f64(int variant, int mode, int hints, int va, int vb, int block) {
    switch (variant) {
        case kFast: return tile_kernel_address<double, kFast>(mode, hints, va, vb, block);
        case kShifted: return tile_kernel_address<double, kShifted>(mode, hints, va, vb, block);
        case kShared: return tile_kernel_f64_shared(mode, hints, va, vb, block);
        case kDirect: return tile_kernel_f64_direct(mode, hints, va, vb, block);
        default: return tile_kernel_address<double, kGeneral>(mode, hints, va, vb, block);
    }
}

}  // namespace hptt
