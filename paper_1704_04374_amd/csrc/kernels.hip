// Device half of the C ABI: the streaming, axpby and generic gfx950 kernels,
// and hptt_exec.
//
// Each kernel is a thin __global__ wrapper around the phase functions of
// kernel_body.h, instantiated for the element type, the vector widths of the
// A and B accesses, the update mode of Eq. (1) and the cache hints.  The
// tile kernel (tile_kernel.h) is instantiated in tile_*.hip.
#include <hip/hip_runtime.h>

#include "device_mem.h"
#include "plan.h"
#include "tile_kernel.h"

namespace hptt {
namespace {

thread_local int32_t g_last_hip_error = 0;

template <typename T, int V, int MODE, int HINT>
__global__ __launch_bounds__(kBlock) void stream_kernel(const T* __restrict__ A,
                                                        T* __restrict__ B, const StreamArgs g,
                                                        T alpha, T beta) {
    constexpr uint64_t per = uint64_t(kBlock) * items_per_lane(int(sizeof(T)), V);
    const uint64_t step = uint64_t(gridDim.x) * per;
    const uint64_t items = g.numItems[log2_width(V)];
    const uint32_t blk = g.xcdGroupLog ? xcd_group_map(blockIdx.x, gridDim.x, uint32_t(g.xcdGroupLog))
                                       : blockIdx.x;
    if (g.flatB) {
        for (uint64_t first = uint64_t(blk) * per; first < items; first += step)
            stream_items_flat<DeviceMem, T, V, MODE, HINT>(g, uint32_t(first), int(threadIdx.x), A,
                                                           B, alpha, beta);
        return;
    }
    for (uint64_t first = uint64_t(blk) * per; first < items; first += step)
        stream_items<DeviceMem, T, V, MODE, HINT>(g, uint32_t(first), int(threadIdx.x), A, B, alpha,
                                                  beta);
}

template <typename T, int V, int MODE, int HINT>
__global__ __launch_bounds__(kBlock) void axpby_kernel(const T* __restrict__ A,
                                                       T* __restrict__ B, const int64_t numel,
                                                       T alpha, T beta) {
    constexpr int64_t per = int64_t(kBlock) * items_per_lane(int(sizeof(T)), V);
    const int64_t vecs = (numel + V - 1) / V;
    const int64_t step = int64_t(gridDim.x) * per;
    for (int64_t first = int64_t(blockIdx.x) * per; first < vecs; first += step)
        axpby_items<DeviceMem, T, V, MODE, HINT>(numel, first, int(threadIdx.x), A, B, alpha, beta);
}

template <typename T, int MODE, int HINT, bool BIG>
__global__ __launch_bounds__(kBlock) void generic_kernel(const T* __restrict__ A,
                                                         T* __restrict__ B, const GenericArgs g,
                                                         T alpha, T beta) {
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    for (int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x; e < g.numel; e += stride)
        generic_elem<DeviceMem, T, MODE, HINT, BIG>(g, e, A, B, alpha, beta);
}

// ---------------------------------------------------------------------------
// Template selection: (mode, store hint) x vector widths -> kernel address
// ---------------------------------------------------------------------------

template <typename T, int MODE, int HINT>
const void* stream_fn(int v) {
    switch (v) {
        case 1: return reinterpret_cast<const void*>(&stream_kernel<T, 1, MODE, HINT>);
        case 2: return reinterpret_cast<const void*>(&stream_kernel<T, 2, MODE, HINT>);
        case 4:
            if constexpr (kMaxVec<T> >= 4)
                return reinterpret_cast<const void*>(&stream_kernel<T, 4, MODE, HINT>);
            return nullptr;
    }
    return nullptr;
}

template <typename T, int MODE, int HINT>
const void* axpby_fn(int v) {
    switch (v) {
        case 1: return reinterpret_cast<const void*>(&axpby_kernel<T, 1, MODE, HINT>);
        case 2: return reinterpret_cast<const void*>(&axpby_kernel<T, 2, MODE, HINT>);
        case 4:
            if constexpr (kMaxVec<T> >= 4)
                return reinterpret_cast<const void*>(&axpby_kernel<T, 4, MODE, HINT>);
            return nullptr;
    }
    return nullptr;
}

template <typename T, int MODE, int HINT>
const void* generic_fn(bool big) {
    return big ? reinterpret_cast<const void*>(&generic_kernel<T, MODE, HINT, true>)
               : reinterpret_cast<const void*>(&generic_kernel<T, MODE, HINT, false>);
}

// Kernel address for the plan's class, with the given vector widths (the
// tile kernel is picked by launch()).
template <typename T, int MODE, int HINT>
const void* select(const hptt_plan_s* p, int va, int vb) {
    switch (p->info.kernel) {
        // the flat walk reads A element by element: only B's width counts
        case HPTT_KERNEL_STREAM:
            return stream_fn<T, MODE, HINT>(p->stream.flatB || va >= vb ? vb : va);
        case HPTT_KERNEL_AXPBY: return axpby_fn<T, MODE, HINT>(va < vb ? va : vb);
        case HPTT_KERNEL_GENERIC:
            return generic_fn<T, MODE, HINT>(p->generic.numel >= (int64_t(1) << 32));
        default: return nullptr;
    }
}

template <typename T, int MODE>
const void* select_hint(const hptt_plan_s* p, int va, int vb) {
    switch (p->info.hints) {
        case 0: return select<T, MODE, 0>(p, va, vb);
        case kNtStore: return select<T, MODE, kNtStore>(p, va, vb);
        case kNtLoad: return select<T, MODE, kNtLoad>(p, va, vb);
        default: return select<T, MODE, kNtStore | kNtLoad>(p, va, vb);
    }
}

template <typename T>
const void* select_mode(const hptt_plan_s* p, int va, int vb) {
    switch (p->info.mode) {
        case kCopy: return select_hint<T, kCopy>(p, va, vb);
        case kScale: return select_hint<T, kScale>(p, va, vb);
        default: return select_hint<T, kAxpby>(p, va, vb);
    }
}

// Widest vector width <= v whose accesses stay aligned for this base pointer.
int aligned_width(int v, uintptr_t ptr, int elem) {
    while (v > 1 && ptr % uintptr_t(v * elem) != 0) v /= 2;
    return v;
}

// Kernel S over more than 2^32 items at width v: one launch per slab
// (stream_slabs_of), each with the slab's base pointers and arguments.
template <typename T>
hptt_status_t stream_slabs(const hptt_plan_s* p, const void* fn, const T* A, T* B, int v,
                           T alpha, T beta, hipStream_t stream) {
    const StreamSlabs s = stream_slabs_of(p->stream, v);
    const int64_t per = int64_t(kBlock) * items_per_lane(int(sizeof(T)), v);
    for (int64_t sl = 0; sl < s.count; ++sl) {
        int64_t offA = 0, offB = 0;
        StreamArgs sa = stream_slab_args(p->stream, s, sl, v, &offA, &offB);
        int64_t grid = (int64_t(sa.numItems[log2_width(v)]) + per - 1) / per;
        if (grid > p->info.grid) grid = p->info.grid;
        const T* a = A + offA;
        T* b = B + offB;
        void* args[5] = {&a, &b, &sa, &alpha, &beta};
        const hipError_t err =
            hipLaunchKernel(fn, dim3(uint32_t(grid)), dim3(kBlock), args, 0, stream);
        if (err != hipSuccess) {
            g_last_hip_error = int32_t(err);
            return HPTT_ERROR_HIP;
        }
    }
    return HPTT_SUCCESS;
}

template <typename T>
hptt_status_t launch(const hptt_plan_s* p, const void* A, void* B, hipStream_t stream) {
    const hptt_plan_info_t& in = p->info;
    const int elem = int(sizeof(T));
    const uintptr_t pa = reinterpret_cast<uintptr_t>(A), pb = reinterpret_cast<uintptr_t>(B);
    // The tile kernel keeps its widths and shifts its runs onto the vector
    // grid of the actual pointers; the others narrow to the pointers' alignment.
    const bool tile = in.kernel == HPTT_KERNEL_TILE;
    const int va = tile ? in.vec_a : aligned_width(in.vec_a, pa, elem);
    const int vb = tile ? in.vec_b : aligned_width(in.vec_b, pb, elem);
    TileArgs targs;
    if (tile) {
        targs = p->tile;
        targs.misA = int32_t((pa / uintptr_t(elem)) % uintptr_t(va));
        targs.misB = int32_t((pb / uintptr_t(elem)) % uintptr_t(vb));
        if (targs.shear) targs.misLineB = int32_t((pb / uintptr_t(elem)) % uintptr_t(targs.lineB));
    }
    const void* fn = nullptr;
    int block = kBlock;
    if (tile) {
        // only the kFast variant takes the plan's workgroup size
        const int variant = tile_variant(targs);
        block = variant == kFast ? in.block : kBlock;
        // Runs that are whole lines relative to the tensors' first elements
        // are not whole lines in memory when those are not on a line: lines
        // are then shared between tiles, so no non-temporal hint (see the
        // plan builder).
        int hints = in.hints;
        if (pb % 128 != 0) hints &= ~kNtStore;
        if (pa % 128 != 0) hints &= ~kNtLoad;
        fn = sizeof(T) == 4 ? tile_kernel_f32(variant, in.mode, hints, va, vb, block)
                            : tile_kernel_f64(variant, in.mode, hints, va, vb, block);
    } else {
        fn = select_mode<T>(p, va, vb);
    }
    if (!fn) return HPTT_ERROR_INVALID_ARGUMENT;
    const T* a = static_cast<const T*>(A);
    T* b = static_cast<T*>(B);
    T alpha = T(p->alpha), beta = T(p->beta);
    size_t lds = 0;
    void* args[5] = {&a, &b, nullptr, &alpha, &beta};
    int64_t numel = in.numel;
    switch (in.kernel) {
        case HPTT_KERNEL_TILE:
            args[2] = &targs;
            lds = size_t(in.lds_bytes);
            break;
        case HPTT_KERNEL_STREAM:
            if (!p->stream.flatB) {
                // the width the row walk launches with (as select() picks it)
                const int v = va >= vb ? vb : va;
                if (p->stream.numItems[log2_width(v)] == 0)
                    return stream_slabs<T>(p, fn, a, b, v, alpha, beta, stream);
            }
            args[2] = const_cast<StreamArgs*>(&p->stream);
            lds = size_t(in.lds_bytes);
            break;
        case HPTT_KERNEL_AXPBY: args[2] = &numel; break;
        case HPTT_KERNEL_GENERIC: args[2] = const_cast<GenericArgs*>(&p->generic); break;
        default: return HPTT_ERROR_INVALID_ARGUMENT;
    }
    hipError_t err = hipSuccess;
    if (lds > 64 * 1024)  // gfx950 has 160 KiB of LDS per CU; above 64 KiB it must be asked for
        err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (err == hipSuccess)
        err = hipLaunchKernel(fn, dim3(uint32_t(in.grid)), dim3(block), args, lds, stream);
    if (err != hipSuccess) {
        g_last_hip_error = int32_t(err);
        return HPTT_ERROR_HIP;
    }
    return HPTT_SUCCESS;
}

}  // namespace
}  // namespace hptt

extern "C" {

hptt_status_t hptt_exec(hptt_plan_t plan, const void* A, void* B, hipStream_t stream) {
    if (!plan) return HPTT_ERROR_INVALID_ARGUMENT;
    const hptt_plan_info_t& in = plan->info;
    if (in.kernel == HPTT_KERNEL_NONE || in.numel == 0) return HPTT_SUCCESS;
    if (!A || !B) return HPTT_ERROR_INVALID_ARGUMENT;
    const uintptr_t a = reinterpret_cast<uintptr_t>(A), b = reinterpret_cast<uintptr_t>(B);
    const uintptr_t elem = uintptr_t(in.elem_bytes);
    if (a % elem != 0 || b % elem != 0) return HPTT_ERROR_INVALID_ARGUMENT;
    const uintptr_t bytesA = uintptr_t(in.footprint_a) * elem;
    const uintptr_t bytesB = uintptr_t(in.footprint_b) * elem;
    if (a < b + bytesB && b < a + bytesA) return HPTT_ERROR_OVERLAP;
    if (plan->dtype == HPTT_FLOAT32) return hptt::launch<float>(plan, A, B, stream);
    return hptt::launch<double>(plan, A, B, stream);
}

int32_t hptt_last_hip_error(void) { return hptt::g_last_hip_error; }

hptt_status_t hptt_load_kernels(void) {
    using namespace hptt;
    // one kernel of each source file: each file's kernels are one code object
    const void* fns[] = {tile_kernel_f32(kFast, kCopy, 0, 1, 1, kBlock),
                         tile_kernel_f32(kShifted, kCopy, 0, 1, 1, kBlock),
                         tile_kernel_f32(kGeneral, kCopy, 0, 1, 1, kBlock),
                         tile_kernel_f32(kShared, kCopy, 0, 1, 1, kBlock),
                         tile_kernel_f64(kFast, kCopy, 0, 1, 1, kBlock),
                         stream_fn<float, kCopy, 0>(1)};
    for (const void* f : fns) {
        if (!f) continue;
        hipFuncAttributes attr;
        const hipError_t err = hipFuncGetAttributes(&attr, f);
        if (err != hipSuccess) {
            g_last_hip_error = int32_t(err);
            return HPTT_ERROR_HIP;
        }
    }
    return HPTT_SUCCESS;
}

}  // extern "C"
