// Device half of the C ABI: the gfx950 kernels and hptt_exec.
//
// Each kernel is a thin __global__ wrapper around the phase functions of
// kernel_body.h, instantiated for the element type, the vector widths of the
// A and B accesses, the update mode of Eq. (1) and the store hint.
#include <hip/hip_runtime.h>

#include "kernel_body.h"
#include "plan.h"

namespace hptt {
namespace {

thread_local int32_t g_last_hip_error = 0;

// Plain global and LDS accesses.  A vector of V elements is one
// global_load/store of V*sizeof(T) bytes; the plan only asks for widths that
// keep every such access aligned.
struct DeviceMem {
    template <typename T, int V, bool NT>
    __device__ __forceinline__ static Vec<T, V> ld(const T* p, int64_t off) {
        Vec<T, V> r;
        if constexpr (V == 1) {
            r.v[0] = NT ? __builtin_nontemporal_load(p + off) : p[off];
        } else {
            typedef T vt __attribute__((ext_vector_type(V)));
            const vt x = NT ? __builtin_nontemporal_load(reinterpret_cast<const vt*>(p + off))
                            : *reinterpret_cast<const vt*>(p + off);
#pragma unroll
            for (int e = 0; e < V; ++e) r.v[e] = x[e];
        }
        return r;
    }
    template <typename T>
    __device__ __forceinline__ static T ld1(const T* p, int64_t off) {
        return p[off];
    }
    template <bool NT, typename T>
    __device__ __forceinline__ static void st1(T* p, int64_t off, T v) {
        if constexpr (NT) __builtin_nontemporal_store(v, p + off);
        else p[off] = v;
    }
    template <bool NT, typename T, int V>
    __device__ __forceinline__ static void st(T* p, int64_t off, const Vec<T, V>& v) {
        if constexpr (V == 1) {
            st1<NT, T>(p, off, v.v[0]);
        } else {
            typedef T vt __attribute__((ext_vector_type(V)));
            vt x;
#pragma unroll
            for (int e = 0; e < V; ++e) x[e] = v.v[e];
            if constexpr (NT) __builtin_nontemporal_store(x, reinterpret_cast<vt*>(p + off));
            else *reinterpret_cast<vt*>(p + off) = x;
        }
    }
    template <typename T>
    __device__ __forceinline__ static T lds_ld(const T* l, int64_t i) {
        return l[i];
    }
    template <typename T>
    __device__ __forceinline__ static void lds_st(T* l, int64_t i, T v) {
        l[i] = v;
    }
};

template <typename T, int VA, int VB, int MODE, int HINT>
__global__ __launch_bounds__(kBlock) void tile_kernel(const T* __restrict__ A, T* __restrict__ B,
                                                      const TileArgs g, T alpha, T beta) {
    extern __shared__ int64_t smem[];
    int64_t* rowOffA = smem;
    int64_t* colOffB = smem + g.runB;
    T* lds = reinterpret_cast<T*>(colOffB + g.runA);
    const int tid = int(threadIdx.x);
    tile_tables<DeviceMem>(g, tid, rowOffA, colOffB);
    __syncthreads();
    bool first = true;
    for (uint32_t t = blockIdx.x; t < g.numTiles; t += gridDim.x) {
        const TileBase tb = tile_base(g, t);
        for (int64_t r0 = 0; r0 < tb.validRows; r0 += g.subRows) {
            if (!first) __syncthreads();  // the previous pass's LDS reads are done
            first = false;
            tile_load<DeviceMem, T, VA, HINT>(g, tb, r0, tid, A, lds, rowOffA);
            __syncthreads();
            tile_store<DeviceMem, T, VB, MODE, HINT>(g, tb, r0, tid, B, lds, colOffB, alpha, beta);
        }
    }
}

template <typename T, int V, int MODE, int HINT>
__global__ __launch_bounds__(kBlock) void stream_kernel(const T* __restrict__ A,
                                                        T* __restrict__ B, const StreamArgs g,
                                                        T alpha, T beta) {
    const uint64_t step = uint64_t(gridDim.x) * kBlock * kItems;
    const uint64_t items = g.numItems[log2_width(V)];
    for (uint64_t first = uint64_t(blockIdx.x) * kBlock * kItems; first < items; first += step)
        stream_items<DeviceMem, T, V, MODE, HINT>(g, uint32_t(first), int(threadIdx.x), A, B, alpha,
                                                  beta);
}

template <typename T, int V, int MODE, int HINT>
__global__ __launch_bounds__(kBlock) void axpby_kernel(const T* __restrict__ A,
                                                       T* __restrict__ B, const int64_t numel,
                                                       T alpha, T beta) {
    const int64_t vecs = (numel + V - 1) / V;
    const int64_t step = int64_t(gridDim.x) * kBlock * kItems;
    for (int64_t first = int64_t(blockIdx.x) * kBlock * kItems; first < vecs; first += step)
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

template <typename T>
constexpr int kMaxVec = int(16 / sizeof(T));

template <typename T, int VA, int MODE, int HINT>
const void* tile_fn_vb(int vb) {
    switch (vb) {
        case 1: return reinterpret_cast<const void*>(&tile_kernel<T, VA, 1, MODE, HINT>);
        case 2: return reinterpret_cast<const void*>(&tile_kernel<T, VA, 2, MODE, HINT>);
        case 4:
            if constexpr (kMaxVec<T> >= 4)
                return reinterpret_cast<const void*>(&tile_kernel<T, VA, 4, MODE, HINT>);
            return nullptr;
    }
    return nullptr;
}

template <typename T, int MODE, int HINT>
const void* tile_fn(int va, int vb) {
    switch (va) {
        case 1: return tile_fn_vb<T, 1, MODE, HINT>(vb);
        case 2: return tile_fn_vb<T, 2, MODE, HINT>(vb);
        case 4:
            if constexpr (kMaxVec<T> >= 4) return tile_fn_vb<T, 4, MODE, HINT>(vb);
            return nullptr;
    }
    return nullptr;
}

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

// Kernel address for the plan's class, with the given vector widths.
template <typename T, int MODE, int HINT>
const void* select(const hptt_plan_s* p, int va, int vb) {
    switch (p->info.kernel) {
        case HPTT_KERNEL_TILE: return tile_fn<T, MODE, HINT>(va, vb);
        case HPTT_KERNEL_STREAM: return stream_fn<T, MODE, HINT>(va < vb ? va : vb);
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
    }
    const void* fn = select_mode<T>(p, va, vb);
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
            args[2] = const_cast<StreamArgs*>(&p->stream);
            lds = size_t(in.lds_bytes);
            break;
        case HPTT_KERNEL_AXPBY: args[2] = &numel; break;
        case HPTT_KERNEL_GENERIC: args[2] = const_cast<GenericArgs*>(&p->generic); break;
        default: return HPTT_ERROR_INVALID_ARGUMENT;
    }
    hipError_t err = hipLaunchKernel(fn, dim3(uint32_t(in.grid)), dim3(kBlock), args, lds, stream);
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

}  // extern "C"
