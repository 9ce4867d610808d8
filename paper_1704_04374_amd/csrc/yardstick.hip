// Measurement kernels: a 16-byte-per-lane streaming copy, an axpby, a fill
// and a read-only sweep.
#include <hip/hip_runtime.h>

#include "hptt_yardstick.h"

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;      // vectors per lane of the fill kernel
constexpr int kReadBlocks = 1024;

struct alignas(16) V16 {
    uint32_t w[4];
};

// One 16-byte vector per lane, a grid that covers the buffer once, and
// non-temporal loads and stores: the fastest plain copy among the unroll
// depths, grid shapes and cache hints tried on MI355X.
__global__ __launch_bounds__(kThreads) void copy_kernel(const V16* __restrict__ src,
                                                        V16* __restrict__ dst, size_t n) {
    typedef uint32_t v4 __attribute__((ext_vector_type(4)));
    const size_t i = size_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i < n) {
        const v4 x = __builtin_nontemporal_load(reinterpret_cast<const v4*>(src) + i);
        __builtin_nontemporal_store(x, reinterpret_cast<v4*>(dst) + i);
    }
}

__global__ __launch_bounds__(kThreads) void read_kernel(const V16* __restrict__ src, size_t n,
                                                        uint32_t* __restrict__ sink) {
    __shared__ uint32_t part[kThreads];
    uint32_t acc = 0;
    for (size_t i = size_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
         i += size_t(gridDim.x) * kThreads) {
        const V16 v = src[i];
        acc ^= v.w[0] ^ v.w[1] ^ v.w[2] ^ v.w[3];
    }
    part[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t x = 0;
        for (int t = 0; t < kThreads; ++t) x ^= part[t];
        sink[blockIdx.x] = x;
    }
}

__global__ __launch_bounds__(kThreads) void fill_kernel(V16* __restrict__ dst, size_t n,
                                                        uint32_t value) {
    const size_t i = size_t(blockIdx.x) * (kThreads * kUnroll) + threadIdx.x;
    V16 v = {{value, value, value, value}};
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (i + size_t(u) * kThreads < n) dst[i + size_t(u) * kThreads] = v;
}

template <typename T>
struct alignas(16) VT {
    T v[16 / sizeof(T)];
};

// y <- alpha*x + beta*y, one 16-byte vector per lane, every access with a
// non-temporal hint (each line is touched once: y's read line is written
// back by the same lane).
template <typename T>
__global__ __launch_bounds__(kThreads) void axpby_kernel(T alpha, const VT<T>* __restrict__ x,
                                                         T beta, VT<T>* __restrict__ y, size_t n) {
#pragma clang fp contract(off)
    constexpr int V = int(16 / sizeof(T));
    typedef T vt __attribute__((ext_vector_type(V)));
    const size_t i = size_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i < n) {
        const vt a = __builtin_nontemporal_load(reinterpret_cast<const vt*>(x) + i);
        const vt b = __builtin_nontemporal_load(reinterpret_cast<const vt*>(y) + i);
        vt c;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            T s = alpha * a[e];
            T t = beta * b[e];
            c[e] = s + t;
        }
        __builtin_nontemporal_store(c, reinterpret_cast<vt*>(y) + i);
    }
}

size_t blocks_for(size_t n16) {
    return (n16 + size_t(kThreads * kUnroll) - 1) / size_t(kThreads * kUnroll);
}

hptt_status_t check_launch() {
    return hipGetLastError() == hipSuccess ? HPTT_SUCCESS : HPTT_ERROR_HIP;
}

}  // namespace

extern "C" {

hptt_status_t hptt_yardstick_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
    if (!src || !dst || bytes % 16 || reinterpret_cast<uintptr_t>(src) % 16 ||
        reinterpret_cast<uintptr_t>(dst) % 16)
        return HPTT_ERROR_INVALID_ARGUMENT;
    const size_t n = bytes / 16;
    if (n == 0) return HPTT_SUCCESS;
    hipLaunchKernelGGL(copy_kernel, dim3(uint32_t((n + kThreads - 1) / kThreads)), dim3(kThreads),
                       0, stream, static_cast<const V16*>(src), static_cast<V16*>(dst), n);
    return check_launch();
}

hptt_status_t hptt_yardstick_read(const void* buf, size_t bytes, void* sink, hipStream_t stream) {
    if (!buf || !sink || bytes % 16 || reinterpret_cast<uintptr_t>(buf) % 16 ||
        reinterpret_cast<uintptr_t>(sink) % 4)
        return HPTT_ERROR_INVALID_ARGUMENT;
    const size_t n = bytes / 16;
    if (n == 0) return HPTT_SUCCESS;
    hipLaunchKernelGGL(read_kernel, dim3(kReadBlocks), dim3(kThreads), 0, stream,
                       static_cast<const V16*>(buf), n, static_cast<uint32_t*>(sink));
    return check_launch();
}

hptt_status_t hptt_yardstick_fill(void* buf, size_t bytes, uint32_t value, hipStream_t stream) {
    if (!buf || bytes % 16 || reinterpret_cast<uintptr_t>(buf) % 16)
        return HPTT_ERROR_INVALID_ARGUMENT;
    const size_t n = bytes / 16;
    if (n == 0) return HPTT_SUCCESS;
    hipLaunchKernelGGL(fill_kernel, dim3(uint32_t(blocks_for(n))), dim3(kThreads), 0, stream,
                       static_cast<V16*>(buf), n, value);
    return check_launch();
}

hptt_status_t hptt_yardstick_axpby(hptt_dtype_t dtype, double alpha, const void* x, double beta,
                                   void* y, size_t n, hipStream_t stream) {
    const size_t elem = dtype == HPTT_FLOAT32 ? 4 : 8;
    if ((dtype != HPTT_FLOAT32 && dtype != HPTT_FLOAT64) || !x || !y || (n * elem) % 16 ||
        reinterpret_cast<uintptr_t>(x) % 16 || reinterpret_cast<uintptr_t>(y) % 16)
        return HPTT_ERROR_INVALID_ARGUMENT;
    const size_t n16 = n * elem / 16;
    if (n16 == 0) return HPTT_SUCCESS;
    const dim3 grid(uint32_t((n16 + kThreads - 1) / kThreads));
    if (dtype == HPTT_FLOAT32)
        hipLaunchKernelGGL(axpby_kernel<float>, grid, dim3(kThreads), 0, stream, float(alpha),
                           static_cast<const VT<float>*>(x), float(beta),
                           static_cast<VT<float>*>(y), n16);
    else
        hipLaunchKernelGGL(axpby_kernel<double>, grid, dim3(kThreads), 0, stream, alpha,
                           static_cast<const VT<double>*>(x), beta, static_cast<VT<double>*>(y),
                           n16);
    return check_launch();
}

}  // extern "C"
