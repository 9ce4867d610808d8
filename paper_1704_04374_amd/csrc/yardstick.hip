// Measurement kernels: a 16-byte-per-lane streaming copy, an axpby and a
// fill.  Each block moves kUnroll vectors per thread with all loads issued
// before the stores, the usual shape of a bandwidth-bound gfx950 kernel.
#include <hip/hip_runtime.h>

#include "hptt_yardstick.h"

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

struct alignas(16) V16 {
    uint32_t w[4];
};

__global__ __launch_bounds__(kThreads) void copy_kernel(const V16* __restrict__ src,
                                                        V16* __restrict__ dst, size_t n) {
    const size_t i = size_t(blockIdx.x) * (kThreads * kUnroll) + threadIdx.x;
    V16 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (i + size_t(u) * kThreads < n) v[u] = src[i + size_t(u) * kThreads];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (i + size_t(u) * kThreads < n) dst[i + size_t(u) * kThreads] = v[u];
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

template <typename T>
__global__ __launch_bounds__(kThreads) void axpby_kernel(T alpha, const VT<T>* __restrict__ x,
                                                         T beta, VT<T>* __restrict__ y, size_t n) {
#pragma clang fp contract(off)
    constexpr int V = int(16 / sizeof(T));
    const size_t i = size_t(blockIdx.x) * (kThreads * kUnroll) + threadIdx.x;
    VT<T> a[kUnroll], b[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (i + size_t(u) * kThreads < n) {
            a[u] = x[i + size_t(u) * kThreads];
            b[u] = y[i + size_t(u) * kThreads];
        }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (i + size_t(u) * kThreads < n) {
            VT<T> c;
#pragma unroll
            for (int e = 0; e < V; ++e) {
                T s = alpha * a[u].v[e];
                T t = beta * b[u].v[e];
                c.v[e] = s + t;
            }
            y[i + size_t(u) * kThreads] = c;
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
    hipLaunchKernelGGL(copy_kernel, dim3(uint32_t(blocks_for(n))), dim3(kThreads), 0, stream,
                       static_cast<const V16*>(src), static_cast<V16*>(dst), n);
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
    const dim3 grid(uint32_t(blocks_for(n16)));
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
