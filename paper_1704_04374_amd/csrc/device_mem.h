// Memory policy of the device kernels: plain global and LDS accesses.  A
// vector of V elements is one global_load/store of V*sizeof(T) bytes; the
// plan only asks for widths that keep every such access aligned, except
// ldu, whose loads need only element alignment.
#pragma once

#include <hip/hip_runtime.h>

#include "kernel_body.h"

namespace hptt {
namespace {

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
    // The aligned vector of V elements at p + off when only some of them
    // belong to the tensor (the caller keeps those and drops the rest): an
    // aligned access of at most 16 bytes lies inside one page, which holds a
    // valid element and so is mapped.  One load instead of one per element.
    template <typename T, int V, bool NT>
    __device__ __forceinline__ static Vec<T, V> ld_part(const T* p, int64_t off) {
        return ld<T, V, NT>(p, off);
    }
    // V consecutive elements from any element boundary: one global_load of
    // V*sizeof(T) bytes at a dword-aligned address (gfx950 serves those
    // in both of its alignment modes).
    template <typename T, int V>
    __device__ __forceinline__ static Vec<T, V> ldu(const T* p, int64_t off) {
        Vec<T, V> r;
        __builtin_memcpy(&r, p + off, sizeof(r));
        return r;
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
    // V elements (16 bytes) from p + off straight into LDS: the wave's 64
    // lanes write the 64 consecutive 16-byte slots from ldsWave on (lane is
    // implied by the hardware; ldsWave must be the same for every lane).
    template <typename T, int V, bool NT>
    __device__ __forceinline__ static void ld_lds(const T* p, int64_t off, T* ldsWave, int) {
        static_assert(V * sizeof(T) == 16, "direct LDS loads move 16 bytes per lane");
#if defined(__HIP_DEVICE_COMPILE__)
        __builtin_amdgcn_global_load_lds(p + off, ldsWave, 16, 0, NT ? 2 : 0);
#endif
    }
    // Wait until this lane's direct LDS loads have landed (before a barrier).
    __device__ __forceinline__ static void wait_ld_lds() {
#if defined(__HIP_DEVICE_COMPILE__)
        __builtin_amdgcn_s_waitcnt(0);
#endif
    }
    // A value the whole wave holds, kept in a scalar register.
    __device__ __forceinline__ static int wave_uniform(int x) {
#if defined(__HIP_DEVICE_COMPILE__)
        return __builtin_amdgcn_readfirstlane(x);
#else
        return x;
#endif
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

template <typename T>
constexpr int kMaxVec = int(16 / sizeof(T));

}  // namespace
}  // namespace hptt
