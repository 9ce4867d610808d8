// Kernel T (stride-1 index moved) as a __global__ template, and the table
// that maps (update mode, cache hints, vector widths) to one instantiation.
// Each tile_*.hip file instantiates it for one element type and variant (fp64:
// all three), so the instantiations compile in parallel; kernels.hip only
// receives the kernel addresses through tile_kernel_f32 / tile_kernel_f64.
#pragma once

#include "device_mem.h"

namespace hptt {

// Address of the tile kernel for (update mode, cache hints, vector widths,
// workgroup size) in variant kFast (256 or 1024 threads), kShifted, kGeneral
// or kShared (256 threads; see tile_variant), or nullptr for an unsupported
// combination.  Defined in tile_f64.hip.
const void* tile_kernel_f32(int variant, int mode, int hints, int va, int vb, int block);
const void* tile_kernel_f64(int variant, int mode, int hints, int va, int vb, int block);

namespace {

// One workgroup of BLOCK threads per tile (or a grid-stride loop over tiles
// when the grid is capped): build the offset tables once, then for each pass
// load A runs into LDS, barrier, and store B runs.  A 1024-thread workgroup
// asks for 8 waves per SIMD, i.e. two workgroups per CU, which keeps its
// registers at 64 VGPRs per lane.  So does variant kFast when it reads B
// (batches of 4 loads and 2 stores): it would otherwise hold 7, limited by
// its scalar registers (MI355X, the 5-D fp32 beta = 1 workload 5.41 ->
// 5.57-5.64 TB/s; with beta = 0 the same cap lost 3-15 %, and on the
// shifted and shared-run variants it lost 3 % of the beta = 1 sweep).
template <int MODE, int VAR, int BLOCK>
constexpr int tile_waves_per_eu() {
    return BLOCK >= 1024 || (MODE == kAxpby && VAR == kFast) ? 8 : 1;
}

template <typename T, int VA, int VB, int MODE, int HINT, int VAR, int BLOCK>
__global__ __launch_bounds__(BLOCK)
__attribute__((amdgpu_waves_per_eu(tile_waves_per_eu<MODE, VAR, BLOCK>())))
void tile_kernel(const T* __restrict__ A, T* __restrict__ B, const TileArgs g, T alpha, T beta) {
    constexpr int LB = VAR == kDirect ? 0 : tile_load_batch(MODE, VAR, BLOCK);
    extern __shared__ int64_t smem[];
    if constexpr (VAR == kDirect) {
        // A fetched straight into LDS, one pass per tile (tile_load_direct)
        int64_t* rowOffA = smem;
        int64_t* colOffB = smem + g.runB;
        T* lds = reinterpret_cast<T*>(colOffB + g.runA);
        const int tid = int(threadIdx.x);
        tile_tables<DeviceMem, BLOCK>(g, tid, rowOffA, colOffB);
        __syncthreads();
        bool first = true;
        for (uint32_t t = blockIdx.x; t < g.numTiles; t += gridDim.x) {
            const TileBase tb = tile_base(g, t);
            if (g.flatR) {
                // past the previous tile's load phase, the only reader of the
                // row table; the barrier also ends its store phase
                tile_rows_flat<DeviceMem, BLOCK>(g, tb, tid, rowOffA);
                __syncthreads();
            } else if (!first) {
                __syncthreads();  // the previous tile's LDS reads are done
            }
            first = false;
            tile_load_direct<DeviceMem, T, VA, HINT, BLOCK>(g, tb, tid, A, lds, rowOffA);
            __syncthreads();
            tile_store_rotated<DeviceMem, T, VA, VB, MODE, HINT, BLOCK>(g, tb, tid, B, lds, colOffB,
                                                                        alpha, beta);
        }
    } else {
        // the variants that stage A through registers
        if constexpr (VAR == kShared) {
            // runs that share indices: one pass per tile, the store phase
            // gathering from LDS at positions from a table or computed
            int64_t* rowOffA = smem;
            int64_t* colOffB = smem + g.subRows;
            int32_t* ldsCol = reinterpret_cast<int32_t*>(colOffB + g.nColS);
            int32_t* ldsRow = ldsCol + g.nColS;
            T* lds = reinterpret_cast<T*>(smem + shared_table_words(g));
            const int tid = int(threadIdx.x);
            tile_tables_shared<DeviceMem, BLOCK>(g, tid, rowOffA, colOffB, ldsCol, ldsRow);
            __syncthreads();
            bool first = true;
            for (uint32_t t = blockIdx.x; t < g.numTiles; t += gridDim.x) {
                const TileBase tb = tile_base<true>(g, t);
                if (!first) __syncthreads();  // the previous tile's LDS reads are done
                first = false;
                tile_load<DeviceMem, T, VA, HINT, VAR, BLOCK, LB, tile_part_loads(MODE, VAR)>(
                    g, tb, 0, tid, A, lds, rowOffA);
                __syncthreads();
                tile_store_shared<DeviceMem, T, VB, MODE, HINT, BLOCK>(g, tb, tid, B, lds, colOffB,
                                                                        ldsCol, ldsRow, alpha, beta);
            }
            return;
        }
        int64_t* rowOffA = smem;
        int64_t* colOffB = smem + g.runB + g.shear;
        T* lds = reinterpret_cast<T*>(colOffB + g.runA);
        const int tid = int(threadIdx.x);
        tile_tables<DeviceMem, BLOCK>(g, tid, rowOffA, colOffB);
        __syncthreads();
        bool first = true;
        for (uint32_t t = blockIdx.x; t < g.numTiles; t += gridDim.x) {
            const TileBase tb = tile_base(g, t);
            if (g.flatR) {
                // every lane is past the previous tile's load phase, the only
                // reader of the row table; the barrier also ends its store phase
                tile_rows_flat<DeviceMem, BLOCK>(g, tb, tid, rowOffA);
                __syncthreads();
                first = true;
            }
            for (int64_t r0 = 0; r0 < tb.validRows; r0 += g.subRows) {
                if (!first) __syncthreads();  // the previous pass's LDS reads are done
                first = false;
                tile_load<DeviceMem, T, VA, HINT, VAR, BLOCK, LB, tile_part_loads(MODE, VAR)>(
                    g, tb, r0, tid, A, lds, rowOffA);
                __syncthreads();
                tile_store<DeviceMem, T, VB, MODE, HINT, VAR, BLOCK>(g, tb, r0, tid, B, lds, colOffB,
                                                                     alpha, beta);
            }
        }
    }
}

template <typename T, int VA, int MODE, int HINT, int VAR, int BLOCK>
const void* tile_vb(int vb) {
    switch (vb) {
        case 1: return reinterpret_cast<const void*>(&tile_kernel<T, VA, 1, MODE, HINT, VAR, BLOCK>);
        case 2: return reinterpret_cast<const void*>(&tile_kernel<T, VA, 2, MODE, HINT, VAR, BLOCK>);
        case 4:
            if constexpr (kMaxVec<T> >= 4)
                return reinterpret_cast<const void*>(
                    &tile_kernel<T, VA, 4, MODE, HINT, VAR, BLOCK>);
            return nullptr;
    }
    return nullptr;
}

template <typename T, int MODE, int HINT, int VAR, int BLOCK>
const void* tile_va(int va, int vb) {
    if constexpr (VAR == kDirect) {  // A vectors of 16 bytes only
        return va == kMaxVec<T> ? tile_vb<T, kMaxVec<T>, MODE, HINT, VAR, BLOCK>(vb) : nullptr;
    } else {
        switch (va) {
            case 1: return tile_vb<T, 1, MODE, HINT, VAR, BLOCK>(vb);
            case 2: return tile_vb<T, 2, MODE, HINT, VAR, BLOCK>(vb);
            case 4:
                if constexpr (kMaxVec<T> >= 4) return tile_vb<T, 4, MODE, HINT, VAR, BLOCK>(vb);
                return nullptr;
        }
        return nullptr;
    }
}

template <typename T, int MODE, int VAR, int BLOCK>
const void* tile_hint(int hints, int va, int vb) {
    switch (hints) {
        case 0: return tile_va<T, MODE, 0, VAR, BLOCK>(va, vb);
        case kNtStore: return tile_va<T, MODE, kNtStore, VAR, BLOCK>(va, vb);
        case kNtLoad: return tile_va<T, MODE, kNtLoad, VAR, BLOCK>(va, vb);
        default: return tile_va<T, MODE, kNtStore | kNtLoad, VAR, BLOCK>(va, vb);
    }
}

template <typename T, int VAR, int BLOCK>
const void* tile_mode(int mode, int hints, int va, int vb) {
    if constexpr (VAR == kDirect) {  // B only written, 16-byte A vectors
        if (mode == kAxpby || va != kMaxVec<T>) return nullptr;
        if (mode == kCopy) return tile_hint<T, kCopy, VAR, BLOCK>(hints, va, vb);
        return tile_hint<T, kScale, VAR, BLOCK>(hints, va, vb);
    } else {
        switch (mode) {
            case kCopy: return tile_hint<T, kCopy, VAR, BLOCK>(hints, va, vb);
            case kScale: return tile_hint<T, kScale, VAR, BLOCK>(hints, va, vb);
            default: return tile_hint<T, kAxpby, VAR, BLOCK>(hints, va, vb);
        }
    }
}

// Variants kShifted, kGeneral and kShared exist for kBlock threads only;
// kFast and kDirect for kBlock and kBigBlock.
template <typename T, int VAR>
const void* tile_kernel_address(int mode, int hints, int va, int vb, int block) {
    if (block == kBlock) return tile_mode<T, VAR, kBlock>(mode, hints, va, vb);
    if constexpr (VAR == kFast || VAR == kDirect)
        if (block == kBigBlock) return tile_mode<T, VAR, kBigBlock>(mode, hints, va, vb);
    return nullptr;
}

}  // namespace
}  // namespace hptt
