// Host emulation of the library's kernels, for CPU tests only.
//
// It runs the same phase functions (kernel_body.h) that the gfx950 kernels
// run, one workgroup at a time and one thread after another between the
// points where the device kernels place a barrier, with a memory policy that
// checks every access:
//   - every global offset lies inside its tensor and every vector access is
//     aligned to its width (relative to a 16-byte aligned base);
//   - B is read only when the plan's mode reads it (beta != 0);
//   - every LDS access stays inside the workgroup's LDS, and never reads a
//     word that was not written earlier in the same tile (a missing barrier or
//     a load/store phase mismatch would read stale LDS on the device);
//   - optionally, how many times each B element is written.
// With A and B NULL it only checks offsets ("dry run"), so the launch
// geometry of full-size problems can be verified without their data.
//
// This file is never linked into libhptt.so: it is built into its own test
// library together with the plan builder, and hptt_exec never reaches it.
#include <stdio.h>
#include <string.h>

#include <vector>

#include "kernel_body.h"
#include "plan.h"

namespace {

struct EmuState {
    int64_t numelA = 0;   // elements addressable from A (its footprint)
    int64_t numelB = 0;   // elements addressable from B
    int64_t misA = 0;     // element offset of A's base from the vector grid
    int64_t misB = 0;
    int forceVariant = -1;  // >= 0: run kernel T in this variant (where it applies)
    const void* A = nullptr;
    void* B = nullptr;
    bool readsB = false;
    uint8_t* counts = nullptr;
    std::vector<uint8_t> lds;       // emulated LDS bytes
    std::vector<uint8_t> written;   // 1 where the current tile wrote LDS
    const uint8_t* ldsBase = nullptr;
    int64_t errors = 0;
    char msg[512] = {0};
    bool dry = false;
};

EmuState* S = nullptr;
const void* kDryA = reinterpret_cast<const void*>(uintptr_t(0x1000000));
void* kDryB = reinterpret_cast<void*>(uintptr_t(0x80000000000));

void fail(const char* what, long long a, long long b) {
    if (S->errors++ == 0) snprintf(S->msg, sizeof(S->msg), "%s (%lld, %lld)", what, a, b);
}

// Distance in bytes from address p to the byte range [base, base + bytes).
intptr_t distance(const void* p, const void* base, int64_t bytes) {
    const intptr_t a = reinterpret_cast<intptr_t>(p), b = reinterpret_cast<intptr_t>(base);
    if (a < b) return b - a;
    if (a >= b + intptr_t(bytes)) return a - (b + intptr_t(bytes)) + 1;
    return 0;
}

// Kernels address a tensor from its first element or from a pointer near it
// (a tile's base, which for a sheared chunk past a row's end may lie beyond
// the tensor).  The tensor meant is the one the pointer is nearer to; the
// element accessed must lie inside it.  off is turned into an offset from
// that tensor's first element before every check.
template <typename T>
bool check_global(const T* p, int64_t& off, int V, bool isStore, bool aligned = true) {
    const intptr_t dA = distance(p, S->A, S->numelA * int64_t(sizeof(T)));
    const intptr_t dB = distance(p, S->B, S->numelB * int64_t(sizeof(T)));
    const bool isA = dA <= dB;
    const bool isB = !isA;
    const intptr_t d = reinterpret_cast<intptr_t>(p) + intptr_t(off) * intptr_t(sizeof(T)) -
                       reinterpret_cast<intptr_t>(isA ? S->A : S->B);
    if (d % intptr_t(sizeof(T)) != 0) { fail("access off the element grid", off, V); return false; }
    off = int64_t(d / intptr_t(sizeof(T)));
    if (isA && isStore) { fail("store into A", off, V); return false; }
    if (isB && !isStore && !S->readsB) { fail("B read although beta == 0", off, V); return false; }
    if (off < 0 || off + V > (isA ? S->numelA : S->numelB)) {
        fail(isA ? "A offset out of bounds" : "B offset out of bounds", off, V);
        return false;
    }
    if (aligned && (off + (isA ? S->misA : S->misB)) % V != 0) {
        fail("misaligned vector access", off, V);
        return false;
    }
    return true;
}

// whether p + off lies inside the tensor p points into (A or B)
template <typename T>
bool is_a(const T* p) {
    return distance(p, S->A, S->numelA * int64_t(sizeof(T))) <=
           distance(p, S->B, S->numelB * int64_t(sizeof(T)));
}
template <typename T>
bool in_tensor(const T* p, int64_t off) {
    const bool isA = is_a(p);
    const intptr_t d = reinterpret_cast<intptr_t>(p) + intptr_t(off) * intptr_t(sizeof(T)) -
                       reinterpret_cast<intptr_t>(isA ? S->A : S->B);
    return d >= 0 && d / intptr_t(sizeof(T)) < (isA ? S->numelA : S->numelB);
}

void check_lds(const void* p, int64_t bytes, bool isStore) {
    const int64_t at = static_cast<const uint8_t*>(p) - S->lds.data();
    if (at < 0 || at + bytes > int64_t(S->lds.size())) { fail("LDS access out of bounds", at, bytes); return; }
    for (int64_t i = 0; i < bytes; ++i) {
        if (isStore) S->written[at + i] = 1;
        else if (!S->written[at + i]) { fail("LDS read of a word not written in this tile", at, bytes); return; }
    }
}

struct HostMem {
    template <typename T, int V, bool NT>
    static hptt::Vec<T, V> ld(const T* p, int64_t off) {
        hptt::Vec<T, V> r;
        memset(&r, 0, sizeof(r));
        int64_t at = off;  // offset from the tensor's first element
        if (check_global(p, at, V, false) && !S->dry) memcpy(&r, p + off, sizeof(r));
        return r;
    }
    // the lane's 16-byte slot is ldsWave + lane * V elements
    template <typename T, int V, bool NT>
    static void ld_lds(const T* p, int64_t off, T* ldsWave, int lane) {
        static_assert(V * sizeof(T) == 16, "direct LDS loads move 16 bytes per lane");
        int64_t at = off;
        hptt::Vec<T, V> r;
        memset(&r, 0, sizeof(r));
        if (check_global(p, at, V, false) && !S->dry) memcpy(&r, p + off, sizeof(r));
        T* slot = ldsWave + int64_t(lane) * V;
        check_lds(slot, sizeof(r), true);
        if (S->errors == 0) memcpy(slot, &r, sizeof(r));
    }
    static void wait_ld_lds() {}
    static int wave_uniform(int x) { return x; }
    template <typename T, int V>
    static hptt::Vec<T, V> ldu(const T* p, int64_t off) {
        hptt::Vec<T, V> r;
        memset(&r, 0, sizeof(r));
        int64_t at = off;
        if (check_global(p, at, V, false, false) && !S->dry) memcpy(&r, p + off, sizeof(r));
        return r;
    }
    // an aligned vector of which at least one element is inside the tensor;
    // only those are copied (the device reads the rest from the same page)
    template <typename T, int V, bool NT>
    static hptt::Vec<T, V> ld_part(const T* p, int64_t off) {
        hptt::Vec<T, V> r;
        memset(&r, 0, sizeof(r));
        int first = -1;
        for (int e = 0; e < V && first < 0; ++e) {
            int64_t at = off + e;
            if (in_tensor(p, at)) first = e;
        }
        if (first < 0) {
            fail("partial vector without an element inside the tensor", off, V);
            return r;
        }
        int64_t at = off + first;
        check_global(p, at, 1, false);  // the tensor, the direction, B read only when beta != 0
        const int64_t start = at - first;
        if ((start + (is_a(p) ? S->misA : S->misB)) % V != 0) {
            fail("misaligned partial vector", start, V);
            return r;
        }
        for (int e = 0; e < V; ++e) {
            int64_t x = off + e;
            if (in_tensor(p, x) && !S->dry) r.v[e] = p[off + e];
        }
        return r;
    }
    template <typename T>
    static T ld1(const T* p, int64_t off) {
        T r = T(0);
        int64_t at = off;
        if (check_global(p, at, 1, false) && !S->dry) r = p[off];
        return r;
    }
    template <bool NT, typename T, int V>
    static void st(T* p, int64_t off, const hptt::Vec<T, V>& v) {
        int64_t at = off;
        if (!check_global(p, at, V, true)) return;
        if (!S->dry) memcpy(p + off, &v, sizeof(v));
        if (S->counts)
            for (int e = 0; e < V; ++e)
                if (S->counts[at + e] < 255) ++S->counts[at + e];
    }
    template <bool NT, typename T>
    static void st1(T* p, int64_t off, T v) {
        int64_t at = off;
        if (!check_global(p, at, 1, true)) return;
        if (!S->dry) p[off] = v;
        if (S->counts && S->counts[at] < 255) ++S->counts[at];
    }
    template <typename T>
    static T lds_ld(const T* l, int64_t i) {
        check_lds(l + i, sizeof(T), false);
        T r;
        memcpy(&r, l + i, sizeof(T));
        return r;
    }
    template <typename T>
    static void lds_st(T* l, int64_t i, T v) {
        check_lds(l + i, sizeof(T), true);
        if (S->errors == 0) memcpy(l + i, &v, sizeof(T));
    }
};

void clear_written(int64_t from, int64_t to) {
    memset(S->written.data() + from, 0, size_t(to - from));
}

// Mirrors tile_kernel in tile_kernel.h, in variant VAR with BLOCK threads.
template <typename T, int VA, int VB, int MODE, int NT, int VAR, int BLOCK>
void emu_tile_variant(const hptt_plan_s* p, const T* A, T* B, int64_t blockStride) {
    using namespace hptt;
    TileArgs g = p->tile;  // with the base pointers' offsets from the vector grid, as at launch
    g.misA = int32_t(S->misA % VA);
    g.misB = int32_t(S->misB % VB);
    if (g.shear) g.misLineB = int32_t(S->misB % g.lineB);
    const T alpha = T(p->alpha), beta = T(p->beta);
    const int64_t ldsBytes = p->info.lds_bytes;
    const int64_t tableBytes = (g.runA + g.runB + g.shear) * int64_t(sizeof(int64_t));
    S->lds.assign(size_t(ldsBytes), 0);
    S->written.assign(size_t(ldsBytes), 0);
    int64_t* rowOffA = reinterpret_cast<int64_t*>(S->lds.data());
    int64_t* colOffB = rowOffA + g.runB + g.shear;
    T* lds = reinterpret_cast<T*>(colOffB + g.runA);
    const int64_t grid = p->info.grid;
    for (int64_t blk = 0; blk < grid && S->errors == 0; blk += blockStride) {
        clear_written(0, ldsBytes);
        for (int tid = 0; tid < BLOCK; ++tid) tile_tables<HostMem, BLOCK>(g, tid, rowOffA, colOffB);
        for (int64_t t = blk; t < g.numTiles && S->errors == 0; t += grid) {
            const TileBase tb = tile_base(g, uint32_t(t));
            if (g.flatR) {
                // the row table is the tile's own: a stale entry must not be read
                clear_written(0, g.runB * int64_t(sizeof(int64_t)));
                for (int tid = 0; tid < BLOCK; ++tid) tile_rows_flat<HostMem, BLOCK>(g, tb, tid, rowOffA);
            }
            if constexpr (VAR == kDirect) {
                if (!tile_direct_lds(g, tb, VA)) {
                    fail("tile of a direct-load plan that direct loads cannot serve", int64_t(t),
                         tb.validCols);
                    return;
                }
                clear_written(tableBytes, ldsBytes);
                for (int tid = 0; tid < BLOCK; ++tid)
                    tile_load_direct<HostMem, T, VA, NT, BLOCK>(g, tb, tid, A, lds, rowOffA);
                for (int tid = 0; tid < BLOCK; ++tid)
                    tile_store_rotated<HostMem, T, VA, VB, MODE, NT, BLOCK>(g, tb, tid, B, lds,
                                                                            colOffB, alpha, beta);
            } else {
                for (int64_t r0 = 0; r0 < tb.validRows && S->errors == 0; r0 += g.subRows) {
                    clear_written(tableBytes, ldsBytes);
                    for (int tid = 0; tid < BLOCK; ++tid)
                        tile_load<HostMem, T, VA, NT, VAR, BLOCK, tile_load_batch(MODE, VAR, BLOCK),
                                  tile_part_loads(MODE, VAR)>(
                            g, tb, r0, tid, A, lds, rowOffA);
                    for (int tid = 0; tid < BLOCK; ++tid)
                        tile_store<HostMem, T, VB, MODE, NT, VAR, BLOCK>(g, tb, r0, tid, B, lds,
                                                                         colOffB, alpha, beta);
                }
            }
        }
    }
}

// Mirrors tile_kernel's shared-run variant (kShared).
template <typename T, int VA, int VB, int MODE, int NT>
void emu_tile_shared(const hptt_plan_s* p, const T* A, T* B, int64_t blockStride) {
    using namespace hptt;
    TileArgs g = p->tile;
    g.misA = int32_t(S->misA % VA);
    g.misB = int32_t(S->misB % VB);
    const T alpha = T(p->alpha), beta = T(p->beta);
    const int64_t ldsBytes = p->info.lds_bytes;
    if (tile_lds_bytes(g, int(sizeof(T))) != ldsBytes) {
        fail("LDS size of the plan differs from the kernel's layout", ldsBytes,
             tile_lds_bytes(g, int(sizeof(T))));
        return;
    }
    const int64_t tableBytes = shared_table_words(g) * int64_t(sizeof(int64_t));
    S->lds.assign(size_t(ldsBytes), 0);
    S->written.assign(size_t(ldsBytes), 0);
    int64_t* smem = reinterpret_cast<int64_t*>(S->lds.data());
    int64_t* rowOffA = smem;
    int64_t* colOffB = smem + g.subRows;
    int32_t* ldsCol = reinterpret_cast<int32_t*>(colOffB + g.nColS);
    int32_t* ldsRow = ldsCol + g.nColS;
    T* lds = reinterpret_cast<T*>(smem + shared_table_words(g));
    const int64_t grid = p->info.grid;
    for (int64_t blk = 0; blk < grid && S->errors == 0; blk += blockStride) {
        clear_written(0, ldsBytes);
        for (int tid = 0; tid < kBlock; ++tid)
            tile_tables_shared<HostMem, kBlock>(g, tid, rowOffA, colOffB, ldsCol, ldsRow);
        for (int64_t t = blk; t < g.numTiles && S->errors == 0; t += grid) {
            const TileBase tb = tile_base<true>(g, uint32_t(t));
            clear_written(tableBytes, ldsBytes);
            for (int tid = 0; tid < kBlock; ++tid)
                tile_load<HostMem, T, VA, NT, kShared, kBlock, tile_load_batch(MODE, kShared, kBlock),
                          tile_part_loads(MODE, kShared)>(
                    g, tb, 0, tid, A, lds, rowOffA);
            for (int tid = 0; tid < kBlock; ++tid)
                tile_store_shared<HostMem, T, VB, MODE, NT, kBlock>(g, tb, tid, B, lds, colOffB,
                                                                     ldsCol, ldsRow, alpha, beta);
        }
    }
}

// The variant and workgroup size hptt_exec would launch, or a forced variant:
// kGeneral serves any plan, kShifted and kFast any plan kDirect serves,
// kShifted any plan kFast serves.
template <typename T, int VA, int VB, int MODE, int NT>
void emu_tile(const hptt_plan_s* p, const T* A, T* B, int64_t blockStride) {
    using namespace hptt;
    TileArgs g = p->tile;
    g.misA = int32_t(S->misA % VA);
    g.misB = int32_t(S->misB % VB);
    int var = tile_variant(g);
    if (var != kShared &&
        (S->forceVariant == kGeneral ||
         (S->forceVariant == kShifted && (var == kFast || var == kDirect)) ||
         (S->forceVariant == kFast && var == kDirect)))
        var = S->forceVariant;
    if constexpr (MODE != kAxpby && sizeof(T) * VA == 16) {
        if (var == kDirect) {
            if (p->info.block == kBigBlock)
                emu_tile_variant<T, VA, VB, MODE, NT, kDirect, kBigBlock>(p, A, B, blockStride);
            else
                emu_tile_variant<T, VA, VB, MODE, NT, kDirect, kBlock>(p, A, B, blockStride);
            return;
        }
    }
    if (var == kDirect) {
        fail("direct-load plan with B read or A vectors narrower than 16 bytes", VA, MODE);
        return;
    }
    if (var == kShared)
        emu_tile_shared<T, VA, VB, MODE, NT>(p, A, B, blockStride);
    else if (var == kGeneral)
        emu_tile_variant<T, VA, VB, MODE, NT, kGeneral, kBlock>(p, A, B, blockStride);
    else if (var == kShifted)
        emu_tile_variant<T, VA, VB, MODE, NT, kShifted, kBlock>(p, A, B, blockStride);
    else if (p->info.block == kBigBlock)
        emu_tile_variant<T, VA, VB, MODE, NT, kFast, kBigBlock>(p, A, B, blockStride);
    else
        emu_tile_variant<T, VA, VB, MODE, NT, kFast, kBlock>(p, A, B, blockStride);
}

// Mirrors stream_kernel in kernels.hip.
template <typename T, int V, int MODE, int NT>
void emu_stream_launch(const hptt::StreamArgs& g, uint64_t grid, const T* A, T* B, T alpha,
                       T beta, int64_t blockStride) {
    using namespace hptt;
    const uint64_t per = uint64_t(kBlock) * items_per_lane(int(sizeof(T)), V);
    const uint64_t step = grid * per;
    for (uint64_t blk0 = 0; blk0 < grid && S->errors == 0; blk0 += uint64_t(blockStride)) {
        const uint64_t blk =
            g.xcdGroupLog ? xcd_group_map(uint32_t(blk0), uint32_t(grid), uint32_t(g.xcdGroupLog))
                          : blk0;
        for (uint64_t first = blk * per;
             first < g.numItems[log2_width(V)] && S->errors == 0; first += step)
            for (int tid = 0; tid < kBlock; ++tid) {
                if (g.flatB)
                    stream_items_flat<HostMem, T, V, MODE, NT>(g, uint32_t(first), tid, A, B, alpha,
                                                               beta);
                else
                    stream_items<HostMem, T, V, MODE, NT>(g, uint32_t(first), tid, A, B, alpha, beta);
            }
    }
}

// Mirrors stream_kernel in kernels.hip, launched once, or once per slab
// (stream_slabs in kernels.hip) when its items exceed 32 bits.
template <typename T, int V, int MODE, int NT>
void emu_stream(const hptt_plan_s* p, const T* A, T* B, int64_t blockStride) {
    using namespace hptt;
    const StreamArgs& g = p->stream;
    const T alpha = T(p->alpha), beta = T(p->beta);
    if (g.flatB || g.numItems[log2_width(V)] != 0) {
        emu_stream_launch<T, V, MODE, NT>(g, uint64_t(p->info.grid), A, B, alpha, beta,
                                          blockStride);
        return;
    }
    const StreamSlabs s = stream_slabs_of(g, V);
    const int64_t per = int64_t(kBlock) * items_per_lane(int(sizeof(T)), V);
    for (int64_t sl = 0; sl < s.count && S->errors == 0; ++sl) {
        int64_t offA = 0, offB = 0;
        const StreamArgs sa = stream_slab_args(g, s, sl, V, &offA, &offB);
        int64_t grid = (int64_t(sa.numItems[log2_width(V)]) + per - 1) / per;
        if (grid > p->info.grid) grid = p->info.grid;
        emu_stream_launch<T, V, MODE, NT>(sa, uint64_t(grid), A + offA, B + offB, alpha, beta,
                                          blockStride);
    }
}

// Mirrors axpby_kernel and generic_kernel in kernels.hip.
template <typename T, int V, int MODE, int NT>
void emu_axpby(const hptt_plan_s* p, const T* A, T* B, int64_t blockStride) {
    using namespace hptt;
    const int64_t numel = p->info.numel, vecs = (numel + V - 1) / V;
    const int64_t per = int64_t(kBlock) * items_per_lane(int(sizeof(T)), V);
    const int64_t grid = p->info.grid, step = grid * per;
    for (int64_t blk = 0; blk < grid && S->errors == 0; blk += blockStride)
        for (int64_t first = blk * per; first < vecs; first += step)
            for (int tid = 0; tid < kBlock; ++tid)
                axpby_items<HostMem, T, V, MODE, NT>(numel, first, tid, A, B, T(p->alpha), T(p->beta));
}

template <typename T, int MODE, int NT>
void emu_generic(const hptt_plan_s* p, const T* A, T* B, int64_t blockStride) {
    using namespace hptt;
    const GenericArgs& g = p->generic;
    const int64_t grid = p->info.grid, stride = grid * kBlock;
    const bool big = g.numel >= (int64_t(1) << 32);
    for (int64_t blk = 0; blk < grid && S->errors == 0; blk += blockStride)
        for (int tid = 0; tid < kBlock; ++tid)
            for (int64_t e = blk * kBlock + tid; e < g.numel; e += stride) {
                if (big) generic_elem<HostMem, T, MODE, NT, true>(g, e, A, B, T(p->alpha), T(p->beta));
                else generic_elem<HostMem, T, MODE, NT, false>(g, e, A, B, T(p->alpha), T(p->beta));
            }
}

template <typename T, int MODE, int NT, int VA, int VB>
void run_widths(const hptt_plan_s* p, const T* A, T* B, int64_t bs) {
    switch (p->info.kernel) {
        case HPTT_KERNEL_TILE: emu_tile<T, VA, VB, MODE, NT>(p, A, B, bs); break;
        case HPTT_KERNEL_STREAM:
            // the flat walk takes B's width alone, as hptt_exec does
            if (p->stream.flatB) emu_stream<T, VB, MODE, NT>(p, A, B, bs);
            else emu_stream<T, (VA < VB ? VA : VB), MODE, NT>(p, A, B, bs);
            break;
        case HPTT_KERNEL_AXPBY: emu_axpby<T, (VA < VB ? VA : VB), MODE, NT>(p, A, B, bs); break;
        case HPTT_KERNEL_GENERIC: emu_generic<T, MODE, NT>(p, A, B, bs); break;
        default: break;
    }
}

template <typename T, int MODE, int NT, int VA>
void run_vb(const hptt_plan_s* p, const T* A, T* B, int vb, int64_t bs) {
    if (vb == 1) run_widths<T, MODE, NT, VA, 1>(p, A, B, bs);
    else if (vb == 2) run_widths<T, MODE, NT, VA, 2>(p, A, B, bs);
    else if constexpr (sizeof(T) == 4) run_widths<T, MODE, NT, VA, 4>(p, A, B, bs);
}

template <typename T, int MODE, int NT>
void run_va(const hptt_plan_s* p, const T* A, T* B, int va, int vb, int64_t bs) {
    if (va == 1) run_vb<T, MODE, NT, 1>(p, A, B, vb, bs);
    else if (va == 2) run_vb<T, MODE, NT, 2>(p, A, B, vb, bs);
    else if constexpr (sizeof(T) == 4) run_vb<T, MODE, NT, 4>(p, A, B, vb, bs);
}

template <typename T, int MODE>
void run_hint(const hptt_plan_s* p, const T* A, T* B, int va, int vb, int64_t bs) {
    switch (p->info.hints) {
        case 0: run_va<T, MODE, 0>(p, A, B, va, vb, bs); break;
        case hptt::kNtStore: run_va<T, MODE, hptt::kNtStore>(p, A, B, va, vb, bs); break;
        case hptt::kNtLoad: run_va<T, MODE, hptt::kNtLoad>(p, A, B, va, vb, bs); break;
        default: run_va<T, MODE, hptt::kNtStore | hptt::kNtLoad>(p, A, B, va, vb, bs);
    }
}

template <typename T>
void run(const hptt_plan_s* p, const T* A, T* B, int va, int vb, int64_t bs) {
    switch (p->info.mode) {
        case hptt::kCopy: run_hint<T, hptt::kCopy>(p, A, B, va, vb, bs); break;
        case hptt::kScale: run_hint<T, hptt::kScale>(p, A, B, va, vb, bs); break;
        default: run_hint<T, hptt::kAxpby>(p, A, B, va, vb, bs);
    }
}

}  // namespace

extern "C" {

// Emulate hptt_exec of `plan` on host buffers A and B (or, with both NULL,
// only the offsets).  va/vb = 0 use the plan's vector widths, others force
// narrower ones as hptt_exec does for less aligned pointers (stream and axpby
// kernels).  misA/misB: the base pointers' element offsets from the 16-byte
// grid, which the tile kernel shifts its runs by (vector accesses are checked
// for alignment relative to that grid).  variant >= 0 runs the tile kernel
// in that variant (kGeneral on any plan, kShifted on plans kFast or kDirect
// serves, kFast on plans kDirect serves; plans whose runs share indices
// always run kShared) instead of the one hptt_exec would launch.
// counts (numel
// bytes, or NULL) is incremented at every B element written.  Only
// workgroups 0, block_stride, 2*block_stride, ... are run.  Returns the
// number of violations; the first is described in msg.  For sub-tensor plans
// A, B and counts cover the footprints (info.footprint_a, footprint_b).
int64_t hptt_emulate_exec(hptt_plan_t plan, const void* A, void* B, int32_t va, int32_t vb,
                          uint8_t* counts, int64_t block_stride, char* msg, size_t msglen,
                          int32_t misA, int32_t misB, int32_t variant) {
    if (!plan) return -1;
    EmuState st;
    S = &st;
    st.forceVariant = variant;
    st.numelA = plan->info.footprint_a;
    st.numelB = plan->info.footprint_b;
    st.misA = misA;
    st.misB = misB;
    st.dry = (A == nullptr && B == nullptr);
    st.A = st.dry ? kDryA : A;
    st.B = st.dry ? kDryB : B;
    st.readsB = plan->info.mode == hptt::kAxpby;
    st.counts = counts;
    if (va <= 0) va = plan->info.vec_a;
    if (vb <= 0) vb = plan->info.vec_b;
    if (block_stride < 1) block_stride = 1;
    if (plan->info.kernel != HPTT_KERNEL_NONE && plan->info.numel > 0) {
        if (plan->dtype == HPTT_FLOAT32)
            run<float>(plan, static_cast<const float*>(st.A), static_cast<float*>(st.B), va, vb, block_stride);
        else
            run<double>(plan, static_cast<const double*>(st.A), static_cast<double*>(st.B), va, vb, block_stride);
    }
    if (msg && msglen) snprintf(msg, msglen, "%s", st.msg);
    S = nullptr;
    return st.errors;
}

// Exhaustive check of the fast division used by every kernel: n / d for the
// given divisor and every dividend in [lo, hi).  Returns the first dividend
// that divides wrongly, or -1.
int64_t hptt_emulate_check_fastdiv(uint32_t d, uint64_t lo, uint64_t hi) {
    const hptt::FastDiv f = hptt::make_fastdiv(d);
    for (uint64_t n = lo; n < hi; ++n)
        if (hptt::fast_div(uint32_t(n), f) != uint32_t(n) / d) return int64_t(n);
    return -1;
}

}  // extern "C"
