// Plan builder: the quick path of plan creation (Section 3.1).  It validates
// the problem, drops extent-1 indices, merges indices that are consecutive in
// both A and B into superindices (Section 3.1, footnote 4), classifies the
// fused problem, and picks one kernel, tile and vector width without any
// search.  Host code only; it makes no HIP call.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "plan.h"

namespace hptt {

int64_t tile_lds_bytes_host(const TileArgs& t, int elem) {
    if (t.shared)  // tables: rowOffA, colOffB (64-bit), ldsCol, ldsRow with posTable (32-bit)
        return (int64_t(t.subRows) + t.nColS + (t.nColS + (t.posTable ? t.runB : 0) + 1) / 2) *
                   int64_t(sizeof(int64_t)) +
               int64_t(t.subRows) * t.pitch * elem;
    return (t.runA + t.runB + t.shear) * int64_t(sizeof(int64_t)) +
           (int64_t(t.nZ) * t.subRows + t.shear) * t.pitch * elem;
}

namespace {

constexpr int64_t kLdsMax = 64 * 1024;     // LDS a kernel-T workgroup may use
constexpr int64_t kLdsMaxBig = 152 * 1024; // ... with kBigBlock threads (one per CU)
constexpr int64_t kLdsBudget = 40 * 1024;  // preferred: at least 4 workgroups per CU
// Shared-run tiles when B is read too (beta != 0): 8 resident workgroups per
// CU (their position table is as large as the tile's data, fp32).  On the
// MI355X sweep's 12 shared-run cases: beta = 1 3.87 TB/s against 3.55 with
// the 40 KiB budget, beta = 0 3.22 against 3.30, so beta = 0 keeps 40 KiB.
constexpr int64_t kSharedLdsBudgetAxpby = 20 * 1024;
constexpr int64_t kLine = 128;             // L2 cache line of gfx950
constexpr int64_t kVecBytes = 16;          // widest global access per lane (dwordx4)
constexpr int64_t kMinTileBytes = 16 * 1024;  // a workgroup round below this is mostly overhead
constexpr double kMinGrid = 2048;          // workgroups a larger tile must still leave (8 per CU)

int64_t gcd64(int64_t a, int64_t b) {
    if (a < 0) a = -a;
    if (b < 0) b = -b;
    while (b) {
        int64_t t = a % b;
        a = b;
        b = t;
    }
    return a;
}

// Largest power-of-two vector width (in elements, at most 16 bytes and at
// most `cap`) that divides `gran`; gran == 0 means every offset is 0.
int32_t vec_width(int64_t gran, int elem, int32_t cap) {
    int32_t v = int32_t(kVecBytes / elem);
    while (cap > 0 && v > cap) v /= 2;
    while (v > 1 && gran % v != 0) v /= 2;
    return v;
}

// Vector width of a tile run of `run` elements whose starts have gcd `gran`:
// the tile kernel shifts runs that start off the vector grid onto it, so the
// width is limited by the run length, not by the alignment: a run on the grid
// takes vectors up to its length, a run off it needs two vectors' worth (its
// first and last vectors are partial).
int32_t run_vec_width(int64_t run, int64_t gran, int elem, int32_t cap) {
    int32_t v = int32_t(kVecBytes / elem);
    while (cap > 0 && v > cap) v /= 2;
    const bool onGrid = gran % v == 0;
    while (v > 1 && (onGrid ? run < v : run < 2 * v)) v /= 2;
    return v;
}

// The fused problem: M indices of A with extents n, B position k holding
// fused A index p[k], and the strides of every A index in A and in B.
struct Fused {
    int M;
    int64_t n[kMaxDims];
    int32_t p[kMaxDims];
    int64_t sA[kMaxDims];  // stride in A of A index d
    int64_t sB[kMaxDims];  // stride in B of A index d
};

// Drop extent-1 indices, then merge maximal groups of B positions whose A
// indices are consecutive and increasing and lie back to back in memory in
// both tensors (each stride equals the previous stride times the previous
// extent): such a group behaves as one index (Section 3.1, footnote 4).
// Strides are the Fortran strides of the enclosing extents (the outer sizes
// of Fig. 3); compact tensors have outer sizes equal to their sizes, and then
// every group of consecutive indices qualifies.
void fuse(const int32_t* perm, int32_t N, const int64_t* sizeA, const int64_t* outerA,
          const int64_t* outerB, Fused& f) {
    int64_t strideA[kMaxDims], strideB[kMaxDims];  // per original A index
    int64_t s = 1;
    for (int d = 0; d < N; ++d) {
        strideA[d] = s;
        s *= outerA[d];
    }
    s = 1;
    for (int k = 0; k < N; ++k) {
        strideB[perm[k]] = s;
        s *= outerB[k];
    }
    int32_t newIdx[kMaxDims];
    int kept = 0;
    for (int d = 0; d < N; ++d) newIdx[d] = sizeA[d] > 1 ? kept++ : -1;
    int64_t n[kMaxDims], sA[kMaxDims], sB[kMaxDims];
    int32_t p[kMaxDims];
    int m = 0;
    for (int d = 0; d < N; ++d)
        if (newIdx[d] >= 0) {
            n[newIdx[d]] = sizeA[d];
            sA[newIdx[d]] = strideA[d];
            sB[newIdx[d]] = strideB[d];
        }
    for (int k = 0; k < N; ++k)
        if (newIdx[perm[k]] >= 0) p[m++] = newIdx[perm[k]];
    if (m == 0) {  // every extent is 1: one element
        f.M = 1;
        f.n[0] = 1;
        f.p[0] = 0;
        f.sA[0] = f.sB[0] = 1;
        return;
    }
    // groups in B order: first A index and extent
    int32_t first[kMaxDims];
    int64_t ext[kMaxDims];
    int G = 0;
    for (int k = 0; k < m; ++k) {
        const int32_t a = p[k], prev = k > 0 ? p[k - 1] : -1;
        const bool join = k > 0 && a == prev + 1 && sA[a] == sA[prev] * n[prev] &&
                          sB[a] == sB[prev] * n[prev];
        if (join) {
            ext[G - 1] *= n[a];
        } else {
            first[G] = a;
            ext[G] = n[a];
            ++G;
        }
    }
    // fused A index of a group = rank of its first A index
    for (int g = 0; g < G; ++g) {
        int rank = 0;
        for (int h = 0; h < G; ++h) rank += first[h] < first[g];
        f.p[g] = rank;
        f.n[rank] = ext[g];
        f.sA[rank] = sA[first[g]];
        f.sB[rank] = sB[first[g]];
    }
    f.M = G;
}

// gcd of the strides (in one tensor) of the fused A indices in `which` that
// have extent > 1; 0 if there are none.
int64_t stride_gcd(const Fused& f, const int64_t* stride, const bool* which) {
    int64_t g = 0;
    for (int d = 0; d < f.M; ++d)
        if (which[d] && f.n[d] > 1) g = gcd64(g, stride[d]);
    return g;
}

// Chunk of an index of extent n that extends a contiguous run whose inner
// part has `inner` elements, aiming at a run of `target` elements.  Runs then
// start at multiples of gcd(chunk stride, `other`), where `other` is the gcd
// of the strides of every index outside the run.  With `aligned`, only chunks
// whose runs start and end on 128-byte lines qualify (no line is then shared
// between workgroups); returns 0 if there is none.  Among the candidates: the
// length closest to target, where falling short counts double and a partial
// last chunk counts by the share of lanes it leaves idle.
int64_t choose_chunk(int64_t inner, int64_t n, int64_t other, int64_t target, int elem,
                     bool aligned) {
    int64_t best = 0;
    double bestScore = 1e30;
    // Line-aligned chunks are multiples of `step` and may be long, up to
    // what one LDS tile could hold; others are looked for up to four times
    // the target.
    const int64_t step = aligned ? kLine / gcd64(kLine, inner * elem) : 1;
    const int64_t kmax = aligned ? kLdsMax / (inner * elem) : (4 * target) / inner;
    for (int64_t k = step; k <= n && (k == 1 || k <= kmax); k += step) {
        const int64_t run = inner * k;
        const int64_t gran = gcd64(k < n ? run : 0, other);
        const bool lineAligned = (gran * elem) % kLine == 0 && (run * elem) % kLine == 0;
        if (aligned && !lineAligned) continue;
        // a run shorter than the target costs twice as much as a longer one;
        // a chunk that does not divide the extent costs the share of the
        // chunks' elements its last, partial chunk leaves idle
        const double ratio = log2(double(run) / double(target));
        const int64_t chunks = (n + k - 1) / k;
        const double idle = double(chunks * k - n) / double(chunks * k);
        const double score = 6.0 * idle + (ratio < 0 ? -2.0 * ratio : ratio);
        if (score < bestScore) {
            bestScore = score;
            best = k;
        }
    }
    return best;
}

void set_div(FastDiv& f, int64_t d) { f = make_fastdiv(uint32_t(d)); }

// Order of the grid digits outside the tile (outer_indices); 0 = A order.
int32_t grid_order(const hptt_options_t& opt) { return opt.grid_order ? opt.grid_order : 1; }

// Direct LDS loads (TileArgs::directLds): tiles whose B is only written, with
// 16-byte A vectors, staged in one pass without stacking or shear, whose LDS
// data starts on 16 bytes (the tables before it hold an even number of
// 64-bit words) and whose row rotation (row / 4) stays below the vectors per
// row.  MI355X, same process, against the register-staged load phase: the
// 6-D fp32 workload 1.05x, 8192x4096 fp64 1.06x, the 2-D fp32 workload
// 1.01x, its transpose-and-compact half 1.02x; with beta != 0 it lost 5 %
// (the 5-D workload), so B read and written keeps the register path.
void set_direct_lds(const hptt_options_t& opt, int elem, hptt_plan_info_t& info, TileArgs& t) {
    const int64_t va = info.vec_a;
    // every tile's columns whole vectors, the last chunk's too
    const bool wholeCols = t.runA % va == 0 && (t.cChunk >= t.cLast || t.cLast % t.cChunk == 0 ||
                                                (t.cInner * (t.cLast % t.cChunk)) % va == 0);
    t.directLds = opt.direct_lds != 2 && info.mode != kAxpby && !t.shared && t.nZ == 1 &&
                          t.shear == 0 && t.subRows >= t.runB && elem * va == 16 && wholeCols &&
                          (t.runA + t.runB + t.shear) % 2 == 0 && ((t.subRows - 1) >> 2) < t.runA / va
                      ? 1
                      : 0;
    info.direct_lds = t.directLds;
}

// XCD groups for short A runs that do not start on lines (TileArgs::
// xcdGroupLog): two tiles next to each other along the A run share a line of
// A at their boundary; dealt round robin to the XCDs, they fetch it into two
// L2s (rocprofv3 on MI355X: 2193x22800 [1,0] fetched 2.46x A's bytes,
// 112582x444 2.35x).  Groups of 16 tiles per XCD, in grid-digit order (the
// diagonal rotation would part the neighbours), fetch each line once.  Runs
// of up to 320 bytes only, where the boundary lines are a large share of the
// run: MI355X, the cases of the 57-case sweep with runs up to 256 bytes,
// -0.4 to +29 % (mean +9.5 %) with beta = 0 and -1.5 to +14 % (mean +3.8 %)
// with beta = 1; runs of 257-320 bytes (fp32 and fp64) -1.6 to +13 %, mean
// +2.6 %; tiles whose columns lie a multiple of 4 KiB apart in B lost up to
// 7 % to the diagonal order's spread over the HBM channels (below).
// Shared-run tiles take the same rule: the five such plans measured (A runs
// of 63-70 elements off the line grid, three of them kept-index tiles)
// gained -0.1 to +5 % (mean +2.6 %) with beta = 0 and -0.7 to +2.8 % (mean
// +1.1 %) with beta = 1, while the long single-row ones lost 1-3 %.
void set_xcd_groups(const hptt_options_t& opt, int elem, hptt_plan_info_t& info, TileArgs& t) {
    if (opt.xcd_group != 0 || opt.tile_order != 0 || t.alignedA || t.runA * elem > 320)
        return;
    // A B stride of the A run's first index that is a multiple of 4 KiB
    // (every column of the tile, and of its neighbours, the same distance
    // from a channel boundary) keeps the diagonal order, which spreads the
    // tiles in flight over the HBM channels (MI355X, beta = 1, 64-element
    // runs: 3001x16384 [1,0], columns 64 KiB apart in B, -7 % in groups;
    // 999x4x12288 [2,0,1], 48 KiB, -6 %).
    if (t.nC > 0 && (t.cStrideB[0] * elem) % 4096 == 0) return;
    t.skew = 0;
    t.xcdGroupLog = 4;
    info.tile_order = 1;
    info.xcd_group = 1 << t.xcdGroupLog;
}

// Grid order of kernel T (both set-ups): diagonal (the second digit
// rotated by skew times the first) unless asked otherwise, and optionally
// contiguous tile ranges per XCD.
void set_tile_order(TileArgs& t, const hptt_options_t& opt, int g, const int64_t* ext,
                    hptt_plan_info_t& info) {
    t.skew = (g >= 2 && opt.tile_order != 1 && opt.tile_order != 4) ? (opt.skew > 0 ? opt.skew : 1)
                                                                     : 0;
    if (t.skew > 1 && uint64_t(ext[0]) * uint64_t(t.skew) >= (uint64_t(1) << 32)) t.skew = 1;
    t.xcdSplit = (opt.tile_order == 3 || opt.tile_order == 4) ? 1 : 0;
    info.tile_order = t.xcdSplit ? (t.skew ? 3 : 4) : t.skew ? 2 : 1;
    int log = 0;
    while (!t.xcdSplit && (int64_t(1) << (log + 1)) <= opt.xcd_group) ++log;
    t.xcdGroupLog = log;
    info.xcd_group = t.xcdSplit ? 0 : 1 << log;
    info.grid_order = grid_order(opt);
}

// Kernel T set-up for targets tA (A-run) and tB (B-run).  Returns false if the
// tile does not fit the LDS budget or the grid is too large.
// The fused indices outside a tile, in the order they become grid digits
// (after the chunk counters): 1 = A order, 2 = by the sum of their strides
// in A and B (the index closest to contiguous in both tensors first, ties in
// A order), 3 = B order.
int outer_indices(const Fused& f, const bool* skip, int32_t order, int* out) {
    int n = 0;
    if (order == 3) {
        for (int k = 0; k < f.M; ++k)
            if (!skip[f.p[k]]) out[n++] = f.p[k];
        return n;
    }
    for (int a = 0; a < f.M; ++a)
        if (!skip[a]) out[n++] = a;
    if (order == 2)
        std::stable_sort(out, out + n, [&](int x, int y) {
            return f.sA[x] + f.sB[x] < f.sA[y] + f.sB[y];
        });
    return n;
}

// Contiguous regions of A plus those of B that a window of kResident
// consecutive tiles touches, for one order of the outer grid digits: a model
// of how scattered the traffic of the workgroups resident at one time is.
// covered[d] = how many values of fused index d the window spans (the tile's
// own run, times the window's count of the digit that chunks it; a digit
// after the window's first partial one contributes one value); a side's
// contiguous block grows over its indices in memory order while each is
// spanned whole (and back to back), and its regions are the window's
// elements over that block.  Flat B runs (flatR) span the flattened B-run
// range: its window count is spread over the B-run indices in B order.
constexpr double kResident = 2048;  // workgroups resident at one time, about 8 per CU

double window_regions(const Fused& f, const TileArgs& t, const int* outer, int no) {
    const int M = f.M;
    double covered[kMaxDims];
    for (int d = 0; d < M; ++d) covered[d] = 1;
    // the window's count of each digit, in digit order
    double P = 1;
    auto take = [&](double e) {
        double c = P >= kResident ? 1 : (P * e <= kResident ? e : kResident / P);
        P *= c;
        return c;
    };
    double cCount = 1, rCount = 1;
    if (t.cChunk < t.cLast) cCount = take(double((t.cLast + t.cChunk - 1) / t.cChunk));
    if (t.rChunk < t.rLast) rCount = take(double((t.rLast + t.rChunk - 1) / t.rChunk));
    for (int i = 0; i < no; ++i) covered[outer[i]] = take(double(f.n[outer[i]]));
    for (int d = 0; d < t.nC; ++d)
        covered[d] = d < t.nC - 1 ? double(f.n[d])
                                  : std::min(double(f.n[d]), double(t.cChunk) * cCount);
    if (t.flatR) {
        double left = std::min(double(t.rLast), double(t.rChunk) * rCount);
        for (int j = 0; j < t.nR; ++j) {
            const double n = double(f.n[f.p[j]]);
            covered[f.p[j]] = left >= n ? n : std::max(1.0, left);
            left = left >= n ? left / n : 1;
        }
    } else {
        for (int j = 0; j < t.nR; ++j)
            covered[f.p[j]] = j < t.nR - 1 ? double(f.n[f.p[j]])
                                           : std::min(double(f.n[f.p[j]]),
                                                      double(t.rChunk) * rCount);
    }
    double total = 1;
    for (int d = 0; d < M; ++d) total *= covered[d];
    auto block = [&](const int64_t* stride, const int* order) {
        double blk = 1;
        int64_t span = 1;  // elements of the contiguous prefix when every index is whole
        for (int i = 0; i < M; ++i) {
            const int d = order[i];
            if (stride[d] != span) break;
            blk *= covered[d];
            span *= f.n[d];
            if (covered[d] < double(f.n[d])) break;
        }
        return blk;
    };
    int orderA[kMaxDims], orderB[kMaxDims];
    for (int d = 0; d < M; ++d) orderA[d] = d;
    for (int k = 0; k < M; ++k) orderB[k] = f.p[k];
    std::stable_sort(orderA, orderA + M, [&](int x, int y) { return f.sA[x] < f.sA[y]; });
    std::stable_sort(orderB, orderB + M, [&](int x, int y) { return f.sB[x] < f.sB[y]; });
    return total / block(f.sA, orderA) + total / block(f.sB, orderB);
}

bool setup_tile(const Fused& f, int elem, int64_t tA, int64_t tB, const hptt_options_t& opt,
                bool alignA, bool alignB, int64_t ldsBudget, int64_t minTile, TileArgs& t,
                hptt_plan_info_t& info, bool shear = false, bool flat = false) {
    memset(&t, 0, sizeof(t));
    const int64_t lineB = kLine / elem;
    const int M = f.M;
    const int p0 = f.p[0];  // A index that is B's stride-1 index (never 0 here)
    // Both runs need a stride-1 index (a sub-tensor whose first extent is 1
    // may have none once that index is dropped).
    if (f.sA[0] != 1 || f.sB[p0] != 1) return false;
    bool outside[kMaxDims];
    // A run: A indices 0, 1, ... (never reaching p0) while they lie back to
    // back in A, the last possibly chunked.
    int64_t inner = 1;
    int d = 0;
    while (d < p0 - 1 && inner * f.n[d] <= tA && f.sA[d + 1] == f.sA[d] * f.n[d])
        inner *= f.n[d++];
    for (int j = 0; j < M; ++j) outside[j] = j > d;
    int64_t cChunk = f.n[d];
    if (inner * f.n[d] > tA)
        cChunk = choose_chunk(inner, f.n[d], stride_gcd(f, f.sA, outside), tA, elem, alignA);
    if (cChunk == 0) return false;
    const int nC = d + 1;
    t.nC = nC;
    t.cInner = inner;
    t.cChunk = cChunk;
    t.cLast = f.n[d];
    for (int k = 0; k < nC; ++k) {
        set_div(t.cExt[k], k == nC - 1 ? cChunk : f.n[k]);
        t.cStrideB[k] = f.sB[k];
    }
    // B run: B positions 0, 1, ... up to (not into) an index of the A run,
    // while they lie back to back in B.
    inner = 1;
    int k = 0;
    while (k + 1 < M && f.p[k + 1] >= nC && inner * f.n[f.p[k]] <= tB &&
           f.sB[f.p[k + 1]] == f.sB[f.p[k]] * f.n[f.p[k]])
        inner *= f.n[f.p[k++]];
    for (int j = 0; j < M; ++j) outside[j] = true;
    for (int j = 0; j <= k; ++j) outside[f.p[j]] = false;
    int64_t rChunk = f.n[f.p[k]];
    const int64_t flatLen = inner * f.n[f.p[k]];  // the flattened B-run range
    if (flat) {
        // flat B runs: whole lines cut from positions 0..k flattened (two
        // or more of them, longer than one run)
        if (k == 0 || shear) return false;
        // the kernel splits a flattened position as a 32-bit number
        if (flatLen >= (int64_t(1) << 32)) return false;
        rChunk = tB >= lineB ? tB / lineB * lineB : lineB;
        if (rChunk >= flatLen) return false;
    } else if (shear) {
        // sheared B runs: one B-run index, chunks of whole lines, and more
        // than one chunk (a run that covers its index needs no shear)
        if (k != 0) return false;
        rChunk = tB >= lineB ? tB / lineB * lineB : lineB;
        if (rChunk >= f.n[f.p[k]]) return false;
    } else if (inner * rChunk > tB) {
        rChunk = choose_chunk(inner, f.n[f.p[k]], stride_gcd(f, f.sB, outside), tB, elem, alignB);
    }
    if (rChunk == 0) return false;
    const int nR = k + 1;
    t.nR = nR;
    t.rInner = flat ? 1 : inner;
    t.rChunk = rChunk;
    t.rLast = flat ? flatLen : f.n[f.p[k]];
    t.flatR = flat ? 1 : 0;
    for (int j = 0; j < nR; ++j) {
        set_div(t.rExt[j], j == nR - 1 && !flat ? rChunk : f.n[f.p[j]]);
        t.rStrideA[j] = f.sA[f.p[j]];
    }
    t.runA = t.cInner * t.cChunk;
    t.runB = t.rInner * t.rChunk;
    // Grid digits: chunk counters first, then the remaining indices in A order.
    bool inRun[kMaxDims] = {false};
    for (int j = 0; j < nC; ++j) inRun[j] = true;
    for (int j = 0; j < nR; ++j) inRun[f.p[j]] = true;
    int g = 0;
    uint64_t tiles = 1;
    int64_t ext[kMaxDims];
    t.gChunkC = t.gChunkR = -1;
    if (t.cChunk < t.cLast) {
        ext[g] = (t.cLast + t.cChunk - 1) / t.cChunk;
        t.gStrideA[g] = t.cChunk * f.sA[nC - 1];
        t.gStrideB[g] = t.cChunk * f.sB[nC - 1];
        t.gChunkC = g++;
    }
    if (t.rChunk < t.rLast) {
        const int a = f.p[nR - 1];
        // sheared runs start up to lineB - 1 rows early: one chunk more at most
        const int64_t span = t.rLast + (shear ? lineB - 1 : 0);
        ext[g] = (span + t.rChunk - 1) / t.rChunk;
        // a flat chunk moves B by its length; its A offsets are in the
        // tile's own row table
        t.gStrideA[g] = flat ? 0 : t.rChunk * f.sA[a];
        t.gStrideB[g] = flat ? t.rChunk * f.sB[p0] : t.rChunk * f.sB[a];
        t.gChunkR = g++;
    }
    // Outer digit order: the one whose resident window touches the fewest
    // regions of A and B (window_regions), A order unless another has at
    // most 0.8 times as many.
    int32_t gorder = opt.grid_order;
    if (gorder == 0) {
        gorder = 1;
        int outer[kMaxDims];
        const int no = outer_indices(f, inRun, 1, outer);
        const double base = window_regions(f, t, outer, no);
        double best = base;
        for (int32_t o = 2; o <= 3; ++o) {
            outer_indices(f, inRun, o, outer);
            const double r = window_regions(f, t, outer, no);
            if (r <= 0.8 * base && r < best) {
                best = r;
                gorder = o;
            }
        }
    }
    {
        int outer[kMaxDims];
        const int no = outer_indices(f, inRun, gorder, outer);
        for (int i = 0; i < no; ++i) {
            const int a = outer[i];
            ext[g] = f.n[a];
            t.gStrideA[g] = f.sA[a];
            t.gStrideB[g] = f.sB[a];
            ++g;
        }
    }
    // LDS pitch: an odd number of elements by default, so the column-wise
    // reads of the store phase spread over the LDS banks.
    int64_t pad = t.runA % 2 == 0 ? 1 : 0;
    if (opt.lds_pad > 0) pad = opt.lds_pad;
    if (opt.lds_pad < 0) pad = 0;
    t.pitch = int32_t(t.runA + pad);
    // Depth: a tile smaller than `minTile` elements stacks nZ tiles along the
    // grid index closest to contiguous in both tensors (smallest sum of
    // strides), in one LDS round, as long as kMinGrid workgroups remain.
    // Not with row passes.
    t.nZ = 1;
    t.gDepth = -1;
    const int64_t area = t.runA * t.runB;
    double tilesBefore = 1;
    for (int j = 0; j < g; ++j) tilesBefore *= double(ext[j]);
    // only tiles below half the minimum are stacked: stacking takes the
    // general variant, which cost more than it gave above that (sweep on
    // MI355X: +1.4 % with beta = 1, +2.2 % with beta = 0; the 5-D beta = 1
    // workload 5.20-5.37 -> 5.43 TB/s)
    int64_t wantZ =
        opt.depth > 0 ? opt.depth : (2 * area >= minTile ? 1 : (minTile + area - 1) / area);
    if (opt.depth == 0 && double(wantZ) > tilesBefore / kMinGrid)
        wantZ = int64_t(tilesBefore / kMinGrid);
    if (opt.row_passes > 1 || shear || flat) wantZ = 1;
    if (wantZ > 1) {
        // among the indices long enough for wantZ the one with the smallest
        // strides; if none is, the longest
        int best = -1;
        for (int j = 0; j < g; ++j) {
            if (j == t.gChunkC || j == t.gChunkR || ext[j] < 2) continue;
            const bool longJ = ext[j] >= wantZ, longB = best >= 0 && ext[best] >= wantZ;
            if (best < 0 || (longJ && !longB) ||
                (longJ == longB && (longJ ? t.gStrideA[j] + t.gStrideB[j] <
                                                t.gStrideA[best] + t.gStrideB[best]
                                          : ext[j] > ext[best])))
                best = j;
        }
        if (best >= 0) {
            const int64_t perTile = t.runB * t.pitch * elem;
            const int64_t tables = (t.runA + t.runB) * int64_t(sizeof(int64_t));
            int64_t z = wantZ < ext[best] ? wantZ : ext[best];
            if (tables + z * perTile > ldsBudget) z = (ldsBudget - tables) / perTile;
            if (z >= 2) {
                t.nZ = int32_t(z);
                t.gDepth = best;
                t.zLast = ext[best];
                t.zStrideA = t.gStrideA[best];
                t.zStrideB = t.gStrideB[best];
                ext[best] = (ext[best] + z - 1) / z;
                t.gStrideA[best] *= z;
                t.gStrideB[best] *= z;
            }
        }
    }
    info.depth = t.nZ;
    t.nG = g;
    set_tile_order(t, opt, g, ext, info);
    info.grid_order = gorder;
    for (int j = 0; j < g; ++j) {
        if (ext[j] >= (int64_t(1) << 32)) return false;
        set_div(t.gExt[j], ext[j]);
        tiles *= uint64_t(ext[j]);
        if (tiles >= (uint64_t(1) << 32)) return false;
    }
    t.numTiles = uint32_t(tiles);
    // Vector widths: A runs start at multiples of granA elements, B runs at
    // multiples of granB (relative to the tensors' first elements).
    int64_t granA = 0, granB = 0;
    for (int j = 0; j < g; ++j)
        if (ext[j] > 1) {
            granA = gcd64(granA, t.gStrideA[j]);
            granB = gcd64(granB, t.gStrideB[j]);
        }
    if (t.nZ > 1) {
        granA = gcd64(granA, t.zStrideA);
        granB = gcd64(granB, t.zStrideB);
    }
    for (int j = 0; j < nR; ++j)
        if (t.rExt[j].d > 1) granA = gcd64(granA, t.rStrideA[j]);
    for (int j = 0; j < nC; ++j)
        if (t.cExt[j].d > 1) granB = gcd64(granB, t.cStrideB[j]);
    if (shear) {
        t.shear = int32_t(lineB - 1);
        t.lineB = int32_t(lineB);
        t.rowsB = t.rLast;
        granB = lineB;  // sheared runs start on lines
    }
    info.vec_a = run_vec_width(t.runA, granA, elem, opt.max_vec);
    info.vec_b = run_vec_width(t.runB, granB, elem, opt.max_vec);
    t.runsOnGridA = granA % info.vec_a == 0 ? 1 : 0;
    t.runsOnGridB = granB % info.vec_b == 0 ? 1 : 0;
    t.misA = t.misB = 0;
    // A runs that start and end on 128-byte lines share no line with another
    // tile, so they can be read with non-temporal loads.
    t.alignedA = (granA == 0 || (granA * elem) % kLine == 0) && (t.runA * elem) % kLine == 0;
    t.alignedB = (granB == 0 || (granB * elem) % kLine == 0) && (t.runB * elem) % kLine == 0;
    info.shear = t.shear;
    info.shared_runs = 0;
    info.flat_runs = flat ? nR : 0;
    // Rows staged through LDS per pass: the whole tile by default.  Staging a
    // tile in several passes keeps its run lengths with less LDS, but each
    // pass adds a barrier round trip; on MI355X that cost more than it saved
    // (the 6-D workload: 96x160 in two passes 4.62 TB/s, 48x160 in one
    // 4.80), so passes are only taken on request.
    t.subRows = int32_t(t.runB);
    if (opt.row_passes > 1) {
        const int64_t want = (t.runB + opt.row_passes - 1) / opt.row_passes;
        t.subRows = int32_t((want + info.vec_b - 1) / info.vec_b * info.vec_b);
    }
    set_div(t.zRows, t.subRows);
    set_div(t.zCols, t.runA);
    // Largest offset inside a tile: the last row's A offset plus the run,
    // and the last column's B offset plus the B run.
    int64_t maxRowA = 0, maxColB = 0;
    for (int j = 0; j < nR; ++j) maxRowA += (int64_t(t.rExt[j].d) - 1) * t.rStrideA[j];
    for (int j = 0; j < nC; ++j) maxColB += (int64_t(t.cExt[j].d) - 1) * t.cStrideB[j];
    t.offsets32 = (maxRowA + t.runA < (int64_t(1) << 31) && maxColB + t.runB < (int64_t(1) << 31))
                      ? 1 : 0;
    const int64_t lds = tile_lds_bytes_host(t, elem);
    if (lds > ldsBudget) return false;
    info.run_a = t.runA;
    info.run_b = t.runB;
    info.dims_a = nC;
    info.dims_b = nR;
    info.lds_pitch = t.pitch;
    info.rows_per_pass = t.subRows;
    info.lds_bytes = int32_t(lds);
    info.tiles = t.numTiles;
    return true;
}

// Kernel T with runs that share indices (variant kShared), for targets tA
// (A run) and tB (B run), in elements.  The A run is A indices 0..d while
// they lie back to back in A, the last one chunked towards tA.  The B run
// walks B positions 0, 1, ... while they lie back to back in B: an index of
// the A run joins it without enlarging the tile (a shared index, S; the
// chunked A index only as the B run's last), another index (R) joins while
// the B run is below tB, the last one chunked towards it.  The tile is
// C x S x R, C being the A-run indices outside the B run.  Returns false if
// no index is shared, or the tile does not fit the LDS budget or the offsets.
bool setup_shared(const Fused& f, int elem, int64_t tA, int64_t tB, const hptt_options_t& opt,
                   int64_t ldsBudget, TileArgs& t, hptt_plan_info_t& info) {
    memset(&t, 0, sizeof(t));
    const int M = f.M;
    if (M < 2 || f.sA[0] != 1 || f.sB[f.p[0]] != 1) return false;
    int64_t inner = 1;
    int d = 0;
    while (d < M - 1 && inner * f.n[d] <= tA && f.sA[d + 1] == f.sA[d] * f.n[d])
        inner *= f.n[d++];
    bool inA[kMaxDims] = {false}, inB[kMaxDims] = {false};
    for (int j = 0; j <= d; ++j) inA[j] = true;
    int64_t cChunk = f.n[d];
    if (inner * f.n[d] > tA) {
        bool outside[kMaxDims];
        for (int j = 0; j < M; ++j) outside[j] = !inA[j];
        cChunk = choose_chunk(inner, f.n[d], stride_gcd(f, f.sA, outside), tA, elem, false);
        if (cChunk == 0) return false;
    }
    const bool chunkA = cChunk < f.n[d];
    // B run
    int64_t bInner = 1;  // B-run elements before its last position
    int64_t bRun = 1;    // B-run elements so far
    int e = 0;           // B positions in the run
    int64_t rChunk = 0;  // extent taken of the B run's last index
    for (; e < M; ++e) {
        const int a = f.p[e];
        if (e > 0 && f.sB[a] != f.sB[f.p[e - 1]] * f.n[f.p[e - 1]]) break;
        int64_t x = f.n[a];
        bool last = false;
        if (inA[a]) {
            // shared: free, but the chunked A index ends the B run
            if (a == d && chunkA) {
                x = cChunk;
                last = true;
            }
        } else {
            if (bRun >= tB) break;
            if (bRun * f.n[a] > tB) {
                bool outside[kMaxDims];
                for (int j = 0; j < M; ++j) outside[j] = j != a;
                x = choose_chunk(bRun, f.n[a], stride_gcd(f, f.sB, outside), tB, elem, false);
                if (x == 0) return false;
                last = true;
            }
        }
        inB[a] = true;
        bInner = bRun;
        rChunk = x;
        bRun *= x;
        if (last) {
            ++e;
            break;
        }
    }
    if (e == 0) return false;
    const int lastB = f.p[e - 1];
    const bool chunkB = rChunk < f.n[lastB];
    int shared = 0;
    for (int j = 0; j < M; ++j) shared += inA[j] && inB[j];
    if (shared == 0) return false;

    t.shared = 1;
    t.runA = inner * cChunk;
    t.runB = bRun;
    t.cInner = inner;
    t.cChunk = cChunk;
    t.cLast = f.n[d];
    t.rInner = bInner;
    t.rChunk = rChunk;
    t.rLast = f.n[lastB];
    // C: A-run indices outside the B run, A order
    int nC = 0;
    int64_t cols = 1;
    t.cInnerS = 0;
    for (int j = 0; j <= d; ++j) {
        if (inB[j]) continue;
        const int64_t x = j == d ? cChunk : f.n[j];
        if (j == d && chunkA) t.cInnerS = int32_t(cols);
        set_div(t.cExt[nC], x);
        t.cStrideB[nC] = f.sB[j];
        t.cLds[nC] = int32_t(f.sA[j]);
        cols *= x;
        ++nC;
    }
    t.nC = nC;
    t.nColS = int32_t(cols);
    // R: B-run indices outside the A run, B order (the load rows)
    int nR = 0;
    int64_t rows = 1;
    int64_t rowWeight[kMaxDims];
    t.rInnerL = 0;
    for (int k = 0; k < e; ++k) {
        const int a = f.p[k];
        if (inA[a]) continue;
        const int64_t x = k == e - 1 ? rChunk : f.n[a];
        if (k == e - 1 && chunkB) t.rInnerL = int32_t(rows);
        set_div(t.rExt[nR], x);
        t.rStrideA[nR] = f.sA[a];
        rowWeight[k] = rows;
        rows *= x;
        ++nR;
    }
    t.nR = nR;
    if (rows >= (int64_t(1) << 30) || cols >= (int64_t(1) << 30)) return false;
    t.subRows = int32_t(rows);
    int64_t pad = t.runA % 2 == 0 ? 1 : 0;
    if (opt.lds_pad > 0) pad = opt.lds_pad;
    if (opt.lds_pad < 0) pad = 0;
    t.pitch = int32_t(t.runA + pad);
    // B-run digits and their LDS weights
    t.nO = e;
    for (int k = 0; k < e; ++k) {
        const int a = f.p[k];
        set_div(t.oExt[k], k == e - 1 ? rChunk : f.n[a]);
        t.oLds[k] = int32_t(inA[a] ? f.sA[a] : rowWeight[k] * t.pitch);
    }
    // grid digits: the chunk counters, then the indices outside the tile
    int g = 0;
    int64_t ext[kMaxDims];
    t.gChunkC = t.gChunkR = -1;
    if (chunkA) {
        ext[g] = (f.n[d] + cChunk - 1) / cChunk;
        t.gStrideA[g] = cChunk * f.sA[d];
        t.gStrideB[g] = cChunk * f.sB[d];
        t.gChunkC = g;
        if (lastB == d) t.gChunkR = g;
        ++g;
    }
    if (chunkB && lastB != d) {
        ext[g] = (f.n[lastB] + rChunk - 1) / rChunk;
        t.gStrideA[g] = rChunk * f.sA[lastB];
        t.gStrideB[g] = rChunk * f.sB[lastB];
        t.gChunkR = g++;
    }
    {
        bool skip[kMaxDims];
        for (int a = 0; a < M; ++a) skip[a] = inA[a] || inB[a];
        int outer[kMaxDims];
        const int no = outer_indices(f, skip, grid_order(opt), outer);
        for (int i = 0; i < no; ++i) {
            const int a = outer[i];
            ext[g] = f.n[a];
            t.gStrideA[g] = f.sA[a];
            t.gStrideB[g] = f.sB[a];
            ++g;
        }
    }
    t.nZ = 1;
    t.gDepth = -1;
    t.nG = g;
    set_tile_order(t, opt, g, ext, info);
    uint64_t tiles = 1;
    for (int j = 0; j < g; ++j) {
        if (ext[j] >= (int64_t(1) << 32)) return false;
        set_div(t.gExt[j], ext[j]);
        tiles *= uint64_t(ext[j]);
        if (tiles >= (uint64_t(1) << 32)) return false;
    }
    t.numTiles = uint32_t(tiles);
    // Vector widths: rows start at multiples of granA in A, columns at
    // multiples of granB in B; runs off the vector grid are shifted onto it.
    int64_t granA = 0, granB = 0;
    for (int j = 0; j < g; ++j)
        if (ext[j] > 1) {
            granA = gcd64(granA, t.gStrideA[j]);
            granB = gcd64(granB, t.gStrideB[j]);
        }
    for (int j = 0; j < nR; ++j)
        if (t.rExt[j].d > 1) granA = gcd64(granA, t.rStrideA[j]);
    for (int j = 0; j < nC; ++j)
        if (t.cExt[j].d > 1) granB = gcd64(granB, t.cStrideB[j]);
    info.vec_a = run_vec_width(t.runA, granA, elem, opt.max_vec);
    info.vec_b = run_vec_width(t.runB, granB, elem, opt.max_vec);
    t.runsOnGridA = granA % info.vec_a == 0 ? 1 : 0;
    t.runsOnGridB = granB % info.vec_b == 0 ? 1 : 0;
    t.alignedA = (granA == 0 || (granA * elem) % kLine == 0) && (t.runA * elem) % kLine == 0;
    t.alignedB = (granB == 0 || (granB * elem) % kLine == 0) && (t.runB * elem) % kLine == 0;
    int64_t maxRowA = 0, maxColB = 0;
    for (int j = 0; j < nR; ++j) maxRowA += (int64_t(t.rExt[j].d) - 1) * t.rStrideA[j];
    for (int j = 0; j < nC; ++j) maxColB += (int64_t(t.cExt[j].d) - 1) * t.cStrideB[j];
    if (maxRowA + t.runA >= (int64_t(1) << 31) || maxColB + t.runB >= (int64_t(1) << 31))
        return false;
    t.offsets32 = 1;
    // B-run positions from an LDS table when two or more columns share it;
    // computed for single-column tiles, where the table would take as much
    // LDS as fp32 data (MI355X, 57-case sweep: single-column tiles +12 to
    // +52 % from the LDS the table no longer takes, on the same tile or a
    // larger one it allows; tiles of 2 and 5-63 columns lost 3 to 21 %
    // without the table).
    t.posTable = t.nColS >= 2 ? 1 : 0;
    const int64_t lds = tile_lds_bytes_host(t, elem);
    if (lds > ldsBudget) return false;
    info.run_a = t.runA;
    info.run_b = t.runB;
    info.dims_a = d + 1;
    info.dims_b = e;
    info.lds_pitch = t.pitch;
    info.rows_per_pass = t.subRows;
    info.lds_bytes = int32_t(lds);
    info.tiles = t.numTiles;
    info.depth = 1;
    info.shear = 0;
    info.shared_runs = shared;
    return true;
}

// Score of a tile shape for the choice between disjoint and shared runs:
// the bytes of each run up to 512 (a run shorter than a few lines wastes
// most of each HBM burst), then the tile up to kMinTileBytes, and a penalty
// for leaving most CUs idle.
double tile_score(int64_t runA, int64_t runB, int64_t tileElems, uint64_t tiles, int elem) {
    const double pa = double(runA * elem < 512 ? runA * elem : 512);
    const double pb = double(runB * elem < 512 ? runB * elem : 512);
    const double area = double(tileElems * elem < kMinTileBytes ? tileElems * elem : kMinTileBytes);
    return pa + pb + 64.0 * area / double(kMinTileBytes) - (tiles < 1024 ? 256.0 : 0.0);
}

// The best shared-run tile over a few pairs of run targets (or the
// requested ones), by tile_score.
bool choose_shared(const Fused& f, int elem, const hptt_options_t& opt, TileArgs& best,
                    hptt_plan_info_t& bestInfo, double& bestScore) {
    static const int64_t aBytes[] = {512, 1024, 2048, 4096, 8192, 16384};
    static const int64_t bBytes[] = {128, 512, 2048, 8192};
    const hptt_plan_info_t base = bestInfo;
    // best tile within an LDS budget (and at most maxRows rows, if > 0)
    auto search = [&](int64_t budget, int32_t maxRows, TileArgs& bt, hptt_plan_info_t& bi,
                      double& bs) {
        bool fnd = false;
        for (int64_t ab : aBytes)
            for (int64_t bb : bBytes) {
                const int64_t tA = opt.run_a > 0 ? opt.run_a : ab / elem;
                const int64_t tB = opt.run_b > 0 ? opt.run_b : bb / elem;
                TileArgs t;
                hptt_plan_info_t in = base;
                if (!setup_shared(f, elem, tA, tB, opt, budget, t, in)) continue;
                if (maxRows > 0 && t.subRows > maxRows) continue;
                const double sc =
                    tile_score(t.runA, t.runB, t.runA * int64_t(t.subRows), t.numTiles, elem);
                if (!fnd || sc > bs) {
                    fnd = true;
                    bs = sc;
                    bt = t;
                    bi = in;
                }
            }
        return fnd;
    };
    const bool readsB = base.mode == kAxpby;
    bool found = search(readsB ? kSharedLdsBudgetAxpby : kLdsBudget, 0, best, bestInfo, bestScore);
    // With B read, fp32 tiles of one or two rows take the larger budget too
    // (MI355X, 40 against 20 KiB: 2x26250x4x238 [1,3,0,2] 1.26x, single-row
    // tiles of 2100 -> 4040 elements; 2925x1207x2x7 [2,0,3,1] 1.13x; taller
    // tiles split from 1.10x to 0.93x, and an fp64 two-row tile lost 5 %).
    if (found && readsB && elem == 4 && best.subRows <= 2) {
        TileArgs t2;
        hptt_plan_info_t i2 = base;
        double s2 = 0;
        if (search(kLdsBudget, 2, t2, i2, s2)) {
            best = t2;
            bestInfo = i2;
            bestScore = s2;
        }
    }
    return found;
}

bool setup_stream(const Fused& f, int elem, const hptt_options_t& opt, StreamArgs& s,
                  hptt_plan_info_t& info) {
    memset(&s, 0, sizeof(s));
    if (f.sA[0] != 1 || f.sB[0] != 1) return false;
    int log = 0;
    while ((int64_t(1) << (log + 1)) <= opt.xcd_group) ++log;
    s.xcdGroupLog = log;
    info.xcd_group = 1 << log;
    s.rowLen = f.n[0];
    int64_t rows = 1;
    for (int d = 1; d < f.M; ++d) rows *= f.n[d];
    s.numRows = rows;
    s.nO = f.M - 1;
    int64_t gran = s.rowLen;  // every row starts on a multiple of gran in both tensors
    for (int k = 1; k < f.M; ++k) {
        set_div(s.oExt[k - 1], f.n[f.p[k]]);
        s.oStrideA[k - 1] = f.sA[f.p[k]];
        s.oStrideB[k - 1] = f.sB[f.p[k]];
        gran = gcd64(gran, gcd64(s.oStrideA[k - 1], s.oStrideB[k - 1]));
    }
    const int32_t v = vec_width(gran, elem, opt.max_vec);
    // Flat walk: B compact (its rows back to back), and rows that would move
    // one element per access (odd row lengths), or two fp32 elements; every
    // B access is then a whole vector.  MI355X, fp32 rows of 55-213
    // elements: +13 to +24 % (e.g. 63-element rows 3.11 -> 3.65 TB/s with
    // beta = 0, 4.25 -> 5.27 with beta = 1), and +27 to +35 % more with beta
    // = 0 since A is read a vector at a time there; fp32 rows of 42 and 66
    // (two elements per access) +12 % and +9 % with beta = 1, and with beta =
    // 0 rows of 42 and 498 +11 % and +14 % (they lost 7-9 % while A was read
    // element by element); fp64 rows of 33-211 elements +5 to +19 % with beta
    // = 0, +2 to +14 % on three of four with beta = 0.5 (-3 % on rows of 95).
    const int32_t vWide = vec_width(0, elem, opt.max_vec);
    bool compactB = f.M < 2 || f.sB[f.p[1]] == s.rowLen;
    for (int k = 1; k + 1 < f.M; ++k)
        compactB = compactB && f.sB[f.p[k + 1]] == f.sB[f.p[k]] * f.n[f.p[k]];
    const int64_t numel = rows * s.rowLen;
    if (opt.flat_runs != 2 && compactB && numel < (int64_t(1) << 32) - int64_t(kBlock) * kMaxItems &&
        s.rowLen >= vWide &&
        (opt.flat_runs == 1 ||
         (v < vWide && (v == 1 || (elem == 4 && v == 2))))) {
        s.flatB = 1;
        set_div(s.L, s.rowLen);
        for (int w = 0; w < 3; ++w) s.numItems[w] = uint32_t((numel + (1 << w) - 1) >> w);
        info.vec_a = info.vec_b = vWide;
        info.run_b = s.rowLen;
        info.tiles = s.numItems[vWide >= 4 ? 2 : vWide >= 2 ? 1 : 0];
        info.flat_runs = 1;
        return true;
    }
    // The kernel splits item and row numbers as 32-bit numbers.  Every outer
    // extent, and a row's vectors, must fit; a width whose items do not fit
    // in all keeps numItems 0, and hptt_exec launches it per slab of the
    // slowest B positions (stream_slabs), each slab's items below the limit.
    for (int k = 1; k < f.M; ++k)
        if (f.n[f.p[k]] >= (int64_t(1) << 32)) return false;
    const int64_t limit = (int64_t(1) << 32) - int64_t(kBlock) * kMaxItems;
    for (int w = 0; w < 3; ++w) {  // every width hptt_exec may launch with
        const int64_t W = (s.rowLen + (1 << w) - 1) >> w;
        if (W >= limit) return false;
        const int64_t items = rows * W;
        set_div(s.W[w], W);
        s.numItems[w] = items < limit ? uint32_t(items) : 0;
    }
    info.vec_a = info.vec_b = v;
    info.run_b = s.rowLen;
    info.tiles = rows * ((s.rowLen + v - 1) / v);
    return true;
}

void setup_generic(const Fused& f, int64_t numel, GenericArgs& g) {
    memset(&g, 0, sizeof(g));
    g.numel = numel;
    g.n = f.M;
    for (int k = 0; k < f.M; ++k) {
        const int64_t e = f.n[f.p[k]];
        g.bExt64[k] = e;
        if (e < (int64_t(1) << 32)) set_div(g.bExt[k], e);
        g.bStrideA[k] = f.sA[f.p[k]];
        g.bStrideB[k] = f.sB[f.p[k]];
    }
}

// Elements from a tensor's first to its last element, inclusive.
int64_t footprint(const Fused& f, const int64_t* stride) {
    int64_t span = 1;
    for (int d = 0; d < f.M; ++d) span += (f.n[d] - 1) * stride[d];
    return span;
}

}  // namespace

hptt_status_t build_plan(const int32_t* perm, int32_t N, const int64_t* sizeA,
                         const int64_t* outerSizeA, const int64_t* outerSizeB, double alpha,
                         double beta, hptt_dtype_t dtype, const hptt_options_t* options,
                         hptt_plan_s* plan) {
    if (!perm || !sizeA || !plan) return HPTT_ERROR_INVALID_ARGUMENT;
    if (N < 1 || N > kMaxDims) return HPTT_ERROR_INVALID_ARGUMENT;
    if (dtype != HPTT_FLOAT32 && dtype != HPTT_FLOAT64) return HPTT_ERROR_INVALID_ARGUMENT;
    bool seen[kMaxDims] = {false};
    for (int k = 0; k < N; ++k) {
        if (perm[k] < 0 || perm[k] >= N || seen[perm[k]]) return HPTT_ERROR_INVALID_ARGUMENT;
        seen[perm[k]] = true;
        if (sizeA[k] < 0) return HPTT_ERROR_INVALID_ARGUMENT;
    }
    // Enclosing extents (Fig. 3's outer sizes): each at least the extent it
    // encloses; NULL means compact.
    int64_t outerA[kMaxDims], outerB[kMaxDims];
    int64_t spanA = 1, spanB = 1;
    for (int k = 0; k < N; ++k) {
        outerA[k] = outerSizeA ? outerSizeA[k] : sizeA[k];
        outerB[k] = outerSizeB ? outerSizeB[k] : sizeA[perm[k]];
        if (outerA[k] < sizeA[k] || outerB[k] < sizeA[perm[k]]) return HPTT_ERROR_INVALID_ARGUMENT;
        if (outerA[k] > 0 && spanA > (int64_t(1) << 60) / outerA[k]) return HPTT_ERROR_INVALID_ARGUMENT;
        if (outerB[k] > 0 && spanB > (int64_t(1) << 60) / outerB[k]) return HPTT_ERROR_INVALID_ARGUMENT;
        spanA *= outerA[k] > 0 ? outerA[k] : 1;
        spanB *= outerB[k] > 0 ? outerB[k] : 1;
    }
    hptt_options_t opt;
    memset(&opt, 0, sizeof(opt));
    if (options) opt = *options;
    if (opt.kernel < HPTT_KERNEL_AUTO || opt.kernel > HPTT_KERNEL_GENERIC ||
        opt.kernel == HPTT_KERNEL_NONE || opt.run_a < 0 || opt.run_b < 0 || opt.max_vec < 0 ||
        opt.store_hint < 0 || opt.store_hint > 2 || opt.load_hint < 0 || opt.load_hint > 2 ||
        opt.lds_pad < -1 || opt.lds_pad > 64 || opt.max_blocks < 0 || opt.tile_order < 0 ||
        opt.tile_order > 4 || opt.row_passes < 0 || opt.row_passes > 64 || opt.depth < 0 ||
        opt.depth > 4096 || opt.min_tile < 0 || opt.exact_runs < 0 ||
        opt.exact_runs > 1 || (opt.block != 0 && opt.block != kBlock && opt.block != kBigBlock) ||
        opt.skew < 0 || opt.skew > 1024 || opt.shear < 0 || opt.shear > 2 || opt.shared_runs < 0 ||
        opt.shared_runs > 2 || opt.flat_runs < 0 || opt.flat_runs > 2 || opt.grid_order < 0 ||
        opt.grid_order > 3 || opt.direct_lds < 0 || opt.direct_lds > 2 || opt.xcd_group < 0 ||
        opt.xcd_group > 1024 || (opt.xcd_group & (opt.xcd_group - 1)) != 0)
        return HPTT_ERROR_INVALID_ARGUMENT;

    const int elem = dtype == HPTT_FLOAT32 ? 4 : 8;
    memset(plan, 0, sizeof(*plan));
    plan->dtype = dtype;
    plan->alpha = dtype == HPTT_FLOAT32 ? double(float(alpha)) : alpha;
    plan->beta = dtype == HPTT_FLOAT32 ? double(float(beta)) : beta;
    hptt_plan_info_t& info = plan->info;
    info.elem_bytes = elem;
    info.block = kBlock;
    info.mode = plan->beta != 0.0 ? kAxpby : (plan->alpha == 1.0 ? kCopy : kScale);
    info.hints = 0;

    int64_t numel = 1;
    bool empty = false;
    for (int d = 0; d < N; ++d) {
        if (sizeA[d] == 0) empty = true;
        else if (numel > (int64_t(1) << 60) / sizeA[d]) return HPTT_ERROR_INVALID_ARGUMENT;
        else numel *= sizeA[d];
    }
    if (empty) numel = 0;
    info.numel = numel;

    Fused f;
    if (empty) {
        f.M = N;
        for (int d = 0; d < N; ++d) {
            f.n[d] = sizeA[d];
            f.p[d] = perm[d];
        }
    } else {
        fuse(perm, N, sizeA, outerA, outerB, f);
        info.footprint_a = footprint(f, f.sA);
        info.footprint_b = footprint(f, f.sB);
    }
    info.ndim = f.M;
    for (int d = 0; d < f.M; ++d) {
        info.size[d] = f.n[d];
        info.perm[d] = f.p[d];
    }
    if (empty) {
        info.kernel = HPTT_KERNEL_NONE;
        return HPTT_SUCCESS;
    }

    // Classes: one fused index -> flat axpby (only when that index has stride
    // 1 in both tensors: a sub-tensor whose first extent is 1 can leave a
    // strided one); A's stride-1 index also B's -> stream; otherwise tiles.
    // Anything a class cannot serve goes to the generic kernel.
    const bool single = f.M == 1;
    const bool unit = f.sA[0] == 1 && f.sB[0] == 1;
    const bool kept = !single && f.p[0] == 0;
    hptt_kernel_t k = opt.kernel;
    if (k == HPTT_KERNEL_AXPBY && !(single && unit)) return HPTT_ERROR_UNSUPPORTED;
    if (k == HPTT_KERNEL_STREAM && !kept) return HPTT_ERROR_UNSUPPORTED;
    if (k == HPTT_KERNEL_TILE && single) return HPTT_ERROR_UNSUPPORTED;
    if (k == HPTT_KERNEL_AUTO) {
        if (single) k = unit ? HPTT_KERNEL_AXPBY : HPTT_KERNEL_GENERIC;
        else if (kept) k = f.n[0] * elem >= 64 ? HPTT_KERNEL_STREAM : HPTT_KERNEL_GENERIC;
        else k = HPTT_KERNEL_TILE;
    }
    const int64_t maxBlocks = opt.max_blocks > 0 ? opt.max_blocks : (int64_t(1) << 31) - 1;

    // A kept stride-1 index too short for whole rows (or any, on request)
    // is shared by the A run and the B run of a tile.
    bool sharedTile = false;
    if (kept && opt.shared_runs != 2 &&
        (opt.kernel == HPTT_KERNEL_TILE ||
         (opt.kernel == HPTT_KERNEL_AUTO && (k == HPTT_KERNEL_GENERIC || opt.shared_runs == 1)))) {
        double sc = 0;
        // A short kept index: A runs of 256 bytes and B runs of 512, tiles in
        // grid-digit order, unless the caller chose them (MI355X, four fp32
        // cases with kept extents of 2 and 3: +3 to +11 % with beta = 0, +20
        // to +23 % on three of them with beta = 1, -4 % on the fourth);
        // the usual search where that tile does not fit or holds less than
        // 8 KiB (a kept extent of 4 whose next A index is short gave 1.8 KiB
        // tiles at a third of the usual search's speed).
        hptt_options_t kopt = opt;
        bool keptTile = false;
        if (opt.run_a == 0 && opt.run_b == 0) {
            kopt.run_a = int32_t(256 / elem);
            kopt.run_b = int32_t(512 / elem);
            if (opt.tile_order == 0) kopt.tile_order = 1;
            TileArgs t;
            hptt_plan_info_t in = info;
            double ksc = 0;
            keptTile = choose_shared(f, elem, kopt, t, in, ksc) &&
                       t.runA * int64_t(t.subRows) * elem >= 8192;
            if (keptTile) {
                plan->tile = t;
                info = in;
            }
        }
        if (keptTile || choose_shared(f, elem, opt, plan->tile, info, sc)) {
            k = HPTT_KERNEL_TILE;
            sharedTile = true;
        } else if (k == HPTT_KERNEL_TILE) {
            return HPTT_ERROR_UNSUPPORTED;
        }
    }
    // disjoint runs need the stride-1 index to move
    if (k == HPTT_KERNEL_TILE && kept && !sharedTile) return HPTT_ERROR_UNSUPPORTED;
    if (sharedTile) {
        const int64_t grid = plan->tile.numTiles;
        info.grid = grid < maxBlocks ? grid : maxBlocks;
        info.block = kBlock;
        set_xcd_groups(opt, elem, info, plan->tile);
    } else if (k == HPTT_KERNEL_TILE) {
        // Tile search, in order of preference (each stage halves the longer
        // target until a tile fits): both runs on whole 128-byte lines within
        // the occupancy budget; B runs aligned, A runs cut to length; A runs
        // aligned, B runs cut to length; both cut to length; finally, both
        // aligned up to the LDS limit.  On MI355X a fourth resident
        // workgroup per CU was measured to be worth more than line-aligned A
        // runs, and aligned B runs more than aligned A runs.
        // Default targets: A runs of 512 bytes, B runs of one 128-byte line
        // (on MI355X short B runs with long A runs measured fastest: the
        // tile stays small, so more workgroups stay resident); 256-byte A
        // runs when B is read as well (the 5-D beta = 1 workload 5.42 ->
        // 5.56 TB/s, the beta = 1 sweep +1.1 %; with beta = 0 they lost).
        const int64_t tA0 =
            opt.run_a > 0 ? opt.run_a : (info.mode == kAxpby ? 256 : 512) / elem;
        const int64_t tB0 = opt.run_b > 0 ? opt.run_b : kLine / elem;
        struct Stage { bool alignA, alignB; int64_t budget; };
        const Stage forced[] = {{false, false, opt.block == kBigBlock ? kLdsMaxBig : kLdsMax}};
        const Stage stages[] = {{true, true, kLdsBudget},  {false, true, kLdsBudget},
                                {true, false, kLdsBudget}, {false, false, kLdsBudget},
                                {true, true, kLdsMax},     {false, false, kLdsMax}};
        const Stage* st = opt.exact_runs ? forced : stages;
        const int nst = opt.exact_runs ? 1 : 6;
        const int64_t minTile = opt.min_tile > 0 ? opt.min_tile : kMinTileBytes / elem;
        int64_t tA = tA0, tB = tB0;
        Stage chosen = st[0];
        bool ok = false;
        for (int s = 0; s < nst && !ok; ++s) {
            tA = tA0;
            tB = tB0;
            chosen = st[s];
            for (int attempt = 0; attempt < 24 && !ok; ++attempt) {
                ok = setup_tile(f, elem, tA, tB, opt, chosen.alignA, chosen.alignB, chosen.budget,
                                minTile, plan->tile, info);
                if (!ok) {
                    if (tA >= tB && tA > 1) tA /= 2;
                    else if (tB > 1) tB /= 2;
                    else break;
                }
            }
        }
        // A tile below minTile elements whose A run is cut short by the
        // tensor (its leading extents end before the target) lets its B run
        // grow instead, and the other way round: longer runs beat stacking.
        if (ok && opt.run_a == 0 && opt.run_b == 0 && opt.exact_runs == 0) {
            const int64_t runA = plan->tile.runA, runB = plan->tile.runB;
            if (runA * runB < minTile && double(plan->tile.numTiles) * plan->tile.nZ >= kMinGrid) {
                int64_t gA = tA, gB = tB;
                if (runA < tA) gB = (minTile + runA - 1) / runA;
                else if (runB < tB) gA = (minTile + runB - 1) / runB;
                TileArgs keep = plan->tile;
                hptt_plan_info_t keepInfo = info;
                bool grown = false;
                for (int attempt = 0; attempt < 8 && !grown && (gA != tA || gB != tB); ++attempt) {
                    grown = setup_tile(f, elem, gA, gB, opt, false, false, kLdsBudget, minTile,
                                       plan->tile, info) &&
                            plan->tile.runA * plan->tile.runB > runA * runB &&
                            double(plan->tile.numTiles) * plan->tile.nZ >= kMinGrid;
                    if (!grown) {
                        if (gB > tB) gB = gB / 2 > tB ? gB / 2 : tB;
                        else if (gA > tA) gA = gA / 2 > tA ? gA / 2 : tA;
                    }
                }
                if (grown) {
                    tA = gA;
                    tB = gB;
                } else {
                    plan->tile = keep;
                    info = keepInfo;
                }
            }
        }
        // B runs that cannot start and end on 128-byte lines leave a partly
        // written line at each end, shared with the neighbouring tile; runs
        // of four lines halve the share of such lines against one-line runs
        // (MI355X, 3251-element B rows: 64x128 tiles 1.3x faster than
        // 128x32), so the A run gives way to a longer B run.
        if (ok && !plan->tile.alignedB && opt.run_a == 0 && opt.run_b == 0 &&
            opt.exact_runs == 0) {
            const int64_t runB = plan->tile.runB;
            TileArgs keep = plan->tile;
            hptt_plan_info_t keepInfo = info;
            const int64_t lB = 4 * kLine / elem;
            bool longer = false;
            // A runs of two lines, else one (a B-run length that divides the
            // index may need the room)
            for (int64_t lA = 2 * kLine / elem; runB < lB && lA >= kLine / elem && !longer;
                 lA /= 2) {
                longer = setup_tile(f, elem, lA, lB, opt, false, false, kLdsBudget, minTile,
                                    plan->tile, info) &&
                         plan->tile.runB > runB;
                if (longer) {
                    tA = lA;
                    tB = lB;
                }
            }
            if (!longer) {
                plan->tile = keep;
                info = keepInfo;
            }
        }
        // B runs that still cannot be whole lines are sheared: each column's
        // run starts on the line at or below the chunk's first row, so no
        // line of B is written by two tiles, at the price of lineB - 1 more
        // A rows staged per tile.
        if (ok && !plan->tile.alignedB && opt.shear != 2 && opt.exact_runs == 0 &&
            opt.row_passes <= 1 && opt.depth <= 1) {
            TileArgs keep = plan->tile;
            hptt_plan_info_t keepInfo = info;
            const int64_t lineB = kLine / elem;
            int64_t sA = opt.run_a > 0 ? opt.run_a : lineB;
            int64_t sB = opt.run_b > 0 ? opt.run_b : 4 * lineB;
            bool sheared = setup_tile(f, elem, sA, sB, opt, false, false, kLdsBudget, minTile,
                                      plan->tile, info, true);
            // A stride-1 index that the one-line A-run target cuts in two,
            // followed in A by the B run's index: the whole index with B runs
            // of two lines instead, so that a tile's A rows are one
            // contiguous block (MI355X: 66x757576 [1,0] +27 % with beta = 0,
            // +8 % with beta = 1; 69x988x733 [1,2,0] +17 % and +4 %)
            if (sheared && opt.run_a == 0 && opt.run_b == 0 && f.p[0] == 1 &&
                plan->tile.nC == 1 && plan->tile.cChunk < plan->tile.cLast &&
                (plan->tile.cLast + plan->tile.cChunk - 1) / plan->tile.cChunk == 2) {
                TileArgs t2 = plan->tile;
                hptt_plan_info_t i2 = info;
                const int64_t whole = plan->tile.cLast;
                if (setup_tile(f, elem, whole, 2 * lineB, opt, false, false, kLdsBudget, minTile,
                               plan->tile, info, true) &&
                    plan->tile.cChunk == whole) {
                    sA = whole;
                    sB = 2 * lineB;
                } else {
                    plan->tile = t2;
                    info = i2;
                }
            }
            // an A run cut short by its extent lets the B run grow towards
            // the smallest tile worth a workgroup round
            const int64_t area0 = keep.runA * keep.runB * keep.nZ;
            if (sheared && opt.run_b == 0 && plan->tile.runA * plan->tile.runB < minTile) {
                TileArgs t1 = plan->tile;
                hptt_plan_info_t i1 = info;
                const int64_t want = (minTile / plan->tile.runA + lineB - 1) / lineB * lineB;
                if (!setup_tile(f, elem, sA, want, opt, false, false, kLdsBudget, minTile,
                                plan->tile, info, true)) {
                    plan->tile = t1;
                    info = i1;
                } else {
                    sB = want;
                }
            }
            // Shearing pays unless its chunks leave many row slots idle: the
            // extra chunk it may need is a large share of a short index
            // (sweep on MI355X, sheared vs unsheared: +1 to +33 % where at
            // most 13 % of the slots idle, 0 to +9 % at 19 %, -2 to -9 % at
            // 23-31 %).  opt.shear = 1 shears wherever it can.
            bool pays = sheared;
            if (sheared && opt.shear != 1) {
                const TileArgs& t = plan->tile;
                const int64_t chunks = (t.rowsB + t.shear + t.runB - 1) / t.runB;
                pays = 5 * (chunks * t.runB - t.rowsB) <= chunks * t.runB;  // idle <= 20 %
            }
            const int64_t area = plan->tile.runA * plan->tile.runB;
            if (!pays || (area < minTile && area < area0)) {
                plan->tile = keep;
                info = keepInfo;
            } else {
                tA = sA;
                tB = sB;
            }
        }
        // B runs that span two or more B indices whose inner extents are
        // not whole lines (a B stride-1 extent of 20 fp32) can only start
        // and end on lines as long runs (160 elements = 5 lines), which
        // makes the tile large; flat B runs are cut from the flattened range
        // of those indices in whole lines instead, the A offsets of their
        // rows tabled per tile.  MI355X: the 6-D fp32 workload 4.86 ->
        // 5.14 TB/s (96x32 flat tiles against 48x160), two 6-D sweep cases
        // +4 % and +14 % with beta = 0 and +3 % and +4 % with beta = 1.  The
        // A-run target stays 512 bytes when B is read: one-line B runs with
        // 256-byte A runs made tiles of 8 KiB that lost 4 % there.
        if (ok && opt.flat_runs != 2 && plan->tile.shear == 0 && plan->tile.nZ == 1 &&
            plan->tile.nR >= 2 && opt.row_passes <= 1 &&
            (opt.flat_runs == 1 ||
             (opt.exact_runs == 0 && (plan->tile.rInner * elem) % kLine != 0 &&
              (!plan->tile.alignedB || plan->tile.runB > 2 * (kLine / elem))))) {
            TileArgs keep = plan->tile;
            hptt_plan_info_t keepInfo = info;
            const int64_t fA = opt.run_a > 0 ? opt.run_a : 512 / elem;
            const int64_t fB = opt.run_b > 0 ? opt.run_b : kLine / elem;
            bool flat = false;
            // exact runs take the LDS limit, as the forced stage above does
            const int64_t fBudget = !opt.exact_runs ? kLdsBudget
                                    : opt.block == kBigBlock ? kLdsMaxBig : kLdsMax;
            for (int aligned = opt.exact_runs ? 0 : 1; aligned >= 0 && !flat; --aligned) {
                flat = setup_tile(f, elem, fA, fB, opt, aligned == 1, true, fBudget, minTile,
                                  plan->tile, info, false, true) &&
                       (plan->tile.alignedB || opt.flat_runs == 1);
            }
            if (!flat) {
                plan->tile = keep;
                info = keepInfo;
            } else {
                tA = fA;
                tB = fB;
            }
        }
        // Small problems: shorter runs (down to one 128-byte line) for more
        // tiles, so that more CUs take part.
        while (ok && opt.run_a == 0 && opt.run_b == 0 && plan->tile.numTiles < 512 &&
               !(opt.shear == 1 && plan->tile.shear > 0) &&
               (tA * elem > kLine || tB * elem > kLine)) {
            TileArgs keep = plan->tile;
            hptt_plan_info_t keepInfo = info;
            if (tA >= tB) tA /= 2;
            else tB /= 2;
            if (!setup_tile(f, elem, tA, tB, opt, chosen.alignA, chosen.alignB, kLdsMax,
                            minTile, plan->tile, info) ||
                plan->tile.numTiles <= keep.numTiles) {
                plan->tile = keep;
                info = keepInfo;
                break;
            }
        }
        // Disjoint runs whose B run is shorter than a line give way to runs
        // that share indices (a B stride-1 extent of 2 whose next B index
        // is in the A run: 8-byte B runs against runs of several lines on
        // both sides), unless those take narrower vectors; so do disjoint
        // runs with narrower vectors than shared ones (2-element A runs
        // read one element per lane: 2x22x2x11885x48 [1,2,0,3,4] 3.66 ->
        // 4.31 TB/s).  Short A runs alone stay: their rows usually follow
        // each other in A (the B run's index comes next in A), so a tile
        // still reads one contiguous block (MI355X sweep: 14x320 tiles 79 %
        // of axpby, the same data as one shared-run row per tile 42 %).
        // (not chosen by itself where a knob asks for what only disjoint
        // runs have: stacking, row passes, shear, 1024 threads, exact runs)
        const bool plain = opt.depth == 0 && opt.row_passes <= 1 && opt.shear != 1 &&
                           opt.block != kBigBlock && opt.exact_runs == 0;
        if (opt.shared_runs == 1 || (opt.shared_runs == 0 && plain)) {
            const bool shortB = ok && plan->tile.runB * elem < kLine;
            const int32_t classicVec = ok ? (info.vec_a < info.vec_b ? info.vec_a : info.vec_b) : 0;
            const int32_t widest = vec_width(0, elem, opt.max_vec);
            if (opt.shared_runs == 1 || !ok || shortB || classicVec < widest) {
                TileArgs t;
                hptt_plan_info_t in = info;
                double sc = 0;
                const bool found = choose_shared(f, elem, opt, t, in, sc);
                const int32_t sharedVec = in.vec_a < in.vec_b ? in.vec_a : in.vec_b;
                if (found && (opt.shared_runs == 1 || !ok || sharedVec > classicVec ||
                              (shortB && sharedVec == classicVec))) {
                    plan->tile = t;
                    info = in;
                    sharedTile = true;
                    ok = true;
                }
            }
        }
        if (!ok) {
            if (opt.kernel == HPTT_KERNEL_TILE) return HPTT_ERROR_UNSUPPORTED;
            k = HPTT_KERNEL_GENERIC;
        } else {
            const int64_t grid = plan->tile.numTiles;
            info.grid = grid < maxBlocks ? grid : maxBlocks;
            info.block = sharedTile ? kBlock : opt.block > 0 ? opt.block : kBlock;
            set_direct_lds(opt, elem, info, plan->tile);
            set_xcd_groups(opt, elem, info, plan->tile);
        }
    }
    if (k == HPTT_KERNEL_STREAM) {
        if (!setup_stream(f, elem, opt, plan->stream, info)) {
            if (opt.kernel == HPTT_KERNEL_STREAM) return HPTT_ERROR_UNSUPPORTED;
            k = HPTT_KERNEL_GENERIC;
        } else {
            const int64_t per = int64_t(kBlock) * items_per_lane(elem, info.vec_a);
            int64_t grid = (info.tiles + per - 1) / per;
            if (grid > (int64_t(1) << 30)) grid = int64_t(1) << 30;
            info.grid = grid < maxBlocks ? grid : maxBlocks;
        }
    }
    if (k == HPTT_KERNEL_AXPBY) {
        info.vec_a = info.vec_b = vec_width(0, elem, opt.max_vec);
        const int64_t vecs = (numel + info.vec_a - 1) / info.vec_a;
        const int64_t per = int64_t(kBlock) * items_per_lane(elem, info.vec_a);
        info.tiles = vecs;
        int64_t grid = (vecs + per - 1) / per;
        if (grid > (int64_t(1) << 30)) grid = int64_t(1) << 30;
        info.grid = grid < maxBlocks ? grid : maxBlocks;
    }
    if (k == HPTT_KERNEL_GENERIC) {
        setup_generic(f, numel, plan->generic);
        info.vec_a = info.vec_b = 1;
        info.tiles = numel;
        int64_t grid = (numel + kBlock - 1) / kBlock;
        if (grid > 65536) grid = 65536;
        info.grid = grid < maxBlocks ? grid : maxBlocks;
    }
    // Cache hints.  Every element is touched once, so by default B is written
    // and A read with non-temporal hints, except runs that share 128-byte
    // lines with a neighbouring tile: an A line read non-temporally is gone
    // when the neighbour wants it, and a partly written B line stored
    // non-temporally reaches HBM as a partial write instead of being merged
    // with the neighbour's part in L2 (2-3.5x slower on MI355X).
    // (the flat walk of kernel S reads A element by element, lines shared
    // between neighbouring vectors)
    const bool loadOk = (k != HPTT_KERNEL_TILE || plan->tile.alignedA) &&
                        !(k == HPTT_KERNEL_STREAM && plan->stream.flatB);
    // Shared-run tiles with B runs of 2 KiB or more store non-temporally
    // even where the runs are not whole lines: the two partly written lines
    // at a run's ends are then a small share of it (MI355X, six sweep cases
    // with 4.5-16 KiB B runs: +3 to +5 % against ordinary stores, with
    // beta = 0 and 1; a 560-byte run lost 1 %).
    const bool storeOk = k != HPTT_KERNEL_TILE || plan->tile.alignedB ||
                         (plan->tile.shared && plan->tile.runB * elem >= 2048);
    const bool ntStore = opt.store_hint == 1 || (opt.store_hint == 0 && storeOk);
    const bool ntLoad = opt.load_hint == 1 || (opt.load_hint == 0 && loadOk && k != HPTT_KERNEL_GENERIC);
    info.hints = (ntStore ? kNtStore : 0) | (ntLoad ? kNtLoad : 0);
    info.kernel = k;
    return HPTT_SUCCESS;
}

void describe_plan(const hptt_plan_s* p, char* buf, size_t len) {
    static const char* kKernel[] = {"auto", "none", "axpby", "stream", "tile", "generic"};
    static const char* kMode[] = {"copy", "scale", "axpby"};
    const hptt_plan_info_t& in = p->info;
    char shape[256] = "", perm[256] = "";
    size_t a = 0, b = 0;
    for (int d = 0; d < in.ndim; ++d) {
        a += snprintf(shape + a, sizeof(shape) - a, "%s%lld", d ? "," : "", (long long)in.size[d]);
        b += snprintf(perm + b, sizeof(perm) - b, "%s%d", d ? "," : "", in.perm[d]);
    }
    snprintf(buf, len,
             "kernel=%s dtype=%s mode=%s fused=(%s) perm=(%s) run_a=%lld run_b=%lld "
             "dims_a=%d dims_b=%d vec=%d/%d pitch=%d rows=%d lds=%d tiles=%lld grid=%lld block=%d "
             "hints=%d order=%d shear=%d shared=%d flat=%d gorder=%d dlds=%d xg=%d",
             kKernel[in.kernel], p->dtype == HPTT_FLOAT32 ? "f32" : "f64", kMode[in.mode], shape,
             perm, (long long)in.run_a, (long long)in.run_b, in.dims_a, in.dims_b, in.vec_a,
             in.vec_b, in.lds_pitch, in.rows_per_pass, in.lds_bytes, (long long)in.tiles,
             (long long)in.grid,
             in.block, in.hints, in.tile_order, in.shear, in.shared_runs, in.flat_runs,
             in.grid_order, in.direct_lds, in.xcd_group);
}

}  // namespace hptt
