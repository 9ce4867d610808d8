// Kernel argument blocks of the transposition library.  The plan builder
// (plan.cpp) fills them once per plan; hptt_exec passes them by value to the
// kernels (kernels.hip), whose bodies live in kernel_body.h.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace hptt {

constexpr int kMaxDims = 16;  // = HPTT_MAX_DIMS
constexpr int kBlock = 256;   // threads per workgroup: 4 waves of 64
constexpr int kBigBlock = 1024;  // kernel T's large workgroup: 16 waves, for large tiles
// Vectors of v elements per lane of the streaming kernels: one 16-byte
// vector's worth, so a lane keeps 16 bytes in flight at any width.  Measured
// on MI355X: with 16-byte vectors one per lane beats four (96^4 fp64 rows
// 5.96 vs 5.49 TB/s, a flat fp64 copy 6.38 vs 5.85), and with one element
// per vector four per lane beat one, two or sixteen.
constexpr int items_per_lane(int elem, int v) { return 16 / (elem * v) > 1 ? 16 / (elem * v) : 1; }
constexpr int kMaxItems = 4;  // items_per_lane(4, 1): the most any width takes
constexpr int kXcds = 8;      // MI355X: workgroups are dealt to 8 XCDs round robin

// Unsigned division of n < 2^32 by a divisor 1 <= d < 2^32 fixed at plan
// time, with one 32x32->64 multiply and a shift (Granlund and Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994, the
// unsigned round-up method): l = ceil(log2 d),
// m = floor(2^32 * (2^l - d) / d) + 1, and n / d = (mulhi(n, m) + n) >> l.
struct FastDiv {
    uint32_t d;
    uint32_t m;
    uint32_t l;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d;
    uint32_t l = 0;
    while (l < 32 && (uint64_t(1) << l) < d) ++l;
    f.l = l;
    f.m = uint32_t((((uint64_t(1) << l) - d) << 32) / d + 1);
    return f;
}

__host__ __device__ __forceinline__ uint32_t fast_div(uint32_t n, const FastDiv& f) {
    uint32_t t = uint32_t((uint64_t(n) * f.m) >> 32);
    return uint32_t((uint64_t(t) + n) >> f.l);
}

// How B is updated (Eq. 1): a raw bit copy (alpha = 1, beta = 0), a scaled
// copy (beta = 0, B not read) or the full update alpha*A + beta*B.
enum Mode : int { kCopy = 0, kScale = 1, kAxpby = 2 };

// Cache hints of the kernels: bit 0 = non-temporal stores of B, and
// non-temporal loads of B where it is read (its lines are then whole, so no
// other workgroup reads them; MI355X, beta = 1: the 5-D fp32 workload +8 %,
// the 4-D fp64 row walk +5 %, the 57-case sweep +3.6 %), bit 1 =
// non-temporal loads of A.
constexpr int kNtStore = 1;
constexpr int kNtLoad = 2;

// Kernel T: the transposition is cut into independent 2-D tiles (the
// macro-tiles of Section 3.2).  A tile's columns form a contiguous run of A
// (fused A indices 0..nC-1, the last one possibly cut into chunks) and its
// rows a contiguous run of B (fused B positions 0..nR-1, the last one
// possibly chunked); every other index, and the chunk counters, span the grid.
struct TileArgs {
    int64_t runA;        // columns per tile = length of each A run (elements)
    int64_t runB;        // rows per tile = length of each B run
    int32_t pitch;       // LDS row pitch in elements (runA plus padding)
    int32_t nC;          // fused A indices inside the A run (A order)
    int32_t nR;          // fused B positions inside the B run (B order)
    int32_t nG;          // grid digits (fastest first)
    uint32_t numTiles;
    int32_t gChunkC;     // grid digit that counts chunks of the last A-run index, or -1
    int32_t gChunkR;     // grid digit that counts chunks of the last B-run index, or -1
    int32_t skew;        // s > 0: grid digit 1 is shifted by s times digit 0 (diagonal order)
    int32_t xcdSplit;    // 1: tile numbers dealt so that each XCD gets a contiguous range
    int32_t xcdGroupLog; // L > 0 (without xcdSplit): each XCD takes 2^L consecutive tiles at a time
    int32_t alignedA;    // 1 when every A run is whole 128-byte lines (set by the plan builder)
    int32_t alignedB;    // 1 when every B run is whole 128-byte lines
    int32_t subRows;     // rows staged through LDS per pass (runB, or runB / passes)
    // Depth: nZ tiles that differ only in one more index are staged together
    // (stacked rows z*subRows + r in LDS), so that tiles of a few hundred
    // elements still give a workgroup a few thousand.  nZ = 1: no depth.
    int32_t nZ;
    int32_t gDepth;      // grid digit that counts chunks of nZ along that index, or -1
    int64_t zLast;       // extent of that index
    int64_t zStrideA;    // its stride in A
    int64_t zStrideB;    // its stride in B
    FastDiv zRows;       // subRows: splits a stacked row into (depth, row)
    FastDiv zCols;       // runA: splits a stacked column into (depth, column)
    // Vector grid.  runsOnGridA = 1 when every A run starts on a multiple of
    // the A vector width (plan time); misA = element offset of the A base
    // pointer from that grid (launch time).  Otherwise each run's vectors are
    // shifted onto the grid, with partial vectors at both ends.  Same for B.
    int32_t runsOnGridA, runsOnGridB;
    int32_t misA, misB;
    // 1 when every offset inside a tile (table entry plus position in the
    // run) is below 2^31, so the specialised variant can use 32-bit offsets.
    int32_t offsets32;
    // Sheared B runs (variants kShifted and kGeneral; one B-run index, no
    // stacking, no row passes).  With shear = lineB - 1 > 0 the B run of column q starts at
    // the 128-byte line of B at or below the chunk's first row, i.e. it is
    // shifted back by d_q = (B address of the column, in elements) mod lineB,
    // so every line of B is written whole by one tile; the tile stages shear
    // rows more (staged row R holds run index rowBase + R - shear, rowBase =
    // j * runB for chunk j) and the run's index of extent rowsB has one
    // chunk more.  misLineB = element offset of the B base pointer from a
    // line (launch time).
    int32_t shear;
    int32_t lineB;
    int32_t misLineB;
    int64_t rowsB;
    // Flat B runs (variants kFast, kShifted and kGeneral; no stacking, no
    // shear).  With flatR = 1 the B run is a chunk of runB consecutive
    // positions of the flattened range of B positions 0..nR-1 (each whole,
    // back to back in B, rLast positions in all), not of its last index
    // alone: a B stride-1 extent that is not a multiple of a 128-byte line
    // then still gives one-line B runs.  rExt holds the whole extents,
    // rInner = 1, rChunk = runB; the chunk digit moves B by runB and A by
    // nothing, and rowOffA is rebuilt for every tile from the chunk's first
    // flattened position (TileBase::rowBase).
    int32_t flatR;
    // Direct LDS loads (variant kDirect: B only written, 16-byte A vectors,
    // one pass, no stacking or shear, every tile's columns whole vectors):
    // with directLds = 1 tiles are fetched with global_load_lds_dwordx4,
    // straight from A into an unpadded LDS tile (tile_load_direct), and
    // written out by tile_store_rotated, wherever the launch would take
    // variant kFast.
    int32_t directLds;
    // Shared runs (variant kShared): the A run and the B run share
    // indices (S).  The tile is the product of the indices of both runs.  Its
    // load phase stages subRows rows, one per value of the B-run indices
    // outside the A run (R, B order, digits rExt / rStrideA), each the whole
    // A run; its store phase writes nColS columns, one per value of the A-run
    // indices outside the B run (C, A order, digits cExt / cStrideB), each the
    // whole B run, reading B-run position b of column c from LDS at
    // pos(b) + ldsCol[c].  ldsCol sums cLds (a C index's position weight in
    // the A run); pos decodes b over the B-run digits oExt (B order) with
    // weights oLds (an S index's position weight in the A run, or pitch times
    // an R index's weight among the rows): from an LDS table ldsRow built
    // once per workgroup when posTable = 1 (many columns share it), else
    // computed per vector (a table as long as the B run would take as much
    // LDS as the tile's own data).  cInnerS / rInnerL: the C
    // columns / R rows before the chunked A-run / B-run index when that index
    // is in C / R, else 0 (every column / row of a tile exists).
    int32_t shared;
    int32_t posTable;
    int32_t nColS;
    int32_t nO;
    int32_t cInnerS;
    int32_t rInnerL;
    int32_t cLds[kMaxDims];
    FastDiv oExt[kMaxDims];
    int32_t oLds[kMaxDims];
    int64_t cInner, cChunk, cLast;  // valid columns = cInner * min(cChunk, cLast - j*cChunk)
    int64_t rInner, rChunk, rLast;  // valid rows    = rInner * min(rChunk, rLast - j*rChunk)
    FastDiv cExt[kMaxDims];         // tile extents of the A-run indices
    int64_t cStrideB[kMaxDims];     // their strides in B
    FastDiv rExt[kMaxDims];         // tile extents of the B-run indices
    int64_t rStrideA[kMaxDims];     // their strides in A
    FastDiv gExt[kMaxDims];         // grid digit extents
    int64_t gStrideA[kMaxDims];     // grid digit strides in A
    int64_t gStrideB[kMaxDims];     // grid digit strides in B
};

// Kernel S: A's stride-1 index is also B's.  Each "row" is one full run of
// that index, contiguous in both tensors.  Work item i = r*W + c is vector c
// of row r (rows in B order, W vectors per row), so consecutive lanes write
// consecutive B vectors and read whole rows of A.
// hptt_exec may narrow the vector width V for less aligned pointers, so the
// plan keeps W and the item count for each width: entry log2(V).
struct StreamArgs {
    int64_t rowLen;             // extent of the kept stride-1 index
    int64_t numRows;            // numel / rowLen
    uint32_t numItems[3];       // numRows * W for V = 1, 2, 4 (flat: ceil(numel / V))
    // Flat walk (B compact, numel < 2^32): item i is B's vector i, elements
    // [i*V, i*V + V) of the flat B range, whatever the row length; its
    // elements come from at most two rows (rowLen >= V), read from A one by
    // one.  L divides a flat B offset into (row, column).
    int32_t flatB;
    // L > 0: the workgroups one XCD receives take block numbers 2^L
    // consecutive at a time (xcd_group_map), so that blocks reading
    // neighbouring rows of A share an L2
    int32_t xcdGroupLog;
    FastDiv L;
    int32_t nO;                 // outer B positions 1..N'-1
    FastDiv W[3];               // vectors per row for V = 1, 2, 4
    FastDiv oExt[kMaxDims];     // extents of B positions 1.. (B order)
    int64_t oStrideA[kMaxDims]; // A strides of the indices at those positions
    int64_t oStrideB[kMaxDims]; // B strides of those positions
};

// Compiled variants of kernel T, picked per launch by tile_variant():
// kFast when every run starts on its vector grid for the actual pointers,
// kShifted when some do not (runs shifted onto the grid, partial vectors at
// both ends) or B runs are sheared onto lines, both with 32-bit offsets
// inside a tile and no stacking; kGeneral otherwise (stacked tiles, 64-bit
// offsets).  kShared serves the plans whose runs share indices (32-bit
// offsets, runs shifted onto the vector grid where they start off it).
// kDirect serves what kFast serves when the plan asks for direct LDS loads
// (TileArgs::directLds).  g.misA / g.misB must already hold the launch's
// pointer offsets.
enum TileVariant : int { kFast = 0, kShifted = 1, kGeneral = 2, kShared = 3, kDirect = 4 };

__host__ __device__ inline int tile_variant(const TileArgs& g) {
    if (g.shared) return kShared;
    if (g.nZ > 1 || !g.offsets32) return kGeneral;
    if (!g.runsOnGridA || !g.runsOnGridB || g.misA != 0 || g.misB != 0 || g.shear > 0)
        return kShifted;
    return g.directLds ? kDirect : kFast;
}

constexpr int log2_width(int v) { return v >= 4 ? 2 : v >= 2 ? 1 : 0; }

// Fallback: one element per thread in B order, any shape.
struct GenericArgs {
    int64_t numel;
    int32_t n;                  // fused rank
    int32_t pad_;
    FastDiv bExt[kMaxDims];     // extents of B positions (used when numel < 2^32)
    int64_t bExt64[kMaxDims];   // the same extents as 64-bit values
    int64_t bStrideA[kMaxDims]; // A stride of the index at each B position
    int64_t bStrideB[kMaxDims]; // B stride of each B position
};

}  // namespace hptt
