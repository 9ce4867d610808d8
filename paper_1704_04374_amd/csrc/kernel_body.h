// Work of each kernel, split at its workgroup barriers into per-thread phase
// functions.  The __global__ wrappers in kernels.hip call the phases with a
// barrier between them; every global and LDS access goes through the memory
// policy `Mem`, which on the device is a plain load or store.
//
// Index arithmetic is hoisted out of the per-element path: each tile
// workgroup builds its offset tables once and its sweeps step their (row,
// column) position incrementally; the streaming kernels split a lane's item
// number with plan-time magic-number division, once per 16-byte vector.
#pragma once

#include "hptt_args.h"

namespace hptt {

template <typename T, int V>
struct alignas(sizeof(T) * V) Vec {
    T v[V];
};

// One element of Eq. (1).  alpha*a and beta*b are rounded separately and then
// added; contraction into a fused multiply-add is switched off so the result
// is the same on every device.
template <int MODE, typename T>
__host__ __device__ __forceinline__ T update(T a, T b, T alpha, T beta) {
#pragma clang fp contract(off)
    if (MODE == kCopy) return a;
    if (MODE == kScale) return alpha * a;
    T x = alpha * a;
    T y = beta * b;
    return x + y;
}

template <typename I>
__host__ __device__ __forceinline__ I imin(I a, I b) { return a < b ? a : b; }

// ---------------------------------------------------------------------------
// Kernel T: 2-D tile staged through LDS
// ---------------------------------------------------------------------------

struct TileBase {
    int64_t a;           // offset of the tile's first element in A
    int64_t b;           // offset of the tile's first element in B
    int64_t validCols;   // columns (A-run elements) inside the tensor
    int64_t validRows;   // rows (B-run elements) inside the tensor
    int64_t validDepth;  // stacked tiles inside the tensor
    int64_t rowBase;     // sheared B runs: run index of the chunk's first row
    // shared runs: validCols is the valid length of the A run and
    // validRows the valid load rows; these two are the valid length of the B
    // run and the valid store columns
    int64_t validRunB;
    int64_t validColsS;
};

// Split the tile number into grid digits (fastest first).  With g.skew = s the
// second digit is rotated by the first (j1 <- (j1 + s*j0) mod n1), a bijection
// of the tiles: workgroups that run at the same time then start their B runs
// (and A runs) at many different offsets modulo a power-of-two stride instead
// of one, which spreads their traffic over the HBM channels.
//
// With g.xcdSplit the workgroup number is first mapped so that the workgroups
// one XCD receives (numbers x, x + 8, x + 16, ...) take a contiguous range of
// tile numbers: tiles that share cache lines then share an L2.  With
// g.xcdGroupLog = L instead, XCD x takes 2^L consecutive tile numbers at a
// time: round n of 8 * 2^L workgroups gives XCD x the tiles from
// (8n + x) * 2^L on, so neighbouring tiles share an L2 while the tiles in
// flight remain a near-contiguous range; the last, incomplete round keeps
// the plain numbering (a bijection either way).
__host__ __device__ inline uint32_t xcd_group_map(uint32_t t, uint32_t n, uint32_t L) {
    const uint32_t span = uint32_t(kXcds) << L;
    if (t < n / span * span) {
        const uint32_t x = t % kXcds, i = t / kXcds;
        t = (i >> L) * span + (x << L) + (i & ((1u << L) - 1u));
    }
    return t;
}

template <bool OVL = false>
__host__ __device__ inline TileBase tile_base(const TileArgs& g, uint32_t t) {
    if (g.xcdSplit) {
        const uint32_t x = t % kXcds, i = t / kXcds;
        const uint32_t q = g.numTiles / kXcds, r = g.numTiles % kXcds;
        t = x * q + (x < r ? x : r) + i;
    } else if (g.xcdGroupLog) {
        t = xcd_group_map(t, g.numTiles, uint32_t(g.xcdGroupLog));
    }
    TileBase tb;
    tb.a = 0;
    tb.b = 0;
    tb.validCols = g.runA;
    tb.validRows = OVL ? int64_t(g.subRows) : g.runB;
    tb.validDepth = g.nZ;
    tb.rowBase = 0;
    tb.validRunB = g.runB;
    tb.validColsS = g.nColS;
    uint32_t j0 = 0;
    for (int k = 0; k < g.nG; ++k) {
        uint32_t q = fast_div(t, g.gExt[k]);
        uint32_t jj = t - q * g.gExt[k].d;
        t = q;
        if (k == 0) j0 = jj;
        if (k == 1 && g.skew) {
            // with XCD groups the rotation advances once per group, so that
            // a group's tiles are neighbours along digit 0
            const uint32_t js = (j0 >> g.xcdGroupLog) * uint32_t(g.skew);  // below 2^32 (plan)
            const uint32_t r = js - fast_div(js, g.gExt[1]) * g.gExt[1].d;  // (s*j0) mod n1
            jj += r;
            if (jj >= g.gExt[1].d) jj -= g.gExt[1].d;
        }
        const int64_t j = int64_t(jj);
        tb.a += j * g.gStrideA[k];
        tb.b += j * g.gStrideB[k];
        if (k == g.gChunkC) {
            const int64_t m = imin(g.cChunk, g.cLast - j * g.cChunk);
            tb.validCols = g.cInner * m;
            if (OVL && g.cInnerS) tb.validColsS = g.cInnerS * m;
        }
        if (OVL && k == g.gChunkR) {
            // the chunked B-run index is the last of the B run, and of the
            // load rows when it is not in the A run
            const int64_t m = imin(g.rChunk, g.rLast - j * g.rChunk);
            tb.validRunB = g.rInner * m;
            if (g.rInnerL) tb.validRows = g.rInnerL * m;
        }
        if (!OVL && k == g.gChunkR) {
            // a sheared chunk reaches shear rows back and always has work
            // (its count is that of the rows plus shear), so it takes one
            // full pass; its rows are checked one by one
            tb.validRows = g.shear ? g.runB : g.rInner * imin(g.rChunk, g.rLast - j * g.rChunk);
            tb.rowBase = j * g.runB;
        }
        if (k == g.gDepth) tb.validDepth = imin(int64_t(g.nZ), g.zLast - j * g.nZ);
    }
    return tb;
}

// Offset tables shared by every tile of the launch: rowOffA[r] is the A
// offset of row r (a B-run position) and colOffB[c] the B offset of column c
// (an A-run position), both relative to the tile origin.  With sheared B
// runs the row table covers the shear rows before the chunk too:
// rowOffA[R] is the offset of run index R - shear (one B-run index).
template <class Mem, int BLOCK = kBlock>
__host__ __device__ inline void tile_tables(const TileArgs& g, int tid, int64_t* rowOffA,
                                            int64_t* colOffB) {
    // flat B runs: the row table belongs to one tile (tile_rows_flat)
    for (int64_t r = tid; r < (g.flatR ? 0 : g.runB + g.shear); r += BLOCK) {
        int64_t off = 0;
        if (g.shear) {
            off = (r - g.shear) * g.rStrideA[0];
        } else {
            uint32_t x = uint32_t(r);
            for (int k = 0; k < g.nR; ++k) {
                uint32_t q = fast_div(x, g.rExt[k]);
                off += int64_t(x - q * g.rExt[k].d) * g.rStrideA[k];
                x = q;
            }
        }
        Mem::template lds_st<int64_t>(rowOffA, r, off);
    }
    for (int64_t c = tid; c < g.runA; c += BLOCK) {
        uint32_t x = uint32_t(c);
        int64_t off = 0;
        for (int k = 0; k < g.nC; ++k) {
            uint32_t q = fast_div(x, g.cExt[k]);
            off += int64_t(x - q * g.cExt[k].d) * g.cStrideB[k];
            x = q;
        }
        Mem::template lds_st<int64_t>(colOffB, c, off);
    }
}

// Row table of one tile with flat B runs: rowOffA[r] = A offset of
// flattened B-run position rowBase + r, split into the B-run digits, for the
// tile's valid rows.  The caller puts a barrier between the previous tile's
// load phase and this call, and another before the next load phase.
template <class Mem, int BLOCK = kBlock>
__host__ __device__ inline void tile_rows_flat(const TileArgs& g, const TileBase& tb, int tid,
                                               int64_t* rowOffA) {
    for (int64_t r = tid; r < tb.validRows; r += BLOCK) {
        uint32_t x = uint32_t(tb.rowBase + r);
        int64_t off = 0;
        for (int k = 0; k < g.nR; ++k) {
            const uint32_t q = fast_div(x, g.rExt[k]);
            off += int64_t(x - q * g.rExt[k].d) * g.rStrideA[k];
            x = q;
        }
        Mem::template lds_st<int64_t>(rowOffA, r, off);
    }
}

// LDS layout of the shared-run variant, in 64-bit words: rowOffA
// (subRows), colOffB (nColS), then the 32-bit ldsCol (nColS) and, with
// posTable, ldsRow (runB), then the subRows rows of the tile.
__host__ __device__ inline int64_t shared_table_words(const TileArgs& g) {
    return int64_t(g.subRows) + g.nColS + (g.nColS + (g.posTable ? g.runB : 0) + 1) / 2;
}

// LDS offset, in column 0, of B-run position b of a shared-run tile: b split
// over the B-run digits oExt (B order), each digit weighted by oLds.  d0
// returns b's first digit.
__host__ __device__ inline int32_t shared_pos(const TileArgs& g, uint32_t b, uint32_t& d0) {
    int32_t off = 0;
    d0 = 0;
    for (int k = 0; k < g.nO; ++k) {
        const uint32_t q = fast_div(b, g.oExt[k]);
        const uint32_t d = b - q * g.oExt[k].d;
        if (k == 0) d0 = d;
        off += int32_t(d) * g.oLds[k];
        b = q;
    }
    return off;
}

// LDS offsets (column 0) of B-run positions ss .. ss + V - 1 that lie in
// [0, rows): from the table ldsRow, or each split on its own (a step of the
// first digit with a split only where it wraps measured no better: the wrap
// branch diverges across lanes).
template <class Mem, int V>
__host__ __device__ inline void shared_positions(const TileArgs& g, const int32_t* ldsRow, int ss,
                                                 int rows, int32_t* pos) {
#pragma unroll
    for (int e = 0; e < V; ++e) {
        if (ss + e < 0 || ss + e >= rows) continue;
        uint32_t d0;
        pos[e] = g.posTable ? Mem::template lds_ld<int32_t>(ldsRow, ss + e)
                            : shared_pos(g, uint32_t(ss + e), d0);
    }
}

// Tables of the shared-run variant, shared by every tile of the launch:
// rowOffA[r] = A offset of load row r (the R digits), colOffB[c] = B offset
// of store column c (the C digits), ldsCol[c] = its position in the A run,
// and with posTable ldsRow[b] = the LDS offset of B-run position b in
// column 0.
template <class Mem, int BLOCK = kBlock>
__host__ __device__ inline void tile_tables_shared(const TileArgs& g, int tid, int64_t* rowOffA,
                                                    int64_t* colOffB, int32_t* ldsCol,
                                                    int32_t* ldsRow) {
    for (int64_t r = tid; r < g.subRows; r += BLOCK) {
        uint32_t x = uint32_t(r);
        int64_t off = 0;
        for (int k = 0; k < g.nR; ++k) {
            const uint32_t q = fast_div(x, g.rExt[k]);
            off += int64_t(x - q * g.rExt[k].d) * g.rStrideA[k];
            x = q;
        }
        Mem::template lds_st<int64_t>(rowOffA, r, off);
    }
    for (int64_t c = tid; c < g.nColS; c += BLOCK) {
        uint32_t x = uint32_t(c);
        int64_t offB = 0;
        int32_t offL = 0;
        for (int k = 0; k < g.nC; ++k) {
            const uint32_t q = fast_div(x, g.cExt[k]);
            const uint32_t digit = x - q * g.cExt[k].d;
            offB += int64_t(digit) * g.cStrideB[k];
            offL += int32_t(digit) * g.cLds[k];
            x = q;
        }
        Mem::template lds_st<int64_t>(colOffB, c, offB);
        Mem::template lds_st<int32_t>(ldsCol, c, offL);
    }
    if (g.posTable)
        for (int64_t b = tid; b < g.runB; b += BLOCK) {
            uint32_t d0;
            Mem::template lds_st<int32_t>(ldsRow, b, shared_pos(g, uint32_t(b), d0));
        }
}

// Vectors a lane loads before the first of them is written to LDS (4, 8 and
// 16 measured within noise of each other on MI355X; 8 was best on average).
constexpr int kBatch = 8;

// Batch of the specialised tile phases for a workgroup of BLOCK threads: a
// 1024-thread workgroup (16 waves) keeps fewer vectors per lane, so that two
// of them fit a CU's registers (at most 64 VGPRs per lane).
constexpr int tile_batch(int block) { return block >= 1024 ? 4 : kBatch; }

// Batch of the specialised store phase when it also reads B (beta != 0):
// its B vectors double the registers a batch holds.  2 in variant kFast (its
// 8 waves per SIMD; 3 or 4 lost 2-3 % on the 5-D and 6-D fp32 workloads),
// 4 in kShifted and kShared, which run 7 waves either way (MI355X, beta = 1
// sweep cases: sheared runs +1 % on average, shared runs +3 to +6 %).
constexpr int axpby_store_batch(int var) { return var == kShifted || var == kShared ? 4 : 2; }

// Batch of the specialised load phase: 4 in variant kFast when B is read as
// well, so that it fits 8 waves per SIMD (the attribute in tile_kernel.h)
// without spilling vector registers; tile_batch otherwise.
constexpr int tile_load_batch(int mode, int var, int block) {
    return mode == kAxpby && var == kFast && block < 1024 ? 4 : tile_batch(block);
}

// Partial vectors at the ends of A runs are fetched whole, as the aligned
// vector that holds them (ld_part), where B is only written: one load
// instead of up to four element loads, each of which the whole wave issues
// (MI355X, against element loads: the beta = 0 sweep +2.2 % on average, up
// to +11 %, 2193x22800 [1,0] +10 %; with beta = 1, B's vectors being read as
// well, the sweep moved by -4 to +3 %, 1.000x on average, and keeps element
// loads).
constexpr bool tile_part_loads(int mode, int) { return mode != kAxpby; }

// Specialised load phase (variant kFast, or kShifted with SHIFT): nZ = 1 and
// offsets inside a tile fit 32 bits, so the per-vector
// arithmetic is 32-bit around one 64-bit tile base pointer.  Without SHIFT
// every run starts on the A vector grid; with SHIFT a run that starts off it
// is covered by one more vector, its first and last ones partial, and
// sheared B runs stage g.shear rows more.  The second sweep of a batch
// recomputes each vector's position from the
// batch's start instead of keeping it (only the shifted column is kept), so
// little besides the data stays live between the two (fewer registers, more
// resident waves).  Same thread-to-vector map as tile_load.
template <class Mem, typename T, int VA, int HINT, int BLOCK, bool SHIFT, int NB, bool PARTV>
__host__ __device__ inline void tile_load_fast(const TileArgs& g, const TileBase& tb, int r0,
                                               int tid, const T* A, T* lds,
                                               const int64_t* rowOffA) {
    const bool shift = SHIFT && (!g.runsOnGridA || g.misA != 0);
    const int W = (int(g.runA) + (shift ? VA - 1 : 0) + VA - 1) / VA;  // vectors per row
    const int rows = int(imin(int64_t(g.subRows), tb.validRows - r0));
    const int vcols = int(tb.validCols);
    const T* Ab = A + tb.a;
    // element offset of the tile origin from the A vector grid
    const int ta = shift ? int((tb.a + g.misA) & (VA - 1)) : 0;
    // sheared B runs: staged row R holds run index rowBase + R - sh, which
    // must lie in [0, rowsB); otherwise row R exists when R < rows
    const int sh = SHIFT ? g.shear : 0;
    const int staged = g.subRows + sh;
    const int rLo = sh ? sh - int(tb.rowBase) : 0;
    const int rHi = sh ? int(g.rowsB - tb.rowBase) + sh : rows;
    int R = tid / W, c = tid % W;
    const int dR = BLOCK / W, dc = BLOCK % W;
    while (R < staged) {
        Vec<T, VA> v[NB];
        int ccs[SHIFT ? NB : 1];
        const int R0 = R, c0 = c;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            int cc = c * VA;
            if (R >= rLo && R < rHi && R < staged) {
                const int rowOff = int(Mem::template lds_ld<int64_t>(rowOffA, r0 + R));
                if (shift) cc -= (ta + rowOff) & (VA - 1);
                const int off = rowOff + cc;
                if (cc >= 0 && cc + VA <= vcols) {
                    v[u] = Mem::template ld<T, VA, (HINT & kNtLoad) != 0>(Ab, off);
                } else if (PARTV && cc + VA > 0 && cc < vcols) {
                    // a partial vector of the run (off is on the vector grid)
                    v[u] = Mem::template ld_part<T, VA, (HINT & kNtLoad) != 0>(Ab, off);
                } else if (!PARTV) {
                    for (int e = 0; e < VA; ++e)
                        if (cc + e >= 0 && cc + e < vcols)
                            v[u].v[e] = Mem::template ld1<T>(Ab, off + e);
                }
            }
            if constexpr (SHIFT) ccs[u] = cc;
            c += dc;
            R += dR;
            if (c >= W) {
                c -= W;
                R += 1;
            }
        }
        R = R0;
        c = c0;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            int cc = c * VA;
            if constexpr (SHIFT) cc = ccs[u];
            if (R >= rLo && R < rHi && R < staged) {
                const int at = R * g.pitch + cc;
#pragma unroll
                for (int e = 0; e < VA; ++e)
                    if (cc + e >= 0 && cc + e < vcols) Mem::template lds_st<T>(lds, at + e, v[u].v[e]);
            }
            c += dc;
            R += dR;
            if (c >= W) {
                c -= W;
                R += 1;
            }
        }
    }
}

// Specialised store phase, the counterpart of tile_load_fast.
template <class Mem, typename T, int VB, int MODE, int HINT, int BLOCK, bool SHIFT>
__host__ __device__ inline void tile_store_fast(const TileArgs& g, const TileBase& tb, int r0,
                                                int tid, T* B, const T* lds,
                                                const int64_t* colOffB, T alpha, T beta) {
    constexpr int NB = MODE == kAxpby ? axpby_store_batch(SHIFT ? kShifted : kFast)
                                      : tile_batch(BLOCK);
    // B runs sheared onto lines (each column's run starts on the line at or
    // below the chunk's first row), or else shifted onto the vector grid
    const bool sheared = SHIFT && g.shear > 0;
    const bool shift = SHIFT && !sheared && (!g.runsOnGridB || g.misB != 0);
    const int W = sheared ? int(g.runB) / VB
                          : (g.subRows + (shift ? VB - 1 : 0) + VB - 1) / VB;  // per column
    const int vcols = int(tb.validCols);
    // element ss of a column's run exists when rows0 <= ss < rows
    const int rows0 = sheared ? -int(tb.rowBase) : 0;
    const int rows = sheared ? int(g.rowsB - tb.rowBase)
                             : int(imin(int64_t(g.subRows), tb.validRows - r0));
    const int sh = sheared ? g.shear : 0;
    T* Bb = B + tb.b + r0;
    // element offset of this pass's origin from the B vector grid / line
    const int tbm = shift ? int((tb.b + r0 + g.misB) & (VB - 1))
                          : sheared ? int((tb.b + r0 + g.misLineB) & (g.lineB - 1)) : 0;
    const int gridMask = sheared ? g.lineB - 1 : VB - 1;
    int q = tid / W, s = tid % W;
    const int dq = BLOCK / W, ds = BLOCK % W;
    while (q < int(g.runA)) {
        Vec<T, VB> x[NB], y[NB];
        int sss[SHIFT ? NB : 1];
        const int q0 = q, s0 = s;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            int ss = s * VB;
            if (q < vcols) {
                int colOff = 0;
                if (shift || sheared || MODE == kAxpby)
                    colOff = int(Mem::template lds_ld<int64_t>(colOffB, q));
                if (shift || sheared) ss -= (tbm + colOff) & gridMask;
                const int base = (ss + sh) * g.pitch + q;
#pragma unroll
                for (int e = 0; e < VB; ++e)
                    if (ss + e >= rows0 && ss + e < rows)
                        x[u].v[e] = Mem::template lds_ld<T>(lds, base + e * g.pitch);
                if (MODE == kAxpby) {
                    const int off = colOff + ss;
                    if (ss >= rows0 && ss + VB <= rows) {
                        y[u] = Mem::template ld<T, VB, (HINT & kNtStore) != 0>(Bb, off);
                    } else {
                        for (int e = 0; e < VB; ++e)
                            if (ss + e >= rows0 && ss + e < rows)
                                y[u].v[e] = Mem::template ld1<T>(Bb, off + e);
                    }
                }
            }
            if constexpr (SHIFT) sss[u] = ss;
            s += ds;
            q += dq;
            if (s >= W) {
                s -= W;
                q += 1;
            }
        }
        q = q0;
        s = s0;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            int ss = s * VB;
            if constexpr (SHIFT) ss = sss[u];
            if (q < vcols && ss + VB > rows0 && ss < rows) {
                const int off = int(Mem::template lds_ld<int64_t>(colOffB, q)) + ss;
                Vec<T, VB> zv;
#pragma unroll
                for (int e = 0; e < VB; ++e)
                    zv.v[e] =
                        update<MODE>(x[u].v[e], MODE == kAxpby ? y[u].v[e] : T(0), alpha, beta);
                if (ss >= rows0 && ss + VB <= rows) {
                    Mem::template st<(HINT & kNtStore) != 0, T, VB>(Bb, off, zv);
                } else {
                    for (int e = 0; e < VB; ++e)
                        if (ss + e >= rows0 && ss + e < rows)
                            Mem::template st1<(HINT & kNtStore) != 0, T>(Bb, off + e, zv.v[e]);
                }
            }
            s += ds;
            q += dq;
            if (s >= W) {
                s -= W;
                q += 1;
            }
        }
    }
}

// Direct LDS loads (TileArgs::directLds): whether this tile can take them
// with A vectors of VA elements: its columns whole vectors, and the rotation
// of its rows (row / 4, below) below the vectors per row.  The plan builder
// sets directLds only where every tile can; the host emulator checks it.
__host__ __device__ inline bool tile_direct_lds(const TileArgs& g, const TileBase& tb, int va) {
    return g.directLds && g.subRows >= g.runB && g.runA % va == 0 && tb.validCols % va == 0 &&
           ((g.subRows - 1) >> 2) < g.runA / va;
}

// Load phase with direct LDS loads: the tile is staged without padding,
// row R (one A run, W = runA / VA vectors) in 16-byte slots R*W .. R*W+W-1.
// Each wave fetches 64 consecutive slots per instruction, one per lane, and
// slot cs of row R holds A vector (cs + R/4) mod W: rotating each group of
// four rows spreads the store phase's column reads (four rows of one column
// per lane) over the LDS banks.  Only the vectors of valid rows and columns
// are fetched; the others' slots are never read.
template <class Mem, typename T, int VA, int HINT, int BLOCK>
__host__ __device__ inline void tile_load_direct(const TileArgs& g, const TileBase& tb, int tid,
                                                 const T* A, T* lds, const int64_t* rowOffA) {
    const int W = int(g.runA) / VA;
    const int rows = int(imin(int64_t(g.subRows), tb.validRows));
    const int vcols = int(tb.validCols);
    const int total = g.subRows * W;
    const int wave = Mem::wave_uniform(tid >> 6), lane = tid & 63;
    const T* Ab = A + tb.a;
    for (int k0 = wave * 64; k0 < total; k0 += BLOCK) {
        const int k = k0 + lane;
        const int R = k / W, cs = k - R * W;
        int c = cs + (R >> 2);
        if (c >= W) c -= W;
        if (k < total && R < rows && c * VA < vcols) {
            const int off = int(Mem::template lds_ld<int64_t>(rowOffA, R)) + c * VA;
            Mem::template ld_lds<T, VA, (HINT & kNtLoad) != 0>(Ab, off, lds + k0 * VA, lane);
        }
    }
    Mem::wait_ld_lds();
}

// Store phase after tile_load_direct (B only written): tile_store_fast's
// thread-to-vector map, element (R, q) read from slot
// R*W + (q/VA - R/4) mod W.  The rows of one B vector share R/4, since a
// vector starts at a multiple of VB <= 4.
template <class Mem, typename T, int VA, int VB, int MODE, int HINT, int BLOCK>
__host__ __device__ inline void tile_store_rotated(const TileArgs& g, const TileBase& tb, int tid,
                                                   T* B, const T* lds, const int64_t* colOffB,
                                                   T alpha, T beta) {
    static_assert(MODE != kAxpby, "direct LDS loads serve tiles whose B is only written");
    constexpr int NB = 4;
    const int WA = int(g.runA) / VA;
    const int W = (g.subRows + VB - 1) / VB;  // vectors per column
    const int vcols = int(tb.validCols);
    const int rows = int(imin(int64_t(g.subRows), tb.validRows));
    T* Bb = B + tb.b;
    int q = tid / W, s = tid % W;
    const int dq = BLOCK / W, ds = BLOCK % W;
    while (q < int(g.runA)) {
        Vec<T, VB> x[NB];
        const int q0 = q, s0 = s;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int ss = s * VB;
            if (q < vcols) {
                int cs = q / VA - (ss >> 2);
                if (cs < 0) cs += WA;
                const int base = (ss * WA + cs) * VA + (q & (VA - 1));
#pragma unroll
                for (int e = 0; e < VB; ++e)
                    if (ss + e < rows) x[u].v[e] = Mem::template lds_ld<T>(lds, base + e * WA * VA);
            }
            s += ds;
            q += dq;
            if (s >= W) {
                s -= W;
                q += 1;
            }
        }
        q = q0;
        s = s0;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int ss = s * VB;
            if (q < vcols && ss < rows) {
                const int off = int(Mem::template lds_ld<int64_t>(colOffB, q)) + ss;
                Vec<T, VB> zv;
#pragma unroll
                for (int e = 0; e < VB; ++e) zv.v[e] = update<MODE>(x[u].v[e], T(0), alpha, beta);
                if (ss + VB <= rows) {
                    Mem::template st<(HINT & kNtStore) != 0, T, VB>(Bb, off, zv);
                } else {
                    for (int e = 0; e < VB; ++e)
                        if (ss + e < rows)
                            Mem::template st1<(HINT & kNtStore) != 0, T>(Bb, off + e, zv.v[e]);
                }
            }
            s += ds;
            q += dq;
            if (s >= W) {
                s -= W;
                q += 1;
            }
        }
    }
}

// Store phase of the shared-run variant (its load phase is
// tile_load_fast's, shifted): column q is the contiguous B run
// colOffB[q] + [0, runB), whose position b sits in LDS at pos(b) + ldsCol[q]
// (shared_positions).  A run that starts off the B vector grid is shifted onto it,
// its first and last vectors partial.  Same thread-to-vector map and
// batching as tile_store_fast.
template <class Mem, typename T, int VB, int MODE, int HINT, int BLOCK>
__host__ __device__ inline void tile_store_shared(const TileArgs& g, const TileBase& tb, int tid,
                                                  T* B, const T* lds, const int64_t* colOffB,
                                                  const int32_t* ldsCol, const int32_t* ldsRow,
                                                  T alpha, T beta) {
    constexpr int NB = MODE == kAxpby ? axpby_store_batch(kShared) : tile_batch(BLOCK);
    const bool shift = !g.runsOnGridB || g.misB != 0;
    const int W = (int(g.runB) + (shift ? VB - 1 : 0) + VB - 1) / VB;  // vectors per column
    const int vcols = int(tb.validColsS);
    const int rows = int(tb.validRunB);
    T* Bb = B + tb.b;
    // element offset of the tile origin from the B vector grid
    const int tbm = shift ? int((tb.b + g.misB) & (VB - 1)) : 0;
    int q = tid / W, s = tid % W;
    const int dq = BLOCK / W, ds = BLOCK % W;
    while (q < g.nColS) {
        Vec<T, VB> x[NB], y[NB];
        int sss[NB];
        const int q0 = q, s0 = s;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            int ss = s * VB;
            if (q < vcols) {
                int colOff = 0;
                if (shift || MODE == kAxpby) colOff = int(Mem::template lds_ld<int64_t>(colOffB, q));
                if (shift) ss -= (tbm + colOff) & (VB - 1);
                const int colL = Mem::template lds_ld<int32_t>(ldsCol, q);
                int32_t pos[VB];
                shared_positions<Mem, VB>(g, ldsRow, ss, rows, pos);
#pragma unroll
                for (int e = 0; e < VB; ++e)
                    if (ss + e >= 0 && ss + e < rows)
                        x[u].v[e] = Mem::template lds_ld<T>(lds, pos[e] + colL);
                if (MODE == kAxpby) {
                    const int off = colOff + ss;
                    if (ss >= 0 && ss + VB <= rows) {
                        y[u] = Mem::template ld<T, VB, (HINT & kNtStore) != 0>(Bb, off);
                    } else {
                        for (int e = 0; e < VB; ++e)
                            if (ss + e >= 0 && ss + e < rows) y[u].v[e] = Mem::template ld1<T>(Bb, off + e);
                    }
                }
            }
            sss[u] = ss;
            s += ds;
            q += dq;
            if (s >= W) {
                s -= W;
                q += 1;
            }
        }
        q = q0;
        s = s0;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int ss = sss[u];
            if (q < vcols && ss + VB > 0 && ss < rows) {
                const int off = int(Mem::template lds_ld<int64_t>(colOffB, q)) + ss;
                Vec<T, VB> zv;
#pragma unroll
                for (int e = 0; e < VB; ++e)
                    zv.v[e] =
                        update<MODE>(x[u].v[e], MODE == kAxpby ? y[u].v[e] : T(0), alpha, beta);
                if (ss >= 0 && ss + VB <= rows) {
                    Mem::template st<(HINT & kNtStore) != 0, T, VB>(Bb, off, zv);
                } else {
                    for (int e = 0; e < VB; ++e)
                        if (ss + e >= 0 && ss + e < rows)
                            Mem::template st1<(HINT & kNtStore) != 0, T>(Bb, off + e, zv.v[e]);
                }
            }
            s += ds;
            q += dq;
            if (s >= W) {
                s -= W;
                q += 1;
            }
        }
    }
}

// Load phase of the pass over tile rows [r0, r0 + subRows) of each of the
// nZ stacked tiles: the rows are contiguous runs of A.  Stacked row R holds
// row r = R mod subRows of depth z = R / subRows and lands in LDS row R.
// Thread tid takes the vectors tid, tid + kBlock, ... of the (stacked row,
// vector) space, vector fastest, so a wave reads whole runs.  Vectors sit on
// the A vector grid: a run that starts off it is covered by one more vector,
// its first and last ones partial (element loads).  Variants kFast,
// kShifted and kShared (see tile_variant) take tile_load_fast instead.
template <class Mem, typename T, int VA, int HINT, int VAR, int BLOCK = kBlock,
          int LB = tile_batch(BLOCK), bool PARTV = true>
__host__ __device__ inline void tile_load(const TileArgs& g, const TileBase& tb, int64_t r0,
                                          int tid, const T* A, T* lds, const int64_t* rowOffA) {
    static_assert(VAR == kFast || BLOCK == kBlock, "only the kFast variant runs kBigBlock");
    if constexpr (VAR != kGeneral) {
        tile_load_fast<Mem, T, VA, HINT, BLOCK, VAR == kShifted || VAR == kShared, LB, PARTV>(
            g, tb, int(r0), tid, A, lds, rowOffA);
        return;
    }
    const bool shift = !g.runsOnGridA || g.misA != 0;
    const bool depth = g.nZ > 1;
    const int64_t W = (g.runA + (shift ? VA - 1 : 0) + VA - 1) / VA;  // vectors per row
    const int64_t rows = imin(int64_t(g.subRows), tb.validRows - r0);  // rows of this pass
    // staged rows: with shear, the shear rows before the chunk come first
    const int64_t stacked = (depth ? int64_t(g.nZ) * g.subRows : int64_t(g.subRows)) + g.shear;
    int64_t R = tid / W, c = tid % W;
    const int64_t dR = kBlock / W, dc = kBlock % W;
    while (R < stacked) {
        Vec<T, VA> v[kBatch];
        int64_t at[kBatch], cc[kBatch];
        bool ok[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            int64_t z = 0, r = R;
            if (depth) {
                z = int64_t(fast_div(uint32_t(R), g.zRows));
                r = R - z * g.subRows;
            }
            // with shear, staged row R is run index rowBase + R - shear
            const int64_t G = tb.rowBase + R - g.shear;
            const bool rowOk = g.shear ? (G >= 0 && G < g.rowsB) : r < rows;
            ok[u] = R < stacked && rowOk && (!depth || z < tb.validDepth);
            cc[u] = c * VA;
            at[u] = 0;
            if (ok[u]) {
                int64_t start = tb.a + Mem::template lds_ld<int64_t>(rowOffA, r0 + r);
                if (depth) start += z * g.zStrideA;
                if (shift) cc[u] -= (start + g.misA) & (VA - 1);
                ok[u] = (!shift || cc[u] + VA > 0) && cc[u] < tb.validCols;
                at[u] = R * g.pitch + cc[u];
                if (ok[u]) {
                    if ((!shift || cc[u] >= 0) && cc[u] + VA <= tb.validCols) {
                        v[u] = Mem::template ld<T, VA, (HINT & kNtLoad) != 0>(A, start + cc[u]);
                    } else {
                        for (int e = 0; e < VA; ++e)
                            if ((!shift || cc[u] + e >= 0) && cc[u] + e < tb.validCols)
                                v[u].v[e] = Mem::template ld1<T>(A, start + cc[u] + e);
                    }
                }
            }
            c += dc;
            R += dR;
            if (c >= W) {
                c -= W;
                R += 1;
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (ok[u]) {
#pragma unroll
                for (int e = 0; e < VA; ++e)
                    if ((!shift || cc[u] + e >= 0) && cc[u] + e < tb.validCols)
                        Mem::template lds_st<T>(lds, at[u] + e, v[u].v[e]);
            }
        }
    }
}

// Store phase of the same pass: the tile's columns are contiguous runs of B,
// of which this pass writes rows [r0, r0 + subRows).  Stacked column Q is
// column q = Q mod runA of depth z = Q / runA.  Thread tid takes the vectors
// tid, tid + kBlock, ... of the (stacked column, vector) space, vector
// fastest, gathers each vector's VB elements from consecutive LDS rows, and
// writes it to B (reading B first when beta != 0).  Vectors sit on the B
// vector grid, as in the load phase.
template <class Mem, typename T, int VB, int MODE, int HINT, int VAR, int BLOCK = kBlock>
__host__ __device__ inline void tile_store(const TileArgs& g, const TileBase& tb, int64_t r0,
                                           int tid, T* B, const T* lds, const int64_t* colOffB,
                                           T alpha, T beta) {
    static_assert(VAR == kFast || BLOCK == kBlock, "only the kFast variant runs kBigBlock");
    if constexpr (VAR != kGeneral) {
        tile_store_fast<Mem, T, VB, MODE, HINT, BLOCK, VAR == kShifted>(g, tb, int(r0), tid, B, lds,
                                                                        colOffB, alpha, beta);
        return;
    }
    constexpr int NB = MODE == kAxpby ? axpby_store_batch(kGeneral) : kBatch;
    // B side: with shear, each column's run starts on the line at or below
    // the chunk's first row (d = the column's offset from that line); else,
    // without the vector grid, vectors are shifted onto it (d < VB).
    const bool sheared = g.shear > 0;
    const bool shift = !sheared && (!g.runsOnGridB || g.misB != 0);
    const bool depth = g.nZ > 1;
    const int64_t W = sheared ? g.runB / VB
                              : (g.subRows + (shift ? VB - 1 : 0) + VB - 1) / VB;  // per column
    const int64_t rows = imin(int64_t(g.subRows), tb.validRows - r0);
    // element ss + e of a column's run exists when lo <= ss + e < hi
    const int64_t lo = sheared ? -tb.rowBase : 0;
    const int64_t hi = sheared ? g.rowsB - tb.rowBase : rows;
    const int64_t cols = depth ? int64_t(g.nZ) * g.runA : g.runA;
    int64_t Q = tid / W, s = tid % W;
    const int64_t dQ = kBlock / W, ds = kBlock % W;
    while (Q < cols) {
        Vec<T, VB> x[NB], y[NB];
        int64_t ss[NB], off[NB];
        bool ok[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            int64_t z = 0, q = Q;
            if (depth) {
                z = int64_t(fast_div(uint32_t(Q), g.zCols));
                q = Q - z * g.runA;
            }
            ok[u] = Q < cols && q < tb.validCols && (!depth || z < tb.validDepth);
            ss[u] = s * VB;
            off[u] = 0;
            if (ok[u]) {
                int64_t start = tb.b + Mem::template lds_ld<int64_t>(colOffB, q) + r0;
                if (depth) start += z * g.zStrideB;
                if (sheared) ss[u] -= (start + g.misLineB) & (g.lineB - 1);
                else if (shift) ss[u] -= (start + g.misB) & (VB - 1);
                ok[u] = ss[u] + VB > lo && ss[u] < hi;
                off[u] = start + ss[u];
                if (ok[u]) {
                    const int64_t base =
                        ((depth ? z * g.subRows : 0) + ss[u] + g.shear) * g.pitch + q;
#pragma unroll
                    for (int e = 0; e < VB; ++e)
                        if (ss[u] + e >= lo && ss[u] + e < hi)
                            x[u].v[e] = Mem::template lds_ld<T>(lds, base + e * g.pitch);
                    if (MODE == kAxpby) {
                        if (ss[u] >= lo && ss[u] + VB <= hi) {
                            y[u] = Mem::template ld<T, VB, (HINT & kNtStore) != 0>(B, off[u]);
                        } else {
                            for (int e = 0; e < VB; ++e)
                                if (ss[u] + e >= lo && ss[u] + e < hi)
                                    y[u].v[e] = Mem::template ld1<T>(B, off[u] + e);
                        }
                    }
                }
            }
            s += ds;
            Q += dQ;
            if (s >= W) {
                s -= W;
                Q += 1;
            }
        }
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            if (ok[u]) {
                Vec<T, VB> zv;
#pragma unroll
                for (int e = 0; e < VB; ++e)
                    zv.v[e] = update<MODE>(x[u].v[e], MODE == kAxpby ? y[u].v[e] : T(0), alpha, beta);
                if (ss[u] >= lo && ss[u] + VB <= hi) {
                    Mem::template st<(HINT & kNtStore) != 0, T, VB>(B, off[u], zv);
                } else {
                    for (int e = 0; e < VB; ++e)
                        if (ss[u] + e >= lo && ss[u] + e < hi)
                            Mem::template st1<(HINT & kNtStore) != 0, T>(B, off[u] + e, zv.v[e]);
                }
            }
        }
    }
}

// LDS layout of kernel T: rowOffA[runB + shear], colOffB[runA], then
// nZ * subRows + shear rows of the tile.  A tile with runB > subRows is
// staged in passes of subRows rows (never with depth or shear).  The
// shared-run variant: its tables (shared_table_words), then subRows
// rows.
__host__ __device__ inline int64_t tile_lds_bytes(const TileArgs& g, int elem) {
    if (g.shared)
        return shared_table_words(g) * int64_t(sizeof(int64_t)) +
               int64_t(g.subRows) * g.pitch * elem;
    return (g.runA + g.runB + g.shear) * int64_t(sizeof(int64_t)) +
           (int64_t(g.nZ) * g.subRows + g.shear) * g.pitch * elem;
}

// ---------------------------------------------------------------------------
// Kernel S: the stride-1 index is kept
// ---------------------------------------------------------------------------


// Block `blk` handles items [blk*kBlock*NI, (blk+1)*kBlock*NI), NI =
// items_per_lane; lane tid takes items first + u*kBlock + tid, so each wave
// covers consecutive B
// vectors.  All loads of a lane are issued before its first store.
template <class Mem, typename T, int V, int MODE, int HINT>
__host__ __device__ inline void stream_items(const StreamArgs& g, uint32_t first, int tid,
                                             const T* A, T* B, T alpha, T beta) {
    const FastDiv& W = g.W[log2_width(V)];
    const uint32_t numItems = g.numItems[log2_width(V)];
    constexpr int NI = items_per_lane(int(sizeof(T)), V);
    Vec<T, V> x[NI], y[NI];
    int64_t offA[NI], offB[NI], col[NI];
    bool ok[NI];
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        const uint64_t item = uint64_t(first) + uint64_t(u) * kBlock + uint64_t(tid);
        ok[u] = item < numItems;
        offA[u] = offB[u] = col[u] = 0;
        if (ok[u]) {
            uint32_t r = fast_div(uint32_t(item), W);
            col[u] = int64_t(uint32_t(item) - r * W.d) * V;
            int64_t a = 0, b = 0;
            for (int k = 0; k < g.nO; ++k) {
                uint32_t q = fast_div(r, g.oExt[k]);
                const int64_t j = int64_t(r - q * g.oExt[k].d);
                a += j * g.oStrideA[k];
                b += j * g.oStrideB[k];
                r = q;
            }
            offA[u] = a + col[u];
            offB[u] = b + col[u];
            if (col[u] + V <= g.rowLen) {
                x[u] = Mem::template ld<T, V, (HINT & kNtLoad) != 0>(A, offA[u]);
                if (MODE == kAxpby) y[u] = Mem::template ld<T, V, (HINT & kNtStore) != 0>(B, offB[u]);
            } else {
                for (int e = 0; e < V; ++e)
                    if (col[u] + e < g.rowLen) {
                        x[u].v[e] = Mem::template ld1<T>(A, offA[u] + e);
                        if (MODE == kAxpby) y[u].v[e] = Mem::template ld1<T>(B, offB[u] + e);
                    }
            }
        }
    }
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        if (!ok[u]) continue;
        Vec<T, V> z;
#pragma unroll
        for (int e = 0; e < V; ++e)
            z.v[e] = update<MODE>(x[u].v[e], MODE == kAxpby ? y[u].v[e] : T(0), alpha, beta);
        if (col[u] + V <= g.rowLen) {
            Mem::template st<(HINT & kNtStore) != 0, T, V>(B, offB[u], z);
        } else {
            for (int e = 0; e < V; ++e)
                if (col[u] + e < g.rowLen) Mem::template st1<(HINT & kNtStore) != 0, T>(B, offB[u] + e, z.v[e]);
        }
    }
}

// Kernel S over more than 2^32 items at width V (StreamArgs::numItems[log2 V]
// is 0): the rows are cut into slabs, launched one by one.  A slab holds the
// rows of the outer B positions 0..m-1 whole and a chunk of `chunk` values of
// position m (the most rows whose items the kernel can still count); the
// slowest positions m+1.. and the chunk number give the slab's base offsets.
// The launch sees nO = m + 1 positions; position m's local value stays below
// its extent, so its split leaves it whole.
struct StreamSlabs {
    int m;           // first outer position not whole in a slab (nO: none)
    int64_t chunk;   // values of position m per slab
    int64_t rows;    // rows of a full slab
    int64_t count;   // slabs
};

inline StreamSlabs stream_slabs_of(const StreamArgs& g, int V) {
    const int64_t limit = (int64_t(1) << 32) - int64_t(kBlock) * kMaxItems;
    const int64_t W = g.W[log2_width(V)].d;
    StreamSlabs s;
    s.m = 0;
    s.rows = 1;
    while (s.m < g.nO && s.rows * int64_t(g.oExt[s.m].d) * W < limit) s.rows *= g.oExt[s.m++].d;
    s.chunk = 1;
    s.count = 1;
    if (s.m < g.nO) {
        const int64_t e = g.oExt[s.m].d;
        s.chunk = (limit - 1) / (s.rows * W);  // >= 1: a row's vectors fit (plan builder)
        if (s.chunk > e) s.chunk = e;
        s.count = (e + s.chunk - 1) / s.chunk;
        for (int k = s.m + 1; k < g.nO; ++k) s.count *= g.oExt[k].d;
        s.rows *= s.chunk;
    }
    return s;
}

// Arguments and base offsets of slab `sl` (0 <= sl < s.count).
inline StreamArgs stream_slab_args(const StreamArgs& g, const StreamSlabs& s, int64_t sl, int V,
                                   int64_t* offA, int64_t* offB) {
    StreamArgs a = g;
    *offA = *offB = 0;
    int64_t rows = s.rows;
    if (s.m < g.nO) {
        const int64_t e = g.oExt[s.m].d, nChunks = (e + s.chunk - 1) / s.chunk;
        const int64_t c = sl % nChunks;
        int64_t x = sl / nChunks;
        *offA += c * s.chunk * g.oStrideA[s.m];
        *offB += c * s.chunk * g.oStrideB[s.m];
        const int64_t here = imin(s.chunk, e - c * s.chunk);
        rows = rows / s.chunk * here;
        for (int k = s.m + 1; k < g.nO; ++k) {
            const int64_t ek = g.oExt[k].d, j = x % ek;
            x /= ek;
            *offA += j * g.oStrideA[k];
            *offB += j * g.oStrideB[k];
        }
        a.nO = s.m + 1;
    }
    a.numRows = rows;
    a.numItems[log2_width(V)] = uint32_t(rows * int64_t(g.W[log2_width(V)].d));
    return a;
}

// A offset of row r of the stride-1-kept walk (rows in B order).
__host__ __device__ inline int64_t stream_row_a(const StreamArgs& g, uint32_t r) {
    int64_t a = 0;
    for (int k = 0; k < g.nO; ++k) {
        const uint32_t q = fast_div(r, g.oExt[k]);
        a += int64_t(r - q * g.oExt[k].d) * g.oStrideA[k];
        r = q;
    }
    return a;
}

// Flat walk of kernel S (g.flatB): item i is B's vector i, so every B access
// is a whole vector even when the row length is not a multiple of the width
// (rows of 63 fp32 would otherwise move one element per access).  The row
// split is done once per vector (twice when the vector crosses into the next
// row); A is read with ordinary loads, since its rows start anywhere: fp32
// with B only written takes one element-aligned vector load where the
// vector's elements lie in one row (MI355X, rows of 55-213 elements +27 to
// +35 %); elsewhere, and where a vector crosses into the next row, element by
// element (the vector load lost 2-6 % when B is read, and with fp64).  Same
// lane map as stream_items.
template <class Mem, typename T, int V, int MODE, int HINT>
__host__ __device__ inline void stream_items_flat(const StreamArgs& g, uint32_t first, int tid,
                                                  const T* A, T* B, T alpha, T beta) {
    const uint32_t numItems = g.numItems[log2_width(V)];
    const int64_t numel = g.numRows * g.rowLen;
    const int rowLen = int(g.L.d);
    constexpr int NI = items_per_lane(int(sizeof(T)), V);
    Vec<T, V> x[NI], y[NI];
    int64_t offB[NI];
    int n[NI];
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        const uint64_t item = uint64_t(first) + uint64_t(u) * kBlock + uint64_t(tid);
        n[u] = 0;
        offB[u] = int64_t(item) * V;
        if (item < numItems) {
            n[u] = int(imin(int64_t(V), numel - offB[u]));  // elements of this vector
            const uint32_t r = fast_div(uint32_t(offB[u]), g.L);
            const int c0 = int(uint32_t(offB[u]) - r * g.L.d);
            const int64_t a0 = stream_row_a(g, r);
            if (sizeof(T) == 4 && MODE != kAxpby && n[u] == V && c0 + V <= rowLen) {
                // inside one row: one load from wherever the row puts it
                x[u] = Mem::template ldu<T, V>(A, a0 + c0);
            } else {
                const int64_t a1 = c0 + n[u] > rowLen ? stream_row_a(g, r + 1) - rowLen : a0;
#pragma unroll
                for (int e = 0; e < V; ++e)
                    if (e < n[u])
                        x[u].v[e] = Mem::template ld1<T>(A, (c0 + e < rowLen ? a0 : a1) + c0 + e);
            }
            if (MODE == kAxpby) {
                if (n[u] == V) {
                    y[u] = Mem::template ld<T, V, (HINT & kNtStore) != 0>(B, offB[u]);
                } else {
                    for (int e = 0; e < V; ++e)
                        if (e < n[u]) y[u].v[e] = Mem::template ld1<T>(B, offB[u] + e);
                }
            }
        }
    }
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        if (n[u] == 0) continue;
        Vec<T, V> z;
#pragma unroll
        for (int e = 0; e < V; ++e)
            z.v[e] = update<MODE>(x[u].v[e], MODE == kAxpby ? y[u].v[e] : T(0), alpha, beta);
        if (n[u] == V) {
            Mem::template st<(HINT & kNtStore) != 0, T, V>(B, offB[u], z);
        } else {
            for (int e = 0; e < V; ++e)
                if (e < n[u]) Mem::template st1<(HINT & kNtStore) != 0, T>(B, offB[u] + e, z.v[e]);
        }
    }
}

// ---------------------------------------------------------------------------
// Identity after fusion: B <- alpha*A + beta*B over a flat range
// ---------------------------------------------------------------------------

// Lane tid of the block starting at vector `first` takes vectors
// first + u*kBlock + tid, u < items_per_lane; vector i covers elements
// [i*V, i*V + V), the last one possibly partial.
template <class Mem, typename T, int V, int MODE, int HINT>
__host__ __device__ inline void axpby_items(int64_t numel, int64_t first, int tid, const T* A,
                                            T* B, T alpha, T beta) {
    constexpr int NI = items_per_lane(int(sizeof(T)), V);
    Vec<T, V> x[NI], y[NI];
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        const int64_t off = (first + int64_t(u) * kBlock + tid) * V;
        if (off + V <= numel) {
            x[u] = Mem::template ld<T, V, (HINT & kNtLoad) != 0>(A, off);
            if (MODE == kAxpby) y[u] = Mem::template ld<T, V, (HINT & kNtStore) != 0>(B, off);
        }
    }
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        const int64_t off = (first + int64_t(u) * kBlock + tid) * V;
        if (off + V <= numel) {
            Vec<T, V> z;
#pragma unroll
            for (int e = 0; e < V; ++e)
                z.v[e] = update<MODE>(x[u].v[e], MODE == kAxpby ? y[u].v[e] : T(0), alpha, beta);
            Mem::template st<(HINT & kNtStore) != 0, T, V>(B, off, z);
        } else {
            for (int64_t e = off; e < numel; ++e) {
                T b = MODE == kAxpby ? Mem::template ld1<T>(B, e) : T(0);
                Mem::template st1<(HINT & kNtStore) != 0, T>(B, e, update<MODE>(Mem::template ld1<T>(A, e), b, alpha, beta));
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Fallback: one B element per thread, any shape
// ---------------------------------------------------------------------------

// Element e (in B order) is split into B's multi-index; its offsets in A and
// B follow from both tensors' strides.
template <class Mem, typename T, int MODE, int HINT, bool BIG>
__host__ __device__ inline void generic_elem(const GenericArgs& g, int64_t e, const T* A, T* B,
                                             T alpha, T beta) {
    int64_t offA = 0, offB = 0;
    if (BIG) {
        int64_t x = e;
        for (int k = 0; k < g.n; ++k) {
            const int64_t j = x % g.bExt64[k];
            offA += j * g.bStrideA[k];
            offB += j * g.bStrideB[k];
            x /= g.bExt64[k];
        }
    } else {
        uint32_t x = uint32_t(e);
        for (int k = 0; k < g.n; ++k) {
            uint32_t q = fast_div(x, g.bExt[k]);
            const int64_t j = int64_t(x - q * g.bExt[k].d);
            offA += j * g.bStrideA[k];
            offB += j * g.bStrideB[k];
            x = q;
        }
    }
    T b = MODE == kAxpby ? Mem::template ld1<T>(B, offB) : T(0);
    Mem::template st1<(HINT & kNtStore) != 0, T>(
        B, offB, update<MODE>(Mem::template ld1<T>(A, offA), b, alpha, beta));
}

}  // namespace hptt
