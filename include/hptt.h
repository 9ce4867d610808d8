/*
 * hptt.h -- C ABI of an MI355X (gfx950) library for the out-of-place tensor
 * transposition of Eq. (1) of the HPTT paper (Springer, Su, Bientinesi,
 * Section 1):
 *
 *     B_{Pi(i_1 .. i_N)}  <-  alpha * A_{i_1 .. i_N}  +  beta * B_{Pi(i_1 .. i_N)}
 *
 * A and B are dense N-dimensional tensors in the Fortran layout of Section 1
 * (the first index has stride 1), Pi is any permutation of the N indices and
 * alpha, beta are scalars.
 *
 * Usage follows the plan/execute split of Section 3.1 and Fig. 3b: a plan is
 * built once on the host from the permutation, the extents, the scalars and
 * the element type, and is then executed any number of times on device
 * pointers and a HIP stream.  A plan holds no pointers to tensor data.
 *
 * Conventions shared by every call:
 *  - perm is 0-based and perm[k] is the index of A that sits at position k of
 *    B, so the compact extents of B are sizeB[k] = sizeA[perm[k]] (Fig. 3b
 *    passes a zero-based permutation; Table 1 names B's indices in this order).
 *  - A and B are compact (no outer sizes), hold numel = prod(sizeA) elements
 *    each, and must not overlap (the operation is out-of-place, Section 3).
 *  - Every function returns a status and never aborts or throws.
 *  - Ownership: a plan owns only host memory.  The caller owns A, B and the
 *    stream and keeps them alive until the work queued on the stream is done.
 */
#ifndef HPTT_HIP_H
#define HPTT_HIP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HPTT_MAX_DIMS 16

typedef struct hptt_plan_s *hptt_plan_t;

/* Element type of A, B, alpha and beta.  The paper's kernels are written for
 * single precision (Fig. 5) and its contraction study runs in double (Fig. 9). */
typedef enum {
    HPTT_FLOAT32 = 0,
    HPTT_FLOAT64 = 1
} hptt_dtype_t;

typedef enum {
    HPTT_SUCCESS = 0,
    HPTT_ERROR_INVALID_ARGUMENT = 1, /* bad perm, rank, extent, null pointer, misaligned element */
    HPTT_ERROR_UNSUPPORTED = 2,      /* a forced option the plan cannot honour, or a problem
                                        beyond an entry point's fixed limit */
    HPTT_ERROR_OVERLAP = 3,          /* A and B share memory */
    HPTT_ERROR_OUT_OF_MEMORY = 4,    /* host allocation of the plan failed */
    HPTT_ERROR_HIP = 5               /* the kernel launch failed */
} hptt_status_t;

/* Kernel classes a plan can execute with. */
typedef enum {
    HPTT_KERNEL_AUTO = 0,    /* options only: let the plan builder choose */
    HPTT_KERNEL_NONE = 1,    /* an extent is 0: execute launches nothing */
    HPTT_KERNEL_AXPBY = 2,   /* the fused permutation is the identity: B <- alpha*A + beta*B */
    HPTT_KERNEL_STREAM = 3,  /* A's stride-1 index is also B's: rows streamed in B order */
    HPTT_KERNEL_TILE = 4,    /* tiles staged through LDS: the stride-1 index moves,
                                or the runs share indices (a short kept one) */
    HPTT_KERNEL_GENERIC = 5  /* one element per thread in B order; any shape */
} hptt_kernel_t;

/* Optional knobs of hptt_create_plan_ex.  Zero-initialise and set what you
 * need; zero means "choose".  They exist to measure each design choice. */
typedef struct {
    hptt_kernel_t kernel;  /* force a kernel class; TILE and STREAM fail with
                              HPTT_ERROR_UNSUPPORTED where they do not apply */
    int32_t run_a;         /* TILE: target length, in elements, of the contiguous
                              A run of a tile (its columns) */
    int32_t run_b;         /* TILE: target length of the contiguous B run (rows) */
    int32_t max_vec;       /* cap on the vector width in elements (1 = scalar) */
    int32_t store_hint;    /* 1: non-temporal stores of B (and, when beta != 0,
                              non-temporal loads of B); 2: ordinary ones */
    int32_t load_hint;     /* 1: non-temporal loads of A; 2: ordinary loads */
    int32_t lds_pad;       /* TILE: LDS row padding in elements, 0 = default, -1 = none */
    int32_t max_blocks;    /* cap on the grid; workgroups loop over tiles beyond it */
    int32_t tile_order;    /* TILE: 1 = tiles in grid-digit order, 2 = diagonal
                              (second grid digit rotated by the first), 3 =
                              diagonal, with each XCD given a contiguous range
                              of tiles, 4 = grid-digit order with contiguous
                              ranges per XCD */
    int32_t exact_runs;    /* TILE: 1 = chunk the runs to the target lengths even
                              where runs then do not start on 128-byte lines */
    int32_t row_passes;    /* TILE: N > 1 = stage each tile through LDS in N passes
                              over its rows (less LDS, one more barrier per pass) */
    int32_t depth;         /* TILE: tiles stacked per workgroup along one more index;
                              0 = as many as a small tile needs, 1 = none */
    int32_t min_tile;      /* TILE: smallest tile (elements) worth a workgroup round;
                              smaller tiles get longer runs or depth; 0 = 16 KiB worth */
    int32_t block;         /* TILE: threads per workgroup, 256 or 1024, when the
                              launch can take the specialised tile kernel (the
                              general one always runs 256); 0 = choose */
    int32_t skew;          /* TILE: diagonal orders rotate the second grid digit by
                              skew times the first; 0 = 1 */
    int32_t shear;         /* TILE: B runs that cannot be whole 128-byte lines are
                              sheared onto lines (each column's run starts on the
                              line at or below the chunk); 0 = where they apply
                              and the problem is not small, 1 = wherever they
                              apply, 2 = never */
    int32_t shared_runs;   /* TILE: runs that share indices (the B run passes
                              through indices of the A run, e.g. a B stride-1
                              extent of 2 or a short kept stride-1 index): 0 =
                              where disjoint runs leave a run shorter than a
                              128-byte line and shared ones are longer, 1 =
                              wherever they apply, 2 = never */
    int32_t flat_runs;     /* TILE: B runs cut from the flattened range of the
                              B indices they span (back to back in B, none in
                              the A run) in whole 128-byte lines, instead of
                              whole multiples of the inner extents: 0 = where
                              those extents are not whole lines and the usual
                              B run is not or is long, 1 = wherever they
                              apply, 2 = never.  STREAM: B (compact) walked as
                              one flat range of whole vectors, A read element
                              by element: 0 = where the row walk would move
                              one element per access (odd row lengths), or two
                              fp32 elements when beta != 0, 1 = wherever B is
                              compact, 2 = never */
    int32_t grid_order;    /* TILE: order of the grid digits of the indices outside
                              the tile (after the chunk counters): 1 = A order, 2 =
                              by the sum of their strides in A and B, 3 = B
                              order; 0 = choose */
    int32_t direct_lds;    /* TILE, beta == 0: A fetched straight into LDS
                              (global_load_lds_dwordx4) by the variant whose runs
                              all start on the 16-byte grid, where A's vectors are
                              16 bytes, the tile is staged in one pass and its
                              column count is whole vectors: 0 = where it
                              applies, 2 = never */
    int32_t xcd_group;     /* TILE, STREAM: workgroups are dealt to MI355X's
                              8 XCDs (each with its own L2) round robin; with
                              k > 1 each XCD takes tile (block) numbers k
                              consecutive at a time, so tiles that share
                              128-byte lines of A (runs that do not start on
                              lines) share an L2 while the tiles in flight
                              stay a near-contiguous range: 0 = choose (STREAM:
                              no grouping), 1 = no grouping, k = a power of two
                              up to 1024.  Ignored with tile_order 3 and 4,
                              which give each XCD one contiguous range */
} hptt_options_t;

/* What the plan builder decided; for inspection and tests. */
typedef struct {
    int32_t ndim;                      /* rank after dropping extent-1 indices and fusing */
    int64_t size[HPTT_MAX_DIMS];       /* fused extents of A */
    int32_t perm[HPTT_MAX_DIMS];       /* fused permutation, same convention as perm */
    hptt_kernel_t kernel;
    int64_t numel;
    int32_t elem_bytes;
    int64_t run_a;                     /* TILE: A-run (columns) of a tile, elements */
    int64_t run_b;                     /* TILE: B-run (rows); STREAM: kept row length */
    int32_t dims_a;                    /* TILE: fused A indices inside the A run */
    int32_t dims_b;                    /* TILE: fused B positions inside the B run */
    int32_t vec_a;                     /* vector width of A accesses (TILE: runs that start
                                          off the vector grid are shifted onto it) */
    int32_t vec_b;                     /* vector width of B accesses */
    int32_t lds_pitch;                 /* TILE: LDS row pitch in elements */
    int32_t rows_per_pass;             /* TILE: tile rows staged through LDS at once */
    int64_t footprint_a;               /* elements from A's first to its last element */
    int64_t footprint_b;               /* the same for B (numel for compact tensors) */
    int32_t lds_bytes;                 /* LDS per workgroup */
    int64_t tiles;                     /* TILE: tiles; STREAM, AXPBY: 16-byte vectors;
                                          GENERIC: elements */
    int64_t grid;                      /* workgroups launched */
    int32_t block;                     /* threads per workgroup (TILE: of the specialised
                                          variant; the general one runs 256) */
    int32_t hints;                     /* bit 0: non-temporal B stores (and B loads
                                          when beta != 0); bit 1: non-temporal A
                                          loads */
    int32_t mode;                      /* 0 raw copy, 1 scale (beta = 0), 2 alpha*A + beta*B */
    int32_t tile_order;                /* TILE: 1 grid-digit order, 2 diagonal, 3 diagonal
                                          with contiguous tile ranges per XCD, 4
                                          grid-digit order with such ranges */
    int32_t depth;                     /* TILE: tiles stacked per workgroup round */
    int32_t shear;                     /* TILE: extra rows staged for sheared B runs
                                          (0: runs not sheared) */
    int32_t shared_runs;               /* TILE: fused indices shared by the A run and
                                          the B run (0: disjoint runs) */
    int32_t flat_runs;                 /* TILE: fused B indices the flat B run is cut
                                          from (0: B runs are not flat); STREAM: 1
                                          when B is walked flat */
    int32_t grid_order;                /* TILE: order of the grid digits outside the tile:
                                          1 A order, 2 by the sum of their strides, 3 B
                                          order (0: not a tile plan) */
    int32_t direct_lds;                /* TILE: 1 when tiles are fetched straight into
                                          LDS (by launches that take the variant
                                          with every run on the 16-byte grid) */
    int32_t xcd_group;                 /* TILE, STREAM: consecutive tile (block) numbers
                                          each XCD takes at a time (1 = plain round
                                          robin; 0 with the contiguous XCD ranges of
                                          tile_order 3 and 4, and for the other
                                          kernels) */
} hptt_plan_info_t;

/*
 * Build a plan for Eq. (1) (Section 1) with the quick path of Section 3.1:
 * indices that are consecutive in both A and B are merged into superindices
 * (Section 3.1, footnote 4), extent-1 indices are dropped, and one kernel and
 * tile shape is chosen from the fused shape without any search.
 *
 *   plan   out: the new plan; set to NULL on any error.
 *   perm   N entries, a permutation of 0..N-1 (see the conventions above).
 *   N      rank, 1 <= N <= HPTT_MAX_DIMS.
 *   sizeA  N extents of A, each >= 0 (any 0 makes the plan a no-op).
 *   alpha, beta  scalars, rounded once to dtype here.  beta == 0 means B is
 *          never read (Eq. 2 counts B once); alpha == 1 with beta == 0 is a
 *          bit-exact copy; alpha == 0 is not short-cut (A is still read).
 *   dtype  element type of A and B.
 * Makes no HIP call.  Errors: HPTT_ERROR_INVALID_ARGUMENT, HPTT_ERROR_OUT_OF_MEMORY.
 * With the environment variable HPTT_LOG set to anything but "" or "0", every
 * plan this or any other plan call creates prints one line to stderr,
 * "[hptt] plan: " followed by hptt_describe_plan's text.
 */
hptt_status_t hptt_create_plan(hptt_plan_t *plan, const int32_t *perm, int32_t N,
                               const int64_t *sizeA, double alpha, double beta,
                               hptt_dtype_t dtype);

/* As hptt_create_plan, with optional knobs (options may be NULL).  A forced
 * kernel class or tile that cannot serve the problem gives
 * HPTT_ERROR_UNSUPPORTED. */
hptt_status_t hptt_create_plan_ex(hptt_plan_t *plan, const int32_t *perm, int32_t N,
                                  const int64_t *sizeA, double alpha, double beta,
                                  hptt_dtype_t dtype, const hptt_options_t *options);

/*
 * As hptt_create_plan_ex, for sub-tensors (Section 3.1, Fig. 3): A and B are
 * parts of larger enclosing tensors, like a BLAS leading dimension, which
 * allows transposing-and-compacting and transposing-and-scattering.
 *
 *   outerSizeA  N extents of the tensor enclosing A, in A's index order, each
 *               >= sizeA[d]; NULL means A is compact.
 *   outerSizeB  N extents of the tensor enclosing B, in B's index order, each
 *               >= sizeB[k] = sizeA[perm[k]]; NULL means B is compact.
 * Strides are the Fortran strides of the enclosing extents.  hptt_exec then
 * takes pointers to the sub-tensors' first elements; elements of the
 * enclosing B outside the sub-tensor are neither read nor written.  Indices
 * are merged into superindices only where they lie back to back in both
 * tensors.  Errors as hptt_create_plan_ex; an outer extent below the extent
 * it encloses is HPTT_ERROR_INVALID_ARGUMENT.
 */
hptt_status_t hptt_create_plan_outer(hptt_plan_t *plan, const int32_t *perm, int32_t N,
                                     const int64_t *sizeA, const int64_t *outerSizeA,
                                     const int64_t *outerSizeB, double alpha, double beta,
                                     hptt_dtype_t dtype, const hptt_options_t *options);

/* What hptt_create_plan_autotune did. */
typedef struct {
    int32_t candidates;      /* distinct plans generated */
    int32_t timed;           /* plans timed before the timeout */
    int32_t from_cache;      /* 1 when the problem was tuned earlier in this process */
    int32_t flushed;         /* 1 when launches were timed cold, with their write-backs */
    int32_t own_mode;        /* 1 when plans were timed writing a scratch tensor in the
                                caller's own update mode */
    float default_ms;        /* the quick path's plan, median of three cold launches */
    float best_ms;           /* the chosen plan, median of three cold launches */
    hptt_options_t options;  /* the chosen plan's knobs (all zero: the quick path's plan) */
    int32_t finalists;       /* candidates screened at least 1 % faster than the quick
                                plan and timed again against it (at most 3) */
    int32_t confirmed;       /* finalists that won again, cold and back to back */
} hptt_autotune_report_t;

/*
 * The autotune path of plan creation (Section 3.1): generate candidate plans
 * (tile shapes, tile orders, cache hints), rank them with the quick path's
 * plan first, then time them on the caller's own tensors, from good to bad,
 * until timeout_seconds have passed, and return a plan with the fastest one's
 * knobs for the given alpha and beta (the quick path's plan unless another
 * is at least 1 % faster).  Each plan is timed in the update mode it will
 * run in, as the median of three launches that each start after a 512 MiB
 * read has evicted the tensors from the caches; each timed span also holds a
 * second such read, which writes back what the launch left dirty in the
 * caches (its clean time is subtracted), so that plans whose stores stay in
 * the caches are charged for them as in back-to-back use.  The (at most)
 * three candidates screened fastest, each at least 1 % ahead of the quick
 * path's plan, are then timed again against it in five alternating rounds,
 * cold as above and in bursts of back-to-back launches that rotate over
 * scratch copies of A's and B's footprints (up to 8 sets, 2 GiB of traffic
 * between two uses of one set, as fits in memory; none beyond the caller's
 * own when A's and B's footprints alone exceed 2 GiB), so that no launch finds
 * its tensors in the caches; a finalist replaces the quick plan only if it is
 * at least 1 % faster in both sums (this confirmation runs after the timeout
 * and adds at most 60 timed spans).  The caller's data are not changed: the plans write a scratch
 * tensor of B's footprint (zeroed first when beta != 0) and B is not
 * touched.  The scratch memory (that tensor, the rotation copies and the
 * flush buffer) is allocated for the call and freed before it returns.  Without memory for
 * the scratch tensor, timing runs, like the paper's, on B itself with
 * alpha = 0 and beta = 1, so B is rewritten with its own value and A is read
 * and multiplied by zero (A must then hold no inf or NaN, footnote 5, and a
 * -0.0 in B comes back as +0.0); without memory for the flush buffer, timing
 * falls back to bursts of four back-to-back launches.  The chosen plan is cached per problem (perm,
 * extents, outer sizes, dtype, update mode, device) for the life of the
 * process; a cached problem returns at once without launching anything.
 *
 *   A, B     device pointers as for hptt_exec (used only for timing).
 *   stream   stream the timing launches are queued on; this call waits for it
 *            (and, through hipFree of the scratch memory, for the device).
 *   timeout_seconds  <= 0 returns the quick path's plan (or the cached one).
 *   report   may be NULL.
 * Errors: as hptt_create_plan_outer and hptt_exec.
 */
hptt_status_t hptt_create_plan_autotune(hptt_plan_t *plan, const int32_t *perm, int32_t N,
                                        const int64_t *sizeA, const int64_t *outerSizeA,
                                        const int64_t *outerSizeB, double alpha, double beta,
                                        hptt_dtype_t dtype, const void *A, void *B,
                                        hipStream_t stream, double timeout_seconds,
                                        hptt_autotune_report_t *report);

/* The candidate knobs hptt_create_plan_autotune would time for a problem, in
 * its order, written to options[0 .. min(count, max_options) - 1].  Returns
 * the count, or minus a status code for an invalid problem.  Makes no HIP
 * call. */
int32_t hptt_autotune_candidates(const int32_t *perm, int32_t N, const int64_t *sizeA,
                                 const int64_t *outerSizeA, const int64_t *outerSizeB,
                                 double alpha, double beta, hptt_dtype_t dtype,
                                 hptt_options_t *options, int32_t max_options);

/* Drop every cached autotuning result of this process. */
hptt_status_t hptt_forget_wisdom(void);

/*
 * Execute a plan (Fig. 3b's plan->exec()): queue the transposition of A into B
 * on `stream` and return without waiting.
 *
 *   A  device pointer to numel elements of dtype (read only); for a sub-tensor
 *      plan, to its first element, with footprint_a elements addressable.
 *   B  device pointer to numel elements of dtype, read only when beta != 0;
 *      for a sub-tensor plan, to its first element (footprint_b addressable).
 *   stream  HIP stream (0 = the null stream).
 * A and B must be aligned to the element size.  Pointers aligned to 16 bytes
 * get 16-byte vector accesses; others get narrower ones (still correct).
 * The plan is not modified, so one plan may execute concurrently on several
 * streams.  numel == 0 returns HPTT_SUCCESS without a launch.
 * Errors: HPTT_ERROR_INVALID_ARGUMENT (null plan; null or misaligned A or B),
 * HPTT_ERROR_OVERLAP (the byte ranges of A and B intersect; for sub-tensors
 * the ranges from first to last element), HPTT_ERROR_HIP
 * (the launch failed; see hptt_last_hip_error).
 */
hptt_status_t hptt_exec(hptt_plan_t plan, const void *A, void *B, hipStream_t stream);

/* Free a plan (NULL is accepted).  The plan must not be used afterwards; work
 * already queued by hptt_exec does not depend on it. */
hptt_status_t hptt_destroy_plan(hptt_plan_t plan);

/* Copy the plan builder's decisions into *info. */
hptt_status_t hptt_plan_info(hptt_plan_t plan, hptt_plan_info_t *info);

/* Write a one-line, NUL-terminated human-readable summary of the plan into
 * buf (at most len bytes, truncated if needed). */
hptt_status_t hptt_describe_plan(hptt_plan_t plan, char *buf, size_t len);

/* Static English name of a status code. */
const char *hptt_status_string(hptt_status_t status);

/* The hipError_t of the last failed launch on this thread (hipSuccess if none). */
int32_t hptt_last_hip_error(void);

/* Load the library's GPU code onto the current device now instead of at the
 * first hptt_exec that needs it.  Optional: a process whose first launches
 * are timed calls it once per device beforehand (the first dispatch of a
 * kernel from a not yet loaded code object leaves the next few milliseconds
 * of kernels several percent slower).  Blocks the calling thread; launches
 * nothing.  Errors: HPTT_ERROR_HIP (see hptt_last_hip_error). */
hptt_status_t hptt_load_kernels(void);

#ifdef __cplusplus
}
#endif

#endif /* HPTT_HIP_H */
