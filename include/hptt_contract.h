/*
 * Tensor contractions cast as transpositions around a matrix-matrix product
 * (the use of transpositions that motivates the paper: Section 1 and the
 * contraction experiment of Section 4.1, Eq. 3):
 *
 *     C_{modesC}  <-  alpha * sum_{contracted modes} A_{modesA} * B_{modesB}
 *                     +  beta * C_{modesC}
 *
 * All tensors are in the Fortran layout of Section 1 (first mode fastest).
 * A mode is one character; the modes of each tensor are distinct.  A mode in
 * A and B but not in C is contracted (summed over); a mode in A and C only,
 * or B and C only, is a free row or column mode; a mode in A, B and C is a
 * batch mode.  Every mode appears in at least two of the three tensors.
 *
 * The plan groups the modes into the matrices of one (batched) product on
 * the GPU's matrix cores (rocBLAS GEMM, column-major, which is the Fortran
 * layout) and transposes, with the library of hptt.h, only the operands
 * whose layout the product cannot read as it is: an operand already ordered
 * [rows, contracted, batch] or [contracted, rows, batch] is read in place
 * (the latter as a transposed matrix); C is written in place when it is
 * ordered [rows, columns, batch] or [columns, rows, batch].  Among the
 * layouts that qualify, the plan picks the one that moves the fewest bytes.
 *
 * Ownership: plans are opaque and own their transposition plans and their
 * rocBLAS handle, which the first execution creates on the device current
 * then (and an execution on another device replaces); execute a plan from
 * one host thread at a time.  The caller owns all tensors and the workspace.
 */
#ifndef HPTT_CONTRACT_H
#define HPTT_CONTRACT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "hptt.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hptt_contraction_s *hptt_contraction_t;

typedef struct {
    int32_t transpose_a;      /* 1: A is transposed into the workspace first */
    int32_t transpose_b;      /* 1: B is transposed into the workspace first */
    int32_t transpose_c;      /* 1: the product goes to the workspace, then is transposed into C */
    int32_t swap;             /* 1: the product is formed as C^T = B^T A^T */
    int32_t op_p;             /* 1: the first GEMM operand (A, or B when swapped) is read
                                 transposed: stored [K, X, L] instead of [X, K, L] */
    int32_t op_q;             /* 1: the second GEMM operand is read transposed: stored
                                 [Y, K, L] instead of [K, Y, L] */
    int64_t gemm_m, gemm_n, gemm_k, batch;   /* GEMM shape (column-major) and batch count */
    int64_t ld_p, ld_q, ld_c;                 /* leading dimensions of the GEMM operands */
    int64_t stride_p, stride_q, stride_c;     /* elements between batch entries */
    char modes_x[17];         /* GEMM rows (M modes, or N modes when swapped), in order */
    char modes_y[17];         /* GEMM columns */
    char modes_k[17];         /* contracted modes */
    char modes_l[17];         /* batch modes */
    int64_t workspace_bytes;  /* device workspace hptt_contraction_exec needs */
    double flops;             /* 2 * m * n * k * batch */
    double bytes_transposed;  /* bytes read and written by the transpositions */
} hptt_contraction_info_t;

/*
 * Plan C = alpha * A . B + beta * C.
 *   modesA, modesB, modesC   NUL-terminated mode strings, one character per
 *                            mode, in storage order (at most 16 modes each).
 *   sizeA, sizeB             extents of A's and B's modes (>= 1; a mode shared
 *                            by A and B has one extent); C's extents follow.
 * Returns HPTT_ERROR_INVALID_ARGUMENT for a repeated mode, a mode found in
 * one tensor only, mismatched or non-positive extents, an unknown dtype;
 * HPTT_ERROR_OUT_OF_MEMORY if the plan cannot be allocated.  Makes no HIP
 * call.
 */
hptt_status_t hptt_contraction_create(hptt_contraction_t *plan, hptt_dtype_t dtype,
                                      double alpha, double beta, const char *modesA,
                                      const int64_t *sizeA, const char *modesB,
                                      const int64_t *sizeB, const char *modesC);

/* Release a plan (NULL is a no-op). */
hptt_status_t hptt_contraction_destroy(hptt_contraction_t plan);

/* The plan's shape and the workspace it needs. */
hptt_status_t hptt_contraction_info(hptt_contraction_t plan, hptt_contraction_info_t *info);

/* One line describing the plan, NUL-terminated, truncated to len bytes. */
hptt_status_t hptt_contraction_describe(hptt_contraction_t plan, char *buf, size_t len);

/*
 * Queue the contraction on `stream`: transpositions of A and B into the
 * workspace where the plan needs them, the GEMM, the transposition of the
 * product into C where needed.  A, B, C and workspace are device pointers;
 * workspace must hold workspace_bytes (256-byte aligned, may be NULL when
 * that is 0) and overlap none of A, B, C.  Returns HPTT_ERROR_INVALID_ARGUMENT
 * for a NULL tensor or a missing or short workspace, HPTT_ERROR_HIP when a
 * launch or the GEMM fails (hptt_last_hip_error and
 * hptt_contraction_last_blas_status say which).
 */
hptt_status_t hptt_contraction_exec(hptt_contraction_t plan, const void *A, const void *B,
                                    void *C, void *workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/*
 * Size of the device array hptt_contraction_exec_no_alloc works in (64 MiB,
 * held by every device the library runs on until the process ends): its last
 * HPTT_CONTRACTION_STATIC_BLAS_BYTES are rocBLAS's workspace, the rest holds
 * the transposed operands and product (a plan's workspace_bytes).
 */
#define HPTT_CONTRACTION_STATIC_BYTES (64u << 20)
#define HPTT_CONTRACTION_STATIC_BLAS_BYTES (16u << 20)

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * contraction as hptt_contraction_exec, on the same kernels, with the
 * workspace taken from a file-scope device array instead of the caller.
 * Allocates nothing: no hipMalloc, hipFree or allocating library call.
 *
 * The first call on a device sets that device up (once, with it current):
 * it looks up the array's device address and creates a rocBLAS handle whose
 * workspace is the array's rocBLAS share, so that rocBLAS never allocates;
 * rocBLAS also loads a GEMM kernel's code the first time that kernel runs.
 * A caller that must never allocate therefore runs each plan once (on
 * tensors of its shape) before, e.g., capturing a graph.
 *
 * Every call on one device works in that device's one array, which keeps the
 * last call's contents (nothing in it needs to start at zero): calls that
 * overlap on one device -- from several host threads, or queued on streams
 * that run concurrently -- race and give wrong results.  Order them on one
 * stream, or use hptt_contraction_exec with a workspace per stream.
 *
 * Returns HPTT_ERROR_INVALID_ARGUMENT for a NULL plan or tensor;
 * HPTT_ERROR_UNSUPPORTED when the plan's workspace_bytes exceed
 * HPTT_CONTRACTION_STATIC_BYTES - HPTT_CONTRACTION_STATIC_BLAS_BYTES (48 MiB),
 * when rocBLAS would need more than HPTT_CONTRACTION_STATIC_BLAS_BYTES for
 * the GEMM, or for a device ordinal of 64 or more; HPTT_ERROR_HIP when the
 * set-up, a launch or the GEMM fails (hptt_contraction_last_blas_status
 * gives rocBLAS's status).  Nothing is queued when the plan does not fit.
 */
hptt_status_t hptt_contraction_exec_no_alloc(hptt_contraction_t plan, const void *A,
                                             const void *B, void *C, hipStream_t stream);

/* The rocBLAS status of this thread's last failed GEMM (0 if none). */
int32_t hptt_contraction_last_blas_status(void);

#ifdef __cplusplus
}
#endif

#endif /* HPTT_CONTRACT_H */
