/*
 * Oracle for the out-of-place tensor transposition of Eq. (1) of the HPTT
 * paper (Springer, Su, Bientinesi; Section 1):
 *
 *     B_{Pi(i_1 .. i_N)}  <-  alpha * A_{i_1 .. i_N}  +  beta * B_{Pi(i_1 .. i_N)}
 *
 * with both tensors stored in the Fortran layout fixed in Section 1 (the
 * first index is the stride-1 index, the last one the slowest).
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test-suite, the smoke check
 * of the entry module and the CPU-baseline leg of the benchmark may build,
 * load or call this file.  It shares no code, header, table or helper with the
 * GPU library: it is a plain, slow, obviously correct CPU definition that the
 * GPU path is compared against.
 *
 * Readings taken where the paper is silent:
 *  - perm is 0-based (Fig. 3b passes a zero-based vector) and perm[k] names
 *    the A index that sits at position k of B (Table 1 and the text below it:
 *    the column "6,1,5,4,3,2" is B_{i6 i1 i5 i4 i3 i2}).  Hence
 *    sizeB[k] = sizeA[perm[k]] (Fig. 3b: perm {2,1,0}, sizeA {8,16,16} gives
 *    a compact B of {16,16,8}).
 *  - beta == 0 overwrites B without reading it (Eq. 2 counts B once, lambda=2).
 *  - alpha == 1 and beta == 0 is a bit-exact copy.
 *  - alpha == 0 is not short-cut: A is still read and multiplied (the
 *    non-destructive autotuning of Section 3.1 relies on alpha = 0, beta = 1
 *    and requires A to be free of inf/NaN, footnote 5).
 *  - Arithmetic happens in the tensor's own precision (the paper's kernels take
 *    float tensors and float scalars, Fig. 5): alpha*a and beta*b are each
 *    rounded once, then their sum is rounded once; no fused multiply-add.
 *    Build with -ffp-contract=off.
 *  - Any extent 0 makes the operation a no-op; extent-1 indices are allowed.
 *  - Outer sizes (Section 3.1, Fig. 3): A and B may be sub-tensors of larger
 *    enclosing tensors, like a BLAS leading dimension.  Their strides are the
 *    Fortran strides of the enclosing extents outerSizeA (in A's index order)
 *    and outerSizeB (in B's index order); the pointers address the
 *    sub-tensors' first elements; elements of B outside the sub-tensor are
 *    neither read nor written.  Each outer extent must be >= the extent it
 *    encloses.  NULL outer sizes mean compact tensors.
 */
#include <stddef.h>
#include <stdint.h>

#define ORACLE_MAX_DIMS 16

/* Return 0 when perm is a permutation of 0..N-1 and every extent is >= 0. */
static int check_problem(int N, const int64_t *sizeA, const int32_t *perm)
{
    int seen[ORACLE_MAX_DIMS] = {0};
    if (N < 1 || N > ORACLE_MAX_DIMS) return 1;
    for (int k = 0; k < N; ++k) {
        if (perm[k] < 0 || perm[k] >= N || seen[perm[k]]) return 2;
        seen[perm[k]] = 1;
        if (sizeA[k] < 0) return 3;
    }
    return 0;
}

/* Compact sizes of B: position k of B carries A index perm[k] (Fig. 3b). */
int oracle_size_b(int N, const int64_t *sizeA, const int32_t *perm, int64_t *sizeB)
{
    int err = check_problem(N, sizeA, perm);
    if (err) return err;
    for (int k = 0; k < N; ++k) sizeB[k] = sizeA[perm[k]];
    return 0;
}

/* Fortran strides of a compact tensor (Section 1): the first index has
 * stride 1 and each next stride is the previous stride times the previous
 * extent (the strides of Fig. 1 follow this rule). */
static void fortran_strides(int N, const int64_t *size, int64_t *stride)
{
    stride[0] = 1;
    for (int d = 1; d < N; ++d) stride[d] = stride[d - 1] * size[d - 1];
}

static int64_t numel_of(int N, const int64_t *size)
{
    int64_t n = 1;
    for (int d = 0; d < N; ++d) n *= size[d];
    return n;
}

/* Offsets of one A multi-index i in A and in B. */
static void offsets(int N, const int64_t *i, const int32_t *perm,
                    const int64_t *strideA, const int64_t *strideB,
                    int64_t *offA, int64_t *offB)
{
    int64_t a = 0, b = 0;
    for (int d = 0; d < N; ++d) a += i[d] * strideA[d];
    for (int k = 0; k < N; ++k) b += i[perm[k]] * strideB[k];
    *offA = a;
    *offB = b;
}

/* Advance the A multi-index in Fortran order; return 0 once it wraps. */
static int next_index(int N, const int64_t *sizeA, int64_t *i)
{
    for (int d = 0; d < N; ++d) {
        if (++i[d] < sizeA[d]) return 1;
        i[d] = 0;
    }
    return 0;
}

/* One element of Eq. (1), in float. */
static float update_f32(float a, float b, float alpha, float beta)
{
    if (beta == 0.0f) {
        if (alpha == 1.0f) return a;         /* bit-exact copy */
        return alpha * a;                    /* B is not read */
    }
    float scaled_a = alpha * a;
    float scaled_b = beta * b;
    return scaled_a + scaled_b;
}

/* One element of Eq. (1), in double. */
static double update_f64(double a, double b, double alpha, double beta)
{
    if (beta == 0.0) {
        if (alpha == 1.0) return a;
        return alpha * a;
    }
    double scaled_a = alpha * a;
    double scaled_b = beta * b;
    return scaled_a + scaled_b;
}

/* Check the outer extents and derive both tensors' strides. */
static int outer_strides(int N, const int64_t *sizeA, const int32_t *perm,
                         const int64_t *outerSizeA, const int64_t *outerSizeB,
                         int64_t *strideA, int64_t *strideB)
{
    int64_t sizeB[ORACLE_MAX_DIMS], outerA[ORACLE_MAX_DIMS], outerB[ORACLE_MAX_DIMS];
    int err = oracle_size_b(N, sizeA, perm, sizeB);
    if (err) return err;
    for (int d = 0; d < N; ++d) {
        outerA[d] = outerSizeA ? outerSizeA[d] : sizeA[d];
        outerB[d] = outerSizeB ? outerSizeB[d] : sizeB[d];
        if (outerA[d] < sizeA[d] || outerB[d] < sizeB[d]) return 5;
    }
    fortran_strides(N, outerA, strideA);
    fortran_strides(N, outerB, strideB);
    return 0;
}

/* The whole transposition: visit every multi-index of A once, in Fortran
 * order, and update the B element it maps to.  Returns 0 on success. */
int oracle_transpose_outer_f32(int N, const int64_t *sizeA, const int32_t *perm,
                               const int64_t *outerSizeA, const int64_t *outerSizeB,
                               float alpha, float beta, const float *A, float *B)
{
    int64_t strideA[ORACLE_MAX_DIMS], strideB[ORACLE_MAX_DIMS];
    int64_t i[ORACLE_MAX_DIMS] = {0};
    int err = outer_strides(N, sizeA, perm, outerSizeA, outerSizeB, strideA, strideB);
    if (err) return err;
    if (numel_of(N, sizeA) == 0) return 0;
    do {
        int64_t offA, offB;
        offsets(N, i, perm, strideA, strideB, &offA, &offB);
        B[offB] = update_f32(A[offA], beta == 0.0f ? 0.0f : B[offB], alpha, beta);
    } while (next_index(N, sizeA, i));
    return 0;
}

int oracle_transpose_outer_f64(int N, const int64_t *sizeA, const int32_t *perm,
                               const int64_t *outerSizeA, const int64_t *outerSizeB,
                               double alpha, double beta, const double *A, double *B)
{
    int64_t strideA[ORACLE_MAX_DIMS], strideB[ORACLE_MAX_DIMS];
    int64_t i[ORACLE_MAX_DIMS] = {0};
    int err = outer_strides(N, sizeA, perm, outerSizeA, outerSizeB, strideA, strideB);
    if (err) return err;
    if (numel_of(N, sizeA) == 0) return 0;
    do {
        int64_t offA, offB;
        offsets(N, i, perm, strideA, strideB, &offA, &offB);
        B[offB] = update_f64(A[offA], beta == 0.0 ? 0.0 : B[offB], alpha, beta);
    } while (next_index(N, sizeA, i));
    return 0;
}

/* Compact tensors: outer sizes equal the sizes. */
int oracle_transpose_f32(int N, const int64_t *sizeA, const int32_t *perm,
                         float alpha, float beta, const float *A, float *B)
{
    return oracle_transpose_outer_f32(N, sizeA, perm, 0, 0, alpha, beta, A, B);
}

int oracle_transpose_f64(int N, const int64_t *sizeA, const int32_t *perm,
                         double alpha, double beta, const double *A, double *B)
{
    return oracle_transpose_outer_f64(N, sizeA, perm, 0, 0, alpha, beta, A, B);
}

/* Expected B values at a list of B offsets, computed one by one: each B
 * offset is split into B's multi-index j (Fortran order over sizeB), the A
 * index is i[perm[k]] = j[k], and Eq. (1) is applied to A at that index and
 * to the prior B value Bin at the same B offset (ignored when beta == 0).
 * For tensors too large to transpose whole on the CPU.  Returns 0 on success,
 * 4 when an offset lies outside B. */
static int locate(int N, const int64_t *sizeA, const int32_t *perm,
                  int64_t offB, int64_t *offA)
{
    int64_t sizeB[ORACLE_MAX_DIMS], strideA[ORACLE_MAX_DIMS], i[ORACLE_MAX_DIMS];
    oracle_size_b(N, sizeA, perm, sizeB);
    fortran_strides(N, sizeA, strideA);
    if (offB < 0 || offB >= numel_of(N, sizeB)) return 4;
    for (int k = 0; k < N; ++k) {
        i[perm[k]] = offB % sizeB[k];
        offB /= sizeB[k];
    }
    int64_t a = 0;
    for (int d = 0; d < N; ++d) a += i[d] * strideA[d];
    *offA = a;
    return 0;
}

int oracle_sample_f32(int N, const int64_t *sizeA, const int32_t *perm,
                      float alpha, float beta, const float *A, const float *Bin,
                      int64_t count, const int64_t *offB, float *out)
{
    int err = check_problem(N, sizeA, perm);
    if (err) return err;
    for (int64_t s = 0; s < count; ++s) {
        int64_t offA;
        err = locate(N, sizeA, perm, offB[s], &offA);
        if (err) return err;
        out[s] = update_f32(A[offA], beta == 0.0f ? 0.0f : Bin[offB[s]], alpha, beta);
    }
    return 0;
}

int oracle_sample_f64(int N, const int64_t *sizeA, const int32_t *perm,
                      double alpha, double beta, const double *A, const double *Bin,
                      int64_t count, const int64_t *offB, double *out)
{
    int err = check_problem(N, sizeA, perm);
    if (err) return err;
    for (int64_t s = 0; s < count; ++s) {
        int64_t offA;
        err = locate(N, sizeA, perm, offB[s], &offA);
        if (err) return err;
        out[s] = update_f64(A[offA], beta == 0.0 ? 0.0 : Bin[offB[s]], alpha, beta);
    }
    return 0;
}
