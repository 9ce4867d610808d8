// Tensor contractions as transposition - GEMM - transposition (Section 1;
// the contraction experiment of Section 4.1).  The plan groups the modes
// into the rows (X), columns (Y), contracted (K) and batch (L) modes of one
// column-major strided-batched GEMM, C'[X,Y,L] = P[X,K,L] . Q[K,Y,L], and
// searches the mode orders and the role of A and B (P = A, Q = B, or the
// transposed product P = B, Q = A) for the arrangement that transposes the
// fewest bytes.  The transpositions are plans of the transposition library.
#include <rocblas/rocblas.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <stdio.h>
#include <string.h>
#include <string>
#include <vector>

#include "hptt_contract.h"

namespace {

constexpr int kMaxModes = 16;
constexpr int64_t kAlign = 256;

thread_local int32_t t_blasStatus = 0;

struct Choice {
    std::string x, y, k, l;  // mode orders of the GEMM's rows, columns, contraction, batch
    int swap = 0;            // 0: P = A, Q = B; 1: P = B, Q = A
    int opP = 0, opQ = 0;    // operand read transposed in place
    bool tP = false, tQ = false, tC = false;
    double cost = 0;         // elements moved by the transpositions
};

// All orders of a mode group worth trying: the order in which the group's
// modes appear in each tensor that holds all of them.
std::vector<std::string> orders(const std::string& group, const std::vector<std::string>& tensors) {
    std::vector<std::string> out;
    for (const std::string& t : tensors) {
        std::string o;
        for (char c : t)
            if (group.find(c) != std::string::npos) o += c;
        if (o.size() == group.size() && std::find(out.begin(), out.end(), o) == out.end())
            out.push_back(o);
    }
    if (out.empty()) out.push_back(group);
    return out;
}

int64_t volume(const std::string& modes, const int64_t* ext) {
    int64_t v = 1;
    for (char c : modes) v *= ext[static_cast<unsigned char>(c)];
    return v;
}

bool valid_modes(const char* m, int* n) {
    if (!m) return false;
    const size_t len = strlen(m);
    if (len > size_t(kMaxModes)) return false;
    for (size_t i = 0; i < len; ++i)
        for (size_t j = i + 1; j < len; ++j)
            if (m[i] == m[j]) return false;
    *n = int(len);
    return true;
}

// perm[k] = position in `from` of the mode at position k of `to`.
void permutation(const std::string& from, const std::string& to, int32_t* perm) {
    for (size_t k = 0; k < to.size(); ++k) perm[k] = int32_t(from.find(to[k]));
}

}  // namespace

struct hptt_contraction_s {
    hptt_dtype_t dtype;
    double alpha, beta;
    std::string ma, mb, mc;
    int64_t ext[256];
    Choice ch;
    hptt_plan_t planP = nullptr, planQ = nullptr, planC = nullptr;
    int64_t offP = 0, offQ = 0, offC = 0, wsBytes = 0;
    rocblas_handle handle = nullptr;
    int handleDevice = -1;
    hptt_contraction_info_t info;
    std::string desc;

    ~hptt_contraction_s() {
        hptt_destroy_plan(planP);
        hptt_destroy_plan(planQ);
        hptt_destroy_plan(planC);
        if (handle) (void)rocblas_destroy_handle(handle);
    }
};

namespace {

hptt_status_t make_transpose(const std::string& from, const std::string& to, const int64_t* ext,
                             double alpha, double beta, hptt_dtype_t dtype, hptt_plan_t* plan) {
    const int n = int(from.size());
    if (n == 0) return HPTT_SUCCESS;  // a scalar needs no transposition (never planned)
    int32_t perm[kMaxModes];
    int64_t size[kMaxModes];
    permutation(from, to, perm);
    for (int d = 0; d < n; ++d) size[d] = ext[static_cast<unsigned char>(from[d])];
    return hptt_create_plan(plan, perm, n, size, alpha, beta, dtype);
}

int64_t align_up(int64_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

}  // namespace

extern "C" {

hptt_status_t hptt_contraction_create(hptt_contraction_t* planOut, hptt_dtype_t dtype,
                                      double alpha, double beta, const char* modesA,
                                      const int64_t* sizeA, const char* modesB,
                                      const int64_t* sizeB, const char* modesC) {
    if (!planOut) return HPTT_ERROR_INVALID_ARGUMENT;
    *planOut = nullptr;
    int na = 0, nb = 0, nc = 0;
    if (dtype != HPTT_FLOAT32 && dtype != HPTT_FLOAT64) return HPTT_ERROR_INVALID_ARGUMENT;
    if (!valid_modes(modesA, &na) || !valid_modes(modesB, &nb) || !valid_modes(modesC, &nc))
        return HPTT_ERROR_INVALID_ARGUMENT;
    if ((na && !sizeA) || (nb && !sizeB)) return HPTT_ERROR_INVALID_ARGUMENT;
    const std::string A(modesA), B(modesB), C(modesC);
    int64_t ext[256];
    for (int64_t& e : ext) e = 0;
    for (int i = 0; i < na; ++i) {
        if (sizeA[i] < 1) return HPTT_ERROR_INVALID_ARGUMENT;
        ext[static_cast<unsigned char>(A[i])] = sizeA[i];
    }
    for (int i = 0; i < nb; ++i) {
        int64_t& e = ext[static_cast<unsigned char>(B[i])];
        if (sizeB[i] < 1 || (e && e != sizeB[i])) return HPTT_ERROR_INVALID_ARGUMENT;
        e = sizeB[i];
    }
    // Classify: rows of A (M), columns of B (N), contracted (K), batch (L).
    std::string M, N, K, L;
    for (char c : C) {
        const bool inA = A.find(c) != std::string::npos, inB = B.find(c) != std::string::npos;
        if (inA && inB) L += c;
        else if (inA) M += c;
        else if (inB) N += c;
        else return HPTT_ERROR_INVALID_ARGUMENT;  // a mode of C from nowhere
    }
    for (char c : A)
        if (C.find(c) == std::string::npos) {
            if (B.find(c) == std::string::npos) return HPTT_ERROR_INVALID_ARGUMENT;
            K += c;
        }
    for (char c : B)
        if (C.find(c) == std::string::npos && A.find(c) == std::string::npos)
            return HPTT_ERROR_INVALID_ARGUMENT;
    const double vA = double(volume(A, ext)), vB = double(volume(B, ext)),
                 vC = double(volume(C, ext));
    // Search mode orders and roles for the fewest extra elements moved: a
    // transposed operand is read and written once more than the GEMM alone
    // would read it; a transposed product is written and read once more.
    Choice best;
    bool found = false;
    for (int swap = 0; swap < 2; ++swap) {
        const std::string& X = swap ? N : M;
        const std::string& Y = swap ? M : N;
        const std::string& P = swap ? B : A;
        const std::string& Q = swap ? A : B;
        for (const std::string& xo : orders(X, {C, P}))
            for (const std::string& yo : orders(Y, {C, Q}))
                for (const std::string& ko : orders(K, {P, Q}))
                    for (const std::string& lo : orders(L, {C, P, Q})) {
                        Choice c;
                        c.x = xo, c.y = yo, c.k = ko, c.l = lo, c.swap = swap;
                        if (P == xo + ko + lo) c.opP = 0;
                        else if (P == ko + xo + lo) c.opP = 1;
                        else c.tP = true;
                        if (Q == ko + yo + lo) c.opQ = 0;
                        else if (Q == yo + ko + lo) c.opQ = 1;
                        else c.tQ = true;
                        c.tC = C != xo + yo + lo;
                        const double vP = swap ? vB : vA, vQ = swap ? vA : vB;
                        c.cost = (c.tP ? 2 * vP : 0) + (c.tQ ? 2 * vQ : 0) + (c.tC ? 2 * vC : 0);
                        if (!found || c.cost < best.cost) {
                            best = c;
                            found = true;
                        }
                    }
    }
    hptt_contraction_s* p = new (std::nothrow) hptt_contraction_s();
    if (!p) return HPTT_ERROR_OUT_OF_MEMORY;
    p->dtype = dtype;
    p->alpha = alpha;
    p->beta = beta;
    p->ma = A, p->mb = B, p->mc = C;
    memcpy(p->ext, ext, sizeof(ext));
    p->ch = best;
    const Choice& c = p->ch;
    const int64_t elem = dtype == HPTT_FLOAT32 ? 4 : 8;
    const std::string& P = c.swap ? B : A;
    const std::string& Q = c.swap ? A : B;
    hptt_status_t st = HPTT_SUCCESS;
    int64_t ws = 0;
    if (c.tP) {  // P -> [X, K, L], read untransposed
        st = make_transpose(P, c.x + c.k + c.l, ext, 1.0, 0.0, dtype, &p->planP);
        p->offP = ws;
        ws = align_up(ws + volume(P, ext) * elem);
    }
    if (st == HPTT_SUCCESS && c.tQ) {  // Q -> [K, Y, L]
        st = make_transpose(Q, c.k + c.y + c.l, ext, 1.0, 0.0, dtype, &p->planQ);
        p->offQ = ws;
        ws = align_up(ws + volume(Q, ext) * elem);
    }
    if (st == HPTT_SUCCESS && c.tC) {  // [X, Y, L] -> C, adding beta * C
        st = make_transpose(c.x + c.y + c.l, C, ext, 1.0, beta, dtype, &p->planC);
        p->offC = ws;
        ws = align_up(ws + volume(C, ext) * elem);
    }
    if (st != HPTT_SUCCESS) {
        delete p;
        return st;
    }
    p->wsBytes = ws;
    hptt_contraction_info_t& in = p->info;
    memset(&in, 0, sizeof(in));
    in.transpose_a = c.swap ? c.tQ : c.tP;
    in.transpose_b = c.swap ? c.tP : c.tQ;
    in.transpose_c = c.tC;
    in.swap = c.swap;
    in.op_p = c.opP;
    in.op_q = c.opQ;
    in.gemm_m = volume(c.x, ext);
    in.gemm_n = volume(c.y, ext);
    in.gemm_k = volume(c.k, ext);
    in.batch = volume(c.l, ext);
    in.ld_p = c.opP ? in.gemm_k : in.gemm_m;
    in.ld_q = c.opQ ? in.gemm_n : in.gemm_k;
    in.ld_c = in.gemm_m;
    in.stride_p = in.gemm_m * in.gemm_k;
    in.stride_q = in.gemm_k * in.gemm_n;
    in.stride_c = in.gemm_m * in.gemm_n;
    snprintf(in.modes_x, sizeof(in.modes_x), "%s", c.x.c_str());
    snprintf(in.modes_y, sizeof(in.modes_y), "%s", c.y.c_str());
    snprintf(in.modes_k, sizeof(in.modes_k), "%s", c.k.c_str());
    snprintf(in.modes_l, sizeof(in.modes_l), "%s", c.l.c_str());
    in.workspace_bytes = ws;
    in.flops = 2.0 * double(in.gemm_m) * double(in.gemm_n) * double(in.gemm_k) * double(in.batch);
    {
        const double vP = c.swap ? vB : vA, vQ = c.swap ? vA : vB;
        in.bytes_transposed = double(elem) * ((c.tP ? 2 * vP : 0) + (c.tQ ? 2 * vQ : 0) +
                                              (c.tC ? (beta != 0 ? 3 : 2) * vC : 0));
    }
    char buf[512];
    snprintf(buf, sizeof(buf),
             "contraction %s=%s*%s dtype=%s gemm=%s%s m=%lld(%s) n=%lld(%s) k=%lld(%s) "
             "batch=%lld(%s) transpose A=%d B=%d C=%d workspace=%lld",
             C.c_str(), A.c_str(), B.c_str(), dtype == HPTT_FLOAT32 ? "f32" : "f64",
             c.opP ? "T" : "N", c.opQ ? "T" : "N", (long long)in.gemm_m, c.x.c_str(),
             (long long)in.gemm_n, c.y.c_str(), (long long)in.gemm_k, c.k.c_str(),
             (long long)in.batch, c.l.c_str(), in.transpose_a, in.transpose_b, in.transpose_c,
             (long long)ws);
    p->desc = buf;
    if (c.swap) p->desc += " (as C^T = B^T A^T)";
    *planOut = p;
    return HPTT_SUCCESS;
}

hptt_status_t hptt_contraction_destroy(hptt_contraction_t plan) {
    delete plan;
    return HPTT_SUCCESS;
}

hptt_status_t hptt_contraction_info(hptt_contraction_t plan, hptt_contraction_info_t* info) {
    if (!plan || !info) return HPTT_ERROR_INVALID_ARGUMENT;
    *info = plan->info;
    return HPTT_SUCCESS;
}

hptt_status_t hptt_contraction_describe(hptt_contraction_t plan, char* buf, size_t len) {
    if (!plan || !buf || len == 0) return HPTT_ERROR_INVALID_ARGUMENT;
    snprintf(buf, len, "%s", plan->desc.c_str());
    return HPTT_SUCCESS;
}

int32_t hptt_contraction_last_blas_status(void) { return t_blasStatus; }

}  // extern "C"

namespace {

// The GEMM of a plan on `handle`, queued on the handle's stream (inside a
// rocBLAS device-memory size query nothing runs: the call only reports the
// workspace the GEMM would need).
rocblas_status gemm(const hptt_contraction_s* p, rocblas_handle handle, const void* P,
                    const void* Q, void* out) {
    const Choice& c = p->ch;
    const hptt_contraction_info_t& in = p->info;
    const int64_t m = in.gemm_m, n = in.gemm_n, k = in.gemm_k;
    const rocblas_operation oP = c.opP ? rocblas_operation_transpose : rocblas_operation_none;
    const rocblas_operation oQ = c.opQ ? rocblas_operation_transpose : rocblas_operation_none;
    if (p->dtype == HPTT_FLOAT32) {
        const float al = float(p->alpha), be = c.tC ? 0.f : float(p->beta);
        return rocblas_sgemm_strided_batched_64(
            handle, oP, oQ, m, n, k, &al, static_cast<const float*>(P), in.ld_p, in.stride_p,
            static_cast<const float*>(Q), in.ld_q, in.stride_q, &be, static_cast<float*>(out),
            in.ld_c, in.stride_c, in.batch);
    }
    const double al = p->alpha, be = c.tC ? 0.0 : p->beta;
    return rocblas_dgemm_strided_batched_64(
        handle, oP, oQ, m, n, k, &al, static_cast<const double*>(P), in.ld_p, in.stride_p,
        static_cast<const double*>(Q), in.ld_q, in.stride_q, &be, static_cast<double*>(out),
        in.ld_c, in.stride_c, in.batch);
}

// Queue a plan with the given workspace (wsBytes of it at least) and rocBLAS
// handle: the transpositions of A and B into the workspace where needed, the
// GEMM, the transposition of the product into C where needed.
hptt_status_t run(const hptt_contraction_s* p, const void* A, const void* B, void* C,
                  void* workspace, rocblas_handle handle, hipStream_t stream) {
    const Choice& c = p->ch;
    char* ws = static_cast<char*>(workspace);
    const void* P = c.swap ? B : A;
    const void* Q = c.swap ? A : B;
    hptt_status_t st = HPTT_SUCCESS;
    if (c.tP) {
        st = hptt_exec(p->planP, P, ws + p->offP, stream);
        P = ws + p->offP;
    }
    if (st == HPTT_SUCCESS && c.tQ) {
        st = hptt_exec(p->planQ, Q, ws + p->offQ, stream);
        Q = ws + p->offQ;
    }
    if (st != HPTT_SUCCESS) return st;
    void* out = c.tC ? static_cast<void*>(ws + p->offC) : C;
    rocblas_status bs = rocblas_set_stream(handle, stream);
    if (bs == rocblas_status_success) bs = gemm(p, handle, P, Q, out);
    if (bs != rocblas_status_success) {
        t_blasStatus = int32_t(bs);
        return HPTT_ERROR_HIP;
    }
    if (c.tC) st = hptt_exec(p->planC, out, C, stream);
    return st;
}

}  // namespace

extern "C" {

hptt_status_t hptt_contraction_exec(hptt_contraction_t p, const void* A, const void* B, void* C,
                                    void* workspace, size_t workspaceBytes, hipStream_t stream) {
    if (!p || !A || !B || !C) return HPTT_ERROR_INVALID_ARGUMENT;
    if (p->wsBytes > 0 && (!workspace || workspaceBytes < size_t(p->wsBytes) ||
                           reinterpret_cast<uintptr_t>(workspace) % kAlign))
        return HPTT_ERROR_INVALID_ARGUMENT;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return HPTT_ERROR_HIP;
    if (!p->handle || p->handleDevice != device) {
        if (p->handle) (void)rocblas_destroy_handle(p->handle);
        p->handle = nullptr;
        const rocblas_status bs = rocblas_create_handle(&p->handle);
        if (bs != rocblas_status_success) {
            t_blasStatus = int32_t(bs);
            p->handle = nullptr;
            return HPTT_ERROR_HIP;
        }
        p->handleDevice = device;
    }
    return run(p, A, B, C, workspace, p->handle, stream);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Execution without allocation: the workspace is a file-scope device array,
// HPTT_CONTRACTION_STATIC_BYTES long; rocBLAS gets its last
// HPTT_CONTRACTION_STATIC_BLAS_BYTES as a user-owned workspace, the
// transposed operands and products the rest.

static __device__ __align__(256) unsigned char scratch[HPTT_CONTRACTION_STATIC_BYTES];

namespace {

constexpr size_t kStaticWorkspace =
    size_t(HPTT_CONTRACTION_STATIC_BYTES) - size_t(HPTT_CONTRACTION_STATIC_BLAS_BYTES);
constexpr int kMaxDevices = 64;

// Per device, set up by the first call on it: the array's device address
// (each device holds its own copy of the array) and a rocBLAS handle whose
// workspace is the array's rocBLAS share, so that no GEMM allocates.
struct StaticDevice {
    char* base = nullptr;
    rocblas_handle handle = nullptr;
};
std::mutex g_staticMutex;
StaticDevice g_static[kMaxDevices];

}  // namespace

extern "C" {

hptt_status_t hptt_contraction_exec_no_alloc(hptt_contraction_t p, const void* A, const void* B,
                                             void* C, hipStream_t stream) {
    if (!p || !A || !B || !C) return HPTT_ERROR_INVALID_ARGUMENT;
    if (size_t(p->wsBytes) > kStaticWorkspace) return HPTT_ERROR_UNSUPPORTED;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return HPTT_ERROR_HIP;
    if (device < 0 || device >= kMaxDevices) return HPTT_ERROR_UNSUPPORTED;
    StaticDevice dev;
    {
        std::lock_guard<std::mutex> lock(g_staticMutex);
        StaticDevice& d = g_static[device];
        if (!d.base) {  // set-up, once per device, with that device current
            void* ptr = nullptr;
            if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
                (void)hipGetLastError();
                return HPTT_ERROR_HIP;
            }
            rocblas_handle h = nullptr;
            rocblas_status bs = rocblas_create_handle(&h);
            if (bs == rocblas_status_success)
                bs = rocblas_set_workspace(h, static_cast<char*>(ptr) + kStaticWorkspace,
                                           size_t(HPTT_CONTRACTION_STATIC_BLAS_BYTES));
            if (bs != rocblas_status_success) {
                if (h) (void)rocblas_destroy_handle(h);
                t_blasStatus = int32_t(bs);
                return HPTT_ERROR_HIP;
            }
            d.handle = h;
            d.base = static_cast<char*>(ptr);
        }
        dev = d;
    }
    // The GEMM must fit rocBLAS's share of the array: ask rocBLAS (a size
    // query runs nothing; the tensors stand in for the operands).
    size_t need = 0;
    rocblas_status bs = rocblas_start_device_memory_size_query(dev.handle);
    if (bs == rocblas_status_success) {
        const rocblas_status q = gemm(p, dev.handle, A, B, C);
        bs = rocblas_stop_device_memory_size_query(dev.handle, &need);
        if (q != rocblas_status_success && q != rocblas_status_size_increased &&
            q != rocblas_status_size_unchanged)
            bs = q;
    }
    if (bs != rocblas_status_success) {
        t_blasStatus = int32_t(bs);
        return HPTT_ERROR_HIP;
    }
    if (need > size_t(HPTT_CONTRACTION_STATIC_BLAS_BYTES)) return HPTT_ERROR_UNSUPPORTED;
    return run(p, A, B, C, dev.base, dev.handle, stream);
}

}  // extern "C"
