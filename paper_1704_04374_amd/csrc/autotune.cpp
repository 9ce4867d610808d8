// The autotune path of plan creation (Section 3.1): generate candidate plans,
// rank them with the heuristic plan first, then time them on the caller's own
// tensors, from good to bad, until a timeout, and keep the fastest (FFTW
// style).  Timing runs with alpha = 0 and beta = 1, so B is rewritten with
// its own value and A is read and multiplied by zero (Section 3.1; A must not
// hold inf or NaN, footnote 5).  Winners are cached per problem for the life
// of the process.
#include <hip/hip_runtime_api.h>

#include <chrono>
#include <map>
#include <mutex>
#include <string.h>
#include <string>
#include <vector>

#include "plan.h"

namespace hptt {
namespace {

constexpr int kMaxCandidates = 256;

// A problem's cache key: everything the plan depends on except alpha and
// beta's values (only whether they make a copy, a scale or an update).
std::string cache_key(const int32_t* perm, int32_t N, const int64_t* sizeA,
                      const int64_t* outerA, const int64_t* outerB, hptt_dtype_t dtype, int mode,
                      int device) {
    std::string k = std::to_string(int(dtype)) + "|" + std::to_string(mode) + "|" +
                    std::to_string(device) + "|";
    for (int d = 0; d < N; ++d) {
        k += std::to_string(perm[d]) + ":" + std::to_string(sizeA[d]) + ":" +
             std::to_string(outerA ? outerA[d] : -1) + ":" + std::to_string(outerB ? outerB[d] : -1) +
             ",";
    }
    return k;
}

std::mutex g_mutex;
std::map<std::string, hptt_options_t> g_wisdom;

bool same_plan(const hptt_plan_s& a, const hptt_plan_s& b) {
    if (a.info.kernel != b.info.kernel || a.info.hints != b.info.hints) return false;
    if (a.info.kernel == HPTT_KERNEL_TILE)
        return memcmp(&a.tile, &b.tile, sizeof(a.tile)) == 0;
    return true;
}

int mode_of(hptt_dtype_t dtype, double alpha, double beta) {
    const double a = dtype == HPTT_FLOAT32 ? double(float(alpha)) : alpha;
    const double b = dtype == HPTT_FLOAT32 ? double(float(beta)) : beta;
    return b != 0.0 ? kAxpby : (a == 1.0 ? kCopy : kScale);
}

}  // namespace

// Candidate options, heuristic plan first, then variations ordered by how
// many knobs they change; candidates that build the same plan as an earlier
// one are dropped.
int autotune_candidates(const int32_t* perm, int32_t N, const int64_t* sizeA,
                        const int64_t* outerA, const int64_t* outerB, double alpha, double beta,
                        hptt_dtype_t dtype, hptt_options_t* out, int maxOut) {
    hptt_plan_s base;
    hptt_status_t st = build_plan(perm, N, sizeA, outerA, outerB, alpha, beta, dtype, nullptr, &base);
    if (st != HPTT_SUCCESS) return -int(st);
    std::vector<hptt_options_t> cand;
    hptt_options_t o;
    memset(&o, 0, sizeof(o));
    cand.push_back(o);  // the quick path's own choice
    const int elem = dtype == HPTT_FLOAT32 ? 4 : 8;
    const int32_t hintsStore[] = {0, 1, 2, 2, 1};
    const int32_t hintsLoad[] = {0, 1, 1, 2, 2};
    if (base.info.kernel == HPTT_KERNEL_TILE) {
        const int32_t aBytes[] = {0, 256, 1024, 128};
        const int32_t bBytes[] = {0, 256, 512};
        std::vector<std::pair<int, hptt_options_t>> var;
        for (int ia = 0; ia < 4; ++ia)
            for (int ib = 0; ib < 3; ++ib)
                for (int ord = 0; ord < 2; ++ord)
                    for (int ex = 0; ex < 2; ++ex)
                        for (int h = 0; h < 5; ++h) {
                            hptt_options_t v;
                            memset(&v, 0, sizeof(v));
                            v.run_a = aBytes[ia] / elem;
                            v.run_b = bBytes[ib] ? bBytes[ib] / elem : 0;
                            if (ia == 0 && ib != 0) v.run_a = 512 / elem;
                            if (ib == 0 && ia != 0) v.run_b = 128 / elem;
                            v.tile_order = ord ? 1 : 0;
                            v.exact_runs = ex;
                            v.store_hint = hintsStore[h];
                            v.load_hint = hintsLoad[h];
                            const int changed = (ia != 0) + (ib != 0) + ord + ex + (h != 0);
                            if (changed) var.push_back({changed, v});
                        }
        for (int c = 1; c <= 5; ++c)
            for (auto& pv : var)
                if (pv.first == c) cand.push_back(pv.second);
    } else if (base.info.kernel == HPTT_KERNEL_STREAM || base.info.kernel == HPTT_KERNEL_AXPBY) {
        for (int h = 1; h < 5; ++h) {
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.store_hint = hintsStore[h];
            v.load_hint = hintsLoad[h];
            cand.push_back(v);
        }
    }
    // drop options that build an already listed plan (or no plan)
    std::vector<hptt_plan_s> built;
    int n = 0;
    for (const hptt_options_t& v : cand) {
        hptt_plan_s p;
        if (build_plan(perm, N, sizeA, outerA, outerB, alpha, beta, dtype, &v, &p) != HPTT_SUCCESS)
            continue;
        bool dup = false;
        for (const hptt_plan_s& q : built)
            if (same_plan(p, q)) {
                dup = true;
                break;
            }
        if (dup) continue;
        built.push_back(p);
        if (n < maxOut && out) out[n] = v;
        ++n;
        if (n >= kMaxCandidates) break;
    }
    return n;
}

hptt_status_t autotune(hptt_plan_t* planOut, const int32_t* perm, int32_t N, const int64_t* sizeA,
                       const int64_t* outerA, const int64_t* outerB, double alpha, double beta,
                       hptt_dtype_t dtype, const void* A, void* B, hipStream_t stream,
                       double timeoutSeconds, hptt_autotune_report_t* report) {
    using clock = std::chrono::steady_clock;
    if (!planOut) return HPTT_ERROR_INVALID_ARGUMENT;
    *planOut = nullptr;
    if (report) memset(report, 0, sizeof(*report));
    {   // nothing to tune when there is nothing to move
        hptt_plan_s base;
        const hptt_status_t st =
            build_plan(perm, N, sizeA, outerA, outerB, alpha, beta, dtype, nullptr, &base);
        if (st != HPTT_SUCCESS) return st;
        if (base.info.kernel == HPTT_KERNEL_NONE)
            return hptt_create_plan_outer(planOut, perm, N, sizeA, outerA, outerB, alpha, beta,
                                          dtype, nullptr);
    }
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return HPTT_ERROR_HIP;
    const int mode = mode_of(dtype, alpha, beta);
    const std::string key = cache_key(perm, N, sizeA, outerA, outerB, dtype, mode, device);
    hptt_options_t best;
    memset(&best, 0, sizeof(best));
    bool cached = false;
    {
        std::lock_guard<std::mutex> lock(g_mutex);
        auto it = g_wisdom.find(key);
        if (it != g_wisdom.end()) {
            best = it->second;
            cached = true;
        }
    }
    if (!cached && timeoutSeconds > 0) {
        std::vector<hptt_options_t> cand(kMaxCandidates);
        const int nc = autotune_candidates(perm, N, sizeA, outerA, outerB, alpha, beta, dtype,
                                           cand.data(), kMaxCandidates);
        if (nc < 0) return hptt_status_t(-nc);
        if (nc > 0 && (!A || !B)) return HPTT_ERROR_INVALID_ARGUMENT;
        hipEvent_t e0, e1;
        if (hipEventCreate(&e0) != hipSuccess) return HPTT_ERROR_HIP;
        if (hipEventCreate(&e1) != hipSuccess) {
            hipEventDestroy(e0);
            return HPTT_ERROR_HIP;
        }
        const auto t0 = clock::now();
        float bestMs = 0.f;
        hptt_status_t err = HPTT_SUCCESS;
        int timed = 0;
        for (int c = 0; c < nc; ++c) {
            // non-destructive timing plan: alpha = 0, beta = 1
            hptt_plan_s tp;
            if (build_plan(perm, N, sizeA, outerA, outerB, 0.0, 1.0, dtype, &cand[c], &tp) !=
                HPTT_SUCCESS)
                continue;
            float ms = 0.f;
            err = hptt_exec(&tp, A, B, stream);  // warm-up
            for (int r = 0; r < 3 && err == HPTT_SUCCESS; ++r) {
                if (hipEventRecord(e0, stream) != hipSuccess) err = HPTT_ERROR_HIP;
                if (err == HPTT_SUCCESS) err = hptt_exec(&tp, A, B, stream);
                if (err == HPTT_SUCCESS && hipEventRecord(e1, stream) != hipSuccess)
                    err = HPTT_ERROR_HIP;
                if (err == HPTT_SUCCESS && hipEventSynchronize(e1) != hipSuccess)
                    err = HPTT_ERROR_HIP;
                float one = 0.f;
                if (err == HPTT_SUCCESS && hipEventElapsedTime(&one, e0, e1) != hipSuccess)
                    err = HPTT_ERROR_HIP;
                if (r == 0 || one < ms) ms = one;  // best of three
            }
            if (err != HPTT_SUCCESS) break;
            ++timed;
            if (c == 0 && report) report->default_ms = ms;
            if (timed == 1 || ms < bestMs) {
                bestMs = ms;
                best = cand[c];
            }
            const double elapsed = std::chrono::duration<double>(clock::now() - t0).count();
            if (elapsed >= timeoutSeconds) break;
        }
        hipEventDestroy(e0);
        hipEventDestroy(e1);
        if (err != HPTT_SUCCESS) return err;
        if (report) {
            report->candidates = nc;
            report->timed = timed;
            report->best_ms = bestMs;
        }
        std::lock_guard<std::mutex> lock(g_mutex);
        g_wisdom[key] = best;
    }
    if (report) {
        report->from_cache = cached ? 1 : 0;
        report->options = best;
    }
    return hptt_create_plan_outer(planOut, perm, N, sizeA, outerA, outerB, alpha, beta, dtype,
                                  &best);
}

void forget_wisdom() {
    std::lock_guard<std::mutex> lock(g_mutex);
    g_wisdom.clear();
}

}  // namespace hptt

extern "C" {

int32_t hptt_autotune_candidates(const int32_t* perm, int32_t N, const int64_t* sizeA,
                                 const int64_t* outerSizeA, const int64_t* outerSizeB,
                                 double alpha, double beta, hptt_dtype_t dtype,
                                 hptt_options_t* options, int32_t max_options) {
    return hptt::autotune_candidates(perm, N, sizeA, outerSizeA, outerSizeB, alpha, beta, dtype,
                                     options, max_options);
}

hptt_status_t hptt_create_plan_autotune(hptt_plan_t* plan, const int32_t* perm, int32_t N,
                                        const int64_t* sizeA, const int64_t* outerSizeA,
                                        const int64_t* outerSizeB, double alpha, double beta,
                                        hptt_dtype_t dtype, const void* A, void* B,
                                        hipStream_t stream, double timeout_seconds,
                                        hptt_autotune_report_t* report) {
    return hptt::autotune(plan, perm, N, sizeA, outerSizeA, outerSizeB, alpha, beta, dtype, A, B,
                          stream, timeout_seconds, report);
}

hptt_status_t hptt_forget_wisdom(void) {
    hptt::forget_wisdom();
    return HPTT_SUCCESS;
}

}  // extern "C"
