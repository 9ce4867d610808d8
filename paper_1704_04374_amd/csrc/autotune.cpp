// The autotune path of plan creation (Section 3.1): generate candidate plans,
// rank them with the heuristic plan first, then time them on the caller's own
// tensors, from good to bad, until a timeout, and keep the fastest (FFTW
// style).  Timing never changes the caller's data: the plans write a scratch
// tensor of B's footprint, so that they are timed in the update mode they
// will run in; without memory for it, timing runs on B itself with alpha = 0
// and beta = 1, so B is rewritten with its own value and A is read and
// multiplied by zero (Section 3.1; A must not hold inf or NaN, footnote 5).
// A 512 MiB read between timed launches evicts the tensors from the
// last-level cache, as the paper's measurements clear the caches (Section 4).
// The few fastest candidates are then timed again, alternating with the
// quick path's plan, cold and in back-to-back bursts; one replaces the quick
// plan only if it wins in both.  Winners are cached per problem for the life
// of the process.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <chrono>
#include <map>
#include <mutex>
#include <string.h>
#include <string>
#include <vector>

#include "hptt_yardstick.h"
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
    if (a.info.kernel != b.info.kernel || a.info.hints != b.info.hints ||
        a.info.vec_a != b.info.vec_a || a.info.vec_b != b.info.vec_b)
        return false;
    if (a.info.kernel == HPTT_KERNEL_TILE)
        return memcmp(&a.tile, &b.tile, sizeof(a.tile)) == 0;
    if (a.info.kernel == HPTT_KERNEL_STREAM)  // row or flat walk, XCD groups
        return memcmp(&a.stream, &b.stream, sizeof(a.stream)) == 0;
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
        // the smallest tile worth a workgroup round: default, twice, none
        const int32_t minTile[] = {0, 32768 / elem, 1};
        std::vector<std::pair<int, hptt_options_t>> var;
        for (int ia = 0; ia < 4; ++ia)
            for (int ib = 0; ib < 3; ++ib)
                for (int ord = 0; ord < 2; ++ord)
                    for (int ex = 0; ex < 2; ++ex)
                        for (int mt = 0; mt < 3; ++mt)
                            for (int h = 0; h < 5; ++h) {
                                hptt_options_t v;
                                memset(&v, 0, sizeof(v));
                                v.run_a = aBytes[ia] / elem;
                                v.run_b = bBytes[ib] ? bBytes[ib] / elem : 0;
                                if (ia == 0 && ib != 0) v.run_a = 512 / elem;
                                if (ib == 0 && ia != 0) v.run_b = 128 / elem;
                                v.tile_order = ord ? 1 : 0;
                                v.exact_runs = ex;
                                v.min_tile = minTile[mt];
                                v.store_hint = hintsStore[h];
                                v.load_hint = hintsLoad[h];
                                const int changed =
                                    (ia != 0) + (ib != 0) + ord + ex + (mt != 0) + (h != 0);
                                if (changed) var.push_back({changed, v});
                            }
        // tiles with and without shared runs, whichever the quick path took
        for (int32_t sr = 1; sr <= 2; ++sr) {
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.shared_runs = sr;
            var.push_back({1, v});
        }
        // flat B runs and runs of whole inner extents, whichever it took
        for (int32_t fr = 1; fr <= 2; ++fr) {
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.flat_runs = fr;
            var.push_back({1, v});
        }
        // the outer grid digits in each order the quick path did not take
        for (int32_t go = 1; go <= 3; ++go) {
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.grid_order = go;
            var.push_back({1, v});
        }
        // tiles dealt to the XCDs in groups of 16 (grid-digit order) or one
        // by one, whichever the quick path did not take
        for (int32_t xg = 1; xg <= 16; xg += 15) {
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.xcd_group = xg;
            if (xg > 1) v.tile_order = 1;
            var.push_back({1, v});
        }
        // tiles staged through registers instead of fetched straight into LDS
        {
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.direct_lds = 2;
            var.push_back({1, v});
        }
        for (int c = 1; c <= 6; ++c)
            for (auto& pv : var)
                if (pv.first == c) cand.push_back(pv.second);
    } else if (base.info.kernel == HPTT_KERNEL_STREAM || base.info.kernel == HPTT_KERNEL_AXPBY) {
        if (base.info.kernel == HPTT_KERNEL_STREAM) {  // the kept index as a shared run of tiles
            hptt_options_t v;
            memset(&v, 0, sizeof(v));
            v.shared_runs = 1;
            cand.push_back(v);
            // B walked flat and by rows, whichever the quick path took
            for (int32_t fr = 1; fr <= 2; ++fr) {
                memset(&v, 0, sizeof(v));
                v.flat_runs = fr;
                cand.push_back(v);
            }
            // blocks dealt to the XCDs 16 or 64 at a time
            for (int32_t xg = 16; xg <= 64; xg *= 4) {
                memset(&v, 0, sizeof(v));
                v.xcd_group = xg;
                cand.push_back(v);
            }
        }
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

namespace {

constexpr size_t kFlushBytes = size_t(512) << 20;  // two last-level caches (256 MB each)
constexpr int kReps = 3;
constexpr int kBurst = 4;
constexpr float kMargin = 0.99f;  // leave the quick plan only for a 1 % gain
// Screening times many candidates three times each, so the fastest of them
// is partly the luckiest: the finalists are timed again against the quick
// plan, in alternating order, before one may replace it.
constexpr int kFinalists = 3;
constexpr int kConfirmRounds = 5;

// Device memory the tuner borrows for its measurements and returns at the end.
struct Scratch {
    void* flush = nullptr;  // read between timed launches so they start cold
    void* sink = nullptr;   // checksums of the flush reads
    void* out = nullptr;    // a stand-in for B, so timing leaves B alone
    // more (A, B) stand-ins, so back-to-back confirmation launches rotate
    // over enough memory that none finds its tensors in the caches
    std::vector<void*> rotA, rotB;
    ~Scratch() {
        if (flush) (void)hipFree(flush);
        if (sink) (void)hipFree(sink);
        if (out) (void)hipFree(out);
        for (void* p : rotA) (void)hipFree(p);
        for (void* p : rotB) (void)hipFree(p);
    }
};

constexpr size_t kRotateBytes = size_t(2) << 30;  // traffic between two uses of one set
constexpr int kMaxSets = 8;

bool try_alloc(void** p, size_t bytes) {
    if (hipMalloc(p, bytes) == hipSuccess) return true;
    *p = nullptr;
    (void)hipGetLastError();  // an allocation failure is not an error of the caller's
    return false;
}

float median3(float a, float b, float c) {
    return a > b ? (b > c ? b : (a > c ? c : a)) : (a > c ? a : (b > c ? c : b));
}

}  // namespace

hptt_status_t autotune(hptt_plan_t* planOut, const int32_t* perm, int32_t N, const int64_t* sizeA,
                       const int64_t* outerA, const int64_t* outerB, double alpha, double beta,
                       hptt_dtype_t dtype, const void* A, void* B, hipStream_t stream,
                       double timeoutSeconds, hptt_autotune_report_t* report) {
    using clock = std::chrono::steady_clock;
    if (!planOut) return HPTT_ERROR_INVALID_ARGUMENT;
    *planOut = nullptr;
    if (report) memset(report, 0, sizeof(*report));
    hptt_plan_s base;
    {
        const hptt_status_t st =
            build_plan(perm, N, sizeA, outerA, outerB, alpha, beta, dtype, nullptr, &base);
        if (st != HPTT_SUCCESS) return st;
        if (base.info.kernel == HPTT_KERNEL_NONE)  // nothing to move, nothing to tune
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
        if (!A || !B) return HPTT_ERROR_INVALID_ARGUMENT;
        // Time in the caller's own update mode, writing a scratch tensor so
        // that B is not touched (with beta != 0 the scratch tensor is zeroed
        // first and then updated in place by every timed launch: the values
        // do not change the timing).  Without memory for it, fall back to the
        // paper's alpha = 0, beta = 1 on B itself, which keeps B's values
        // (but turns a -0.0 into +0.0 and any inf or NaN of A into NaN).
        Scratch scratch;
        const size_t elem = dtype == HPTT_FLOAT32 ? 4 : 8;
        const size_t outBytes = (size_t(base.info.footprint_b) * elem + 15) / 16 * 16;
        bool ownMode = try_alloc(&scratch.out, outBytes);
        if (ownMode && mode == kAxpby &&
            hptt_yardstick_fill(scratch.out, outBytes, 0, stream) != HPTT_SUCCESS)
            return HPTT_ERROR_HIP;
        const double tAlpha = ownMode ? alpha : 0.0, tBeta = ownMode ? beta : 1.0;
        void* const target = ownMode ? scratch.out : B;
        const bool flush = try_alloc(&scratch.flush, kFlushBytes) &&
                           try_alloc(&scratch.sink, 4096 * sizeof(uint32_t));
        // Buffer sets the confirmation bursts rotate over: set 0 is the
        // caller's A with the timing target, the others scratch copies of
        // their footprints (zeroed: the values do not change the timing).
        // Fewer sets when memory is short (then bursts partly reuse the
        // caches, as a caller reusing its tensors would).
        const size_t inBytes = (size_t(base.info.footprint_a) * elem + 15) / 16 * 16;
        std::vector<const void*> setA{A};
        std::vector<void*> setB{target};
        {
            // (one set when a launch alone moves kRotateBytes: it evicts itself)
            const size_t perSet = inBytes + outBytes;
            const size_t want = std::min<size_t>(kMaxSets, (kRotateBytes + perSet - 1) / perSet);
            // each copy sits as far from a 256-byte boundary as the original,
            // so that every set launches the same kernel variant and hints
            const size_t offA = reinterpret_cast<uintptr_t>(A) % 256;
            const size_t offB = reinterpret_cast<uintptr_t>(target) % 256;
            while (setA.size() < want) {
                void *a = nullptr, *b = nullptr;
                if (!try_alloc(&a, inBytes + 256)) break;
                scratch.rotA.push_back(a);
                if (!try_alloc(&b, outBytes + 256)) break;
                scratch.rotB.push_back(b);
                if (hptt_yardstick_fill(a, inBytes + 256, 0, stream) != HPTT_SUCCESS ||
                    hptt_yardstick_fill(b, outBytes + 256, 0, stream) != HPTT_SUCCESS)
                    return HPTT_ERROR_HIP;
                setA.push_back(static_cast<const char*>(a) + offA);
                setB.push_back(static_cast<char*>(b) + offB);
            }
        }
        hipEvent_t e0, e1;
        if (hipEventCreate(&e0) != hipSuccess) return HPTT_ERROR_HIP;
        if (hipEventCreate(&e1) != hipSuccess) {
            (void)hipEventDestroy(e0);
            return HPTT_ERROR_HIP;
        }
        // One measurement: [flush] e0 launch(es) [flush] e1.  The second flush
        // is inside the timed span: it writes back the lines the launch left
        // dirty in the caches, a cost a lone launch with write-back stores
        // would hide and back-to-back launches pay.  Its clean time is
        // measured alone and subtracted.  Without flush memory: kBurst
        // launches back to back.
        auto span = [&](hptt_plan_s* tp, float* ms) -> hptt_status_t {
            hptt_status_t e = HPTT_SUCCESS;
            if (flush) e = hptt_yardstick_read(scratch.flush, kFlushBytes, scratch.sink, stream);
            if (e == HPTT_SUCCESS && hipEventRecord(e0, stream) != hipSuccess) e = HPTT_ERROR_HIP;
            for (int b = 0; b < (flush ? 1 : kBurst) && e == HPTT_SUCCESS; ++b)
                if (tp) e = hptt_exec(tp, A, target, stream);
            if (e == HPTT_SUCCESS && flush)
                e = hptt_yardstick_read(scratch.flush, kFlushBytes, scratch.sink, stream);
            if (e == HPTT_SUCCESS && hipEventRecord(e1, stream) != hipSuccess) e = HPTT_ERROR_HIP;
            if (e == HPTT_SUCCESS && hipEventSynchronize(e1) != hipSuccess) e = HPTT_ERROR_HIP;
            if (e == HPTT_SUCCESS && hipEventElapsedTime(ms, e0, e1) != hipSuccess)
                e = HPTT_ERROR_HIP;
            return e;
        };
        auto measure = [&](hptt_plan_s* tp, float* out) -> hptt_status_t {
            float ms[kReps] = {};
            hptt_status_t e = HPTT_SUCCESS;
            for (int r = 0; r < kReps && e == HPTT_SUCCESS; ++r) e = span(tp, &ms[r]);
            *out = median3(ms[0], ms[1], ms[2]);
            return e;
        };
        // Back-to-back use: [flush] e0 n launches over the rotating sets e1,
        // per launch (n = two rounds of the sets, at least kBurst).
        const int burstLaunches = std::max<int>(kBurst, 2 * int(setA.size()));
        auto burst = [&](hptt_plan_s* tp, float* ms) -> hptt_status_t {
            hptt_status_t e = HPTT_SUCCESS;
            if (flush) e = hptt_yardstick_read(scratch.flush, kFlushBytes, scratch.sink, stream);
            if (e == HPTT_SUCCESS && hipEventRecord(e0, stream) != hipSuccess) e = HPTT_ERROR_HIP;
            for (int b = 0; b < burstLaunches && e == HPTT_SUCCESS; ++b)
                e = hptt_exec(tp, setA[b % setA.size()], setB[b % setB.size()], stream);
            if (e == HPTT_SUCCESS && hipEventRecord(e1, stream) != hipSuccess) e = HPTT_ERROR_HIP;
            if (e == HPTT_SUCCESS && hipEventSynchronize(e1) != hipSuccess) e = HPTT_ERROR_HIP;
            if (e == HPTT_SUCCESS && hipEventElapsedTime(ms, e0, e1) != hipSuccess)
                e = HPTT_ERROR_HIP;
            *ms /= burstLaunches;
            return e;
        };
        const auto t0 = clock::now();
        float bestMs = 0.f, quickMs = 0.f, flushMs = 0.f;
        hptt_status_t err = flush ? measure(nullptr, &flushMs) : HPTT_SUCCESS;
        int timed = 0;
        std::vector<std::pair<float, int>> ahead;  // screened faster than the quick plan
        for (int c = 0; c < nc && err == HPTT_SUCCESS; ++c) {
            hptt_plan_s tp;
            if (build_plan(perm, N, sizeA, outerA, outerB, tAlpha, tBeta, dtype, &cand[c], &tp) !=
                HPTT_SUCCESS)
                continue;
            err = hptt_exec(&tp, A, target, stream);  // warm-up
            float m = 0.f;
            if (err == HPTT_SUCCESS) err = measure(&tp, &m);
            if (err != HPTT_SUCCESS) break;
            m = flush ? m - flushMs : m / kBurst;
            ++timed;
            if (c == 0) quickMs = bestMs = m;
            else if (m < kMargin * quickMs) ahead.push_back({m, c});
            const double elapsed = std::chrono::duration<double>(clock::now() - t0).count();
            if (elapsed >= timeoutSeconds) break;
        }
        // Confirmation: each finalist against the quick plan, kConfirmRounds
        // rounds in alternating order, summed cold (as screened) and in
        // back-to-back bursts; it must beat the quick plan by the margin in
        // both.  The confirmed finalist with the fastest bursts is chosen.
        std::sort(ahead.begin(), ahead.end());
        if (ahead.size() > size_t(kFinalists)) ahead.resize(kFinalists);
        int confirmed = 0;
        float bestBurst = 0.f;
        hptt_plan_s qp;
        if (err == HPTT_SUCCESS && !ahead.empty() &&
            build_plan(perm, N, sizeA, outerA, outerB, tAlpha, tBeta, dtype, &cand[0], &qp) !=
                HPTT_SUCCESS)
            ahead.clear();
        for (const auto& fin : ahead) {
            hptt_plan_s fp;
            if (build_plan(perm, N, sizeA, outerA, outerB, tAlpha, tBeta, dtype, &cand[fin.second],
                           &fp) != HPTT_SUCCESS)
                continue;
            float qCold = 0.f, fCold = 0.f, qBurst = 0.f, fBurst = 0.f;
            for (int r = 0; r < kConfirmRounds && err == HPTT_SUCCESS; ++r) {
                hptt_plan_s* order[2] = {&qp, &fp};
                if (r & 1) std::swap(order[0], order[1]);
                for (hptt_plan_s* tp : order) {
                    float c = 0.f, b = 0.f;
                    if (flush && err == HPTT_SUCCESS) err = span(tp, &c);
                    if (err == HPTT_SUCCESS) err = burst(tp, &b);
                    if (err != HPTT_SUCCESS) break;
                    (tp == &qp ? qCold : fCold) += flush ? c - flushMs : 0.f;
                    (tp == &qp ? qBurst : fBurst) += b;
                }
            }
            if (err != HPTT_SUCCESS) break;
            if (fCold <= kMargin * qCold && fBurst < kMargin * qBurst &&
                (confirmed == 0 || fBurst < bestBurst)) {
                bestBurst = fBurst;
                best = cand[fin.second];
                bestMs = fin.first;
            }
            confirmed += fCold <= kMargin * qCold && fBurst < kMargin * qBurst;
        }
        (void)hipEventDestroy(e0);
        (void)hipEventDestroy(e1);
        if (err != HPTT_SUCCESS) return err;
        if (report) {
            report->candidates = nc;
            report->timed = timed;
            report->default_ms = quickMs;
            report->best_ms = bestMs;
            report->flushed = flush ? 1 : 0;
            report->own_mode = ownMode ? 1 : 0;
            report->finalists = int32_t(ahead.size());
            report->confirmed = confirmed;
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
