// Host-code check built with AddressSanitizer and UndefinedBehaviorSanitizer
// (CPU only, test infrastructure): the plan builder (plan.cpp, api.cpp), the
// autotuner's candidate enumeration (autotune.cpp), the kernels' phase
// functions run by the host emulator (emulate.cpp) and the CPU oracle
// (oracle.c), driven through the C ABI over
//   - random problems of rank 1-6 with small odd extents, both dtypes, several
//     alpha/beta pairs and forced knob sets, each compared bit for bit with the
//     oracle (Eq. 1);
//   - random sub-tensors with outer sizes (Fig. 3) against the oracle;
//   - rank 7-16 problems with extents 2-3;
//   - base pointers off the 16-byte grid;
//   - every autotune candidate of a few problems;
//   - a strided dry run of each named full-size workload (offsets only).
// Exit status 0 when every result matched and no check failed; a sanitizer
// report aborts the program (-fno-sanitize-recover).
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <random>
#include <vector>

#include "hptt.h"
#include "hptt_yardstick.h"

extern "C" {
int64_t hptt_emulate_exec(hptt_plan_t plan, const void* A, void* B, int32_t va, int32_t vb,
                          uint8_t* counts, int64_t block_stride, char* msg, size_t msglen,
                          int32_t misA, int32_t misB, int32_t variant);
int oracle_transpose_outer_f32(int N, const int64_t* sizeA, const int32_t* perm,
                               const int64_t* outerA, const int64_t* outerB, float alpha,
                               float beta, const float* A, float* B);
int oracle_transpose_outer_f64(int N, const int64_t* sizeA, const int32_t* perm,
                               const int64_t* outerA, const int64_t* outerB, double alpha,
                               double beta, const double* A, double* B);

// The device half of the library (kernels.hip, yardstick.hip) is not built
// here; the autotuner's timing path refers to it but is never called.
hptt_status_t hptt_exec(hptt_plan_t, const void*, void*, hipStream_t) { return HPTT_ERROR_HIP; }
hptt_status_t hptt_yardstick_read(const void*, size_t, void*, hipStream_t) { return HPTT_ERROR_HIP; }
hptt_status_t hptt_yardstick_fill(void*, size_t, uint32_t, hipStream_t) { return HPTT_ERROR_HIP; }
}

namespace {

std::mt19937_64 rng(1704);
int failures = 0;
int64_t checked = 0;

int64_t pick(const std::vector<int64_t>& v) { return v[rng() % v.size()]; }

int64_t prod(const std::vector<int64_t>& v) {
    int64_t p = 1;
    for (int64_t x : v) p *= x;
    return p;
}

int64_t footprint(const std::vector<int64_t>& size, const std::vector<int64_t>& outer) {
    int64_t span = 1, stride = 1;
    for (size_t d = 0; d < size.size(); ++d) {
        if (size[d] == 0) return 0;
        span += (size[d] - 1) * stride;
        stride *= outer[d];
    }
    return span;
}

template <typename T>
void fill(std::vector<T>& v, size_t from = 0) {
    for (size_t i = from; i < v.size(); ++i) v[i] = T(int64_t(rng() % 2048) - 1024) / T(1024);
}

template <typename T>
bool run_one(const std::vector<int64_t>& size, const std::vector<int32_t>& perm,
             const std::vector<int64_t>* outerA, const std::vector<int64_t>* outerB, double alpha,
             double beta, const hptt_options_t* opt, int mis) {
    const int N = int(size.size());
    const hptt_dtype_t dt = sizeof(T) == 4 ? HPTT_FLOAT32 : HPTT_FLOAT64;
    std::vector<int64_t> sizeB(N);
    for (int k = 0; k < N; ++k) sizeB[k] = size[perm[k]];
    const std::vector<int64_t> oa = outerA ? *outerA : size, ob = outerB ? *outerB : sizeB;
    hptt_plan_t p = nullptr;
    hptt_status_t st = hptt_create_plan_outer(&p, perm.data(), N, size.data(),
                                              outerA ? outerA->data() : nullptr,
                                              outerB ? outerB->data() : nullptr, alpha, beta, dt,
                                              opt);
    if (st == HPTT_ERROR_UNSUPPORTED) return true;  // a forced knob that does not apply
    if (st != HPTT_SUCCESS) {
        printf("plan failed: %s\n", hptt_status_string(st));
        ++failures;
        return false;
    }
    char desc[512];
    hptt_describe_plan(p, desc, sizeof(desc));
    hptt_plan_info_t info;
    hptt_plan_info(p, &info);
    // A and B in one allocation, far apart: the emulator attributes an access
    // to the tensor its base pointer is nearer to (a tile's base may lie past
    // its tensor's end), so the two must not be neighbours in memory.  Each
    // starts `mis` elements off the 16-byte vector grid.
    const int64_t fa = footprint(size, oa), fb = footprint(sizeB, ob);
    const int64_t gap = 2 * (fa + fb) + 4096, offB = (fa + gap) / 16 * 16;
    std::vector<T> buf(size_t(offB + fb + 2 * mis + 16)), want;
    fill(buf);
    T* const pa = buf.data() + mis;
    T* const pb = buf.data() + offB + mis;
    want.assign(pb, pb + fb);
    const T a = T(alpha), b = T(beta);
    int err;
    if constexpr (sizeof(T) == 4)
        err = oracle_transpose_outer_f32(N, size.data(), perm.data(), oa.data(), ob.data(), a, b,
                                         pa, want.data());
    else
        err = oracle_transpose_outer_f64(N, size.data(), perm.data(), oa.data(), ob.data(), a, b,
                                         pa, want.data());
    if (err) {
        printf("oracle rejected a problem the plan accepted: %s\n", desc);
        ++failures;
        hptt_destroy_plan(p);
        return false;
    }
    // as hptt_exec: the tile kernel shifts its runs onto the pointers' vector
    // grid, the other kernels narrow their vectors to the pointers' alignment
    int va = 0, vb = 0;
    if (info.kernel != HPTT_KERNEL_TILE && mis) {
        auto narrow = [&](int v) {
            while (v > 1 && (mis * int(sizeof(T))) % (v * int(sizeof(T))) != 0) v /= 2;
            return v;
        };
        va = narrow(info.vec_a);
        vb = narrow(info.vec_b);
    }
    std::vector<uint8_t> counts(size_t(fb), 0);
    char msg[512] = "";
    const int64_t bad = hptt_emulate_exec(p, pa, pb, va, vb, counts.data(), 1, msg, sizeof(msg),
                                          mis, mis, -1);
    bool ok = bad == 0 && memcmp(pb, want.data(), want.size() * sizeof(T)) == 0;
    int64_t written = 0;
    for (uint8_t c : counts) {
        if (c > 1) ok = false;
        written += c;
    }
    if (written != prod(size)) ok = false;
    if (!ok) {
        printf("MISMATCH (%lld violations: %s) %s\n", (long long)bad, msg, desc);
        ++failures;
    }
    ++checked;
    hptt_destroy_plan(p);
    return ok;
}

std::vector<int32_t> random_perm(int n) {
    std::vector<int32_t> p(n);
    for (int i = 0; i < n; ++i) p[i] = i;
    for (int i = n - 1; i > 0; --i) std::swap(p[i], p[rng() % (i + 1)]);
    return p;
}

const double kAB[][2] = {{1.0, 0.0}, {1.5, 0.0}, {-0.375, 1.25}, {2.0, 0.5}, {0.0, 1.0}};

hptt_options_t knob_set(int i) {
    hptt_options_t o;
    memset(&o, 0, sizeof(o));
    switch (i % 12) {
        case 1: o.kernel = HPTT_KERNEL_GENERIC; break;
        case 2: o.run_a = 4, o.run_b = 4; break;
        case 3: o.run_a = 3, o.run_b = 5; break;
        case 4: o.max_blocks = 3; break;
        case 5: o.row_passes = 3; break;
        case 6: o.tile_order = 3, o.grid_order = 2; break;
        case 7: o.grid_order = 3; break;
        case 8: o.depth = 3; break;
        case 9: o.shared_runs = 1; break;
        case 10: o.flat_runs = 1; break;
        case 11: o.max_vec = 1, o.block = 1024; break;
        default: break;
    }
    return o;
}

}  // namespace

int main() {
    const std::vector<int64_t> ext = {1, 2, 3, 5, 7, 17, 33, 64, 65};
    // random compact problems
    for (int it = 0; it < 1500; ++it) {
        std::vector<int64_t> size;
        do {
            size.assign(1 + rng() % 6, 0);
            for (auto& s : size) s = pick(ext);
        } while (prod(size) > 20000);
        const auto perm = random_perm(int(size.size()));
        const double* ab = kAB[it % 5];
        const hptt_options_t o = knob_set(it / 5);
        const int mis = (it % 7 == 3) ? int(1 + rng() % 3) : 0;
        if (it % 2) run_one<float>(size, perm, nullptr, nullptr, ab[0], ab[1], &o, mis);
        else run_one<double>(size, perm, nullptr, nullptr, ab[0], ab[1], &o, mis % 2);
    }
    fprintf(stderr, "[host check] compact problems done\n");
    // random sub-tensors with outer sizes
    for (int it = 0; it < 400; ++it) {
        std::vector<int64_t> size;
        do {
            size.assign(1 + rng() % 5, 0);
            for (auto& s : size) s = pick(ext);
        } while (prod(size) > 20000);
        const int n = int(size.size());
        const auto perm = random_perm(n);
        std::vector<int64_t> oa(n), ob(n);
        for (int d = 0; d < n; ++d) oa[d] = size[d] + pick({0, 0, 1, 3, 8});
        for (int k = 0; k < n; ++k) ob[k] = size[perm[k]] + pick({0, 0, 1, 3, 8});
        const double* ab = kAB[it % 5];
        const hptt_options_t o = knob_set(it);
        if (it % 2) run_one<float>(size, perm, &oa, &ob, ab[0], ab[1], &o, 0);
        else run_one<double>(size, perm, &oa, &ob, ab[0], ab[1], &o, 0);
    }
    fprintf(stderr, "[host check] sub-tensors done\n");
    // high ranks: 7 to 16 indices of extent 2 or 3
    for (int n = 7; n <= 16; ++n) {
        std::vector<int64_t> size(n);
        for (auto& s : size) s = 2 + rng() % 2;
        while (prod(size) > (int64_t(1) << 17)) size[rng() % n] = 2;
        const auto perm = random_perm(n);
        run_one<float>(size, perm, nullptr, nullptr, 1.0, 0.0, nullptr, 0);
        run_one<double>(size, perm, nullptr, nullptr, -0.375, 1.25, nullptr, 0);
    }
    fprintf(stderr, "[host check] high ranks done\n");
    // every autotune candidate of a few problems
    const std::vector<std::vector<int64_t>> tuneSizes = {{97, 65, 33}, {3, 2, 40, 33, 17},
                                                         {24, 13, 9, 10}, {5, 7, 17, 3, 2, 3}};
    for (size_t i = 0; i < tuneSizes.size(); ++i) {
        const auto& size = tuneSizes[i];
        const auto perm = i == 2 ? std::vector<int32_t>{0, 3, 2, 1} : random_perm(int(size.size()));
        std::vector<hptt_options_t> cand(256);
        const int32_t nc = hptt_autotune_candidates(perm.data(), int32_t(size.size()), size.data(),
                                                    nullptr, nullptr, 1.0, 1.0, HPTT_FLOAT32,
                                                    cand.data(), 256);
        if (nc < 1) {
            printf("no autotune candidates\n");
            ++failures;
        }
        for (int32_t c = 0; c < nc && c < 256; ++c)
            run_one<float>(size, perm, nullptr, nullptr, 0.0, 1.0, &cand[c], 0);
    }
    fprintf(stderr, "[host check] autotune candidates done\n");
    // named full-size workloads: every 13th workgroup, offsets only
    struct W {
        std::vector<int64_t> size;
        std::vector<int32_t> perm;
        double a, b;
        hptt_dtype_t dt;
    };
    const std::vector<W> named = {
        {{8192, 8192}, {1, 0}, 1.0, 0.0, HPTT_FLOAT32},
        {{24, 20, 16, 24, 18, 20}, {5, 2, 0, 4, 1, 3}, 1.5, 0.0, HPTT_FLOAT32},
        {{96, 96, 96, 96}, {0, 3, 2, 1}, 2.0, 0.5, HPTT_FLOAT64},
        {{3, 2, 640, 480, 96}, {4, 2, 0, 3, 1}, 1.0, 1.0, HPTT_FLOAT32}};
    for (const W& w : named) {
        hptt_plan_t p = nullptr;
        if (hptt_create_plan(&p, w.perm.data(), int32_t(w.size.size()), w.size.data(), w.a, w.b,
                             w.dt) != HPTT_SUCCESS) {
            ++failures;
            continue;
        }
        char msg[512] = "";
        const int64_t bad = hptt_emulate_exec(p, nullptr, nullptr, 0, 0, nullptr, 13, msg,
                                              sizeof(msg), 0, 0, -1);
        if (bad) {
            printf("dry run: %lld violations: %s\n", (long long)bad, msg);
            ++failures;
        }
        ++checked;
        hptt_destroy_plan(p);
    }
    // argument errors return status codes
    {
        hptt_plan_t p = reinterpret_cast<hptt_plan_t>(1);
        const int32_t perm[2] = {0, 0};
        const int64_t size[2] = {4, 4};
        if (hptt_create_plan(&p, perm, 2, size, 1.0, 0.0, HPTT_FLOAT32) !=
                HPTT_ERROR_INVALID_ARGUMENT || p != nullptr)
            ++failures;
    }
    printf("host check: %lld problems, %d failures\n", (long long)checked, failures);
    return failures == 0 ? 0 : 1;
}
