// Host half of the C ABI: plan creation, inspection and destruction.  None of
// these functions makes a HIP call; hptt_exec lives in kernels.hip.  With the
// environment variable HPTT_LOG set (and not "0"), every plan created prints
// its description to stderr.
#include <new>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "plan.h"

extern "C" {

hptt_status_t hptt_create_plan_outer(hptt_plan_t* plan, const int32_t* perm, int32_t N,
                                     const int64_t* sizeA, const int64_t* outerSizeA,
                                     const int64_t* outerSizeB, double alpha, double beta,
                                     hptt_dtype_t dtype, const hptt_options_t* options) {
    if (!plan) return HPTT_ERROR_INVALID_ARGUMENT;
    *plan = nullptr;
    hptt_plan_s* p = new (std::nothrow) hptt_plan_s;
    if (!p) return HPTT_ERROR_OUT_OF_MEMORY;
    hptt_status_t st = hptt::build_plan(perm, N, sizeA, outerSizeA, outerSizeB, alpha, beta,
                                        dtype, options, p);
    if (st != HPTT_SUCCESS) {
        delete p;
        return st;
    }
    *plan = p;
    // HPTT_LOG=1: one line per new plan on stderr (fused shape, kernel, tile, grid)
    const char* log = getenv("HPTT_LOG");
    if (log && log[0] && strcmp(log, "0") != 0) {
        char desc[512];
        hptt::describe_plan(p, desc, sizeof(desc));
        fprintf(stderr, "[hptt] plan: %s\n", desc);
    }
    return HPTT_SUCCESS;
}

hptt_status_t hptt_create_plan_ex(hptt_plan_t* plan, const int32_t* perm, int32_t N,
                                  const int64_t* sizeA, double alpha, double beta,
                                  hptt_dtype_t dtype, const hptt_options_t* options) {
    return hptt_create_plan_outer(plan, perm, N, sizeA, nullptr, nullptr, alpha, beta, dtype,
                                  options);
}

hptt_status_t hptt_create_plan(hptt_plan_t* plan, const int32_t* perm, int32_t N,
                               const int64_t* sizeA, double alpha, double beta,
                               hptt_dtype_t dtype) {
    return hptt_create_plan_outer(plan, perm, N, sizeA, nullptr, nullptr, alpha, beta, dtype,
                                  nullptr);
}

hptt_status_t hptt_destroy_plan(hptt_plan_t plan) {
    delete plan;
    return HPTT_SUCCESS;
}

hptt_status_t hptt_plan_info(hptt_plan_t plan, hptt_plan_info_t* info) {
    if (!plan || !info) return HPTT_ERROR_INVALID_ARGUMENT;
    *info = plan->info;
    return HPTT_SUCCESS;
}

hptt_status_t hptt_describe_plan(hptt_plan_t plan, char* buf, size_t len) {
    if (!plan || !buf || len == 0) return HPTT_ERROR_INVALID_ARGUMENT;
    hptt::describe_plan(plan, buf, len);
    return HPTT_SUCCESS;
}

const char* hptt_status_string(hptt_status_t status) {
    switch (status) {
        case HPTT_SUCCESS: return "success";
        case HPTT_ERROR_INVALID_ARGUMENT: return "invalid argument";
        case HPTT_ERROR_UNSUPPORTED: return "unsupported option for this problem";
        case HPTT_ERROR_OVERLAP: return "A and B overlap";
        case HPTT_ERROR_OUT_OF_MEMORY: return "out of host memory";
        case HPTT_ERROR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

}  // extern "C"
