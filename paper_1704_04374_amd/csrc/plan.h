// The plan object behind hptt_plan_t and the host-only plan builder.
#pragma once

#include "hptt.h"
#include "hptt_args.h"

struct hptt_plan_s {
    hptt_plan_info_t info;
    hptt_dtype_t dtype;
    double alpha;  // rounded to dtype
    double beta;   // rounded to dtype
    hptt::TileArgs tile;
    hptt::StreamArgs stream;
    hptt::GenericArgs generic;
};

namespace hptt {

// Fill *plan for Eq. (1); no HIP call.  options may be NULL.
// outerSizeA / outerSizeB may be NULL (compact tensors).
hptt_status_t build_plan(const int32_t* perm, int32_t N, const int64_t* sizeA,
                         const int64_t* outerSizeA, const int64_t* outerSizeB, double alpha,
                         double beta, hptt_dtype_t dtype, const hptt_options_t* options,
                         hptt_plan_s* plan);

// LDS bytes of kernel T: the two offset tables and the padded tile.
int64_t tile_lds_bytes_host(const TileArgs& t, int elem);

// One-line summary of a plan.
void describe_plan(const hptt_plan_s* plan, char* buf, size_t len);

}  // namespace hptt
