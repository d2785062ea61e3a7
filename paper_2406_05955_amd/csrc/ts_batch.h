// Batched path entry (ts_batch.hip), used by the ts_ffn_sparse and
// ts_moe_sparse entry points when several tokens share the weights.
#pragma once

#include <hip/hip_runtime.h>

#include "ts_plan.h"
#include "turbosparse.h"

namespace ts {

// One pass for up to kBxMaxTokens tokens (plan p).  x / out point at the
// pass's first token; topk / topw are the MoE routing table of those tokens
// (null for the FFN); stats arrays are indexed from stats_base.  dense: take
// every row (the dense comparator).  xtok (MoE): the router has written
// every token's x as bf16 high / low parts at the
// workspace's x-fragment offset (moe_router's xs layout, hpad / 8 chunks per
// token), and the gate+up kernel gathers its group's tokens from there.
ts_status run_batch(const float *x, const void *wg, const void *wu, const void *wd, size_t expert_stride,
                    const int32_t *topk, const float *topw, const BatchPlan &p, float *out,
                    const ts_ffn_stats *stats, int stats_base, void *ws, hipStream_t st, bool dense,
                    bool xtok = false);

}  // namespace ts
