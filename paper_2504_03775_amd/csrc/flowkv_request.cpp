// One request moved in one call (FlowKV, arXiv 2504.03775, section 3.1's
// statement of the problem, with section 3.3's alignment and transfer): the
// planner's records go straight into the inline launch, without a round trip
// through the caller.  Host code; it composes the library's own entry points.
#include <cstdint>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;

// Plan one request into a stack buffer of the inline capacity and hand it to
// the inline launch: the planner's records are in the form the compact
// inline arguments need.
extern "C" int flowkv_transfer_request(const flowkv_pool* src, const flowkv_pool* dst,
                                       const int32_t* src_ids, const int32_t* dst_ids,
                                       int32_t n_blocks, const flowkv_launch_config* cfg,
                                       int64_t* n_runs, void* hip_stream) {
  if (!src || !dst || !n_runs) return fail(FLOWKV_EINVAL, "NULL pool or n_runs");
  if (n_blocks < 0) return fail(FLOWKV_EINVAL, "negative block count %d", n_blocks);
  int64_t cap = 0;
  const int rcap = flowkv_inline_capacity(src, dst, &cap);
  if (rcap) return rcap;
  static_assert(FLOWKV_INLINE_RUNS_BLOCK_MAJOR >= FLOWKV_INLINE_RUNS_LAYER_MAJOR &&
                    FLOWKV_INLINE_RUNS_BLOCK_MAJOR >= FLOWKV_INLINE_RUNS,
                "the stack buffer holds the largest inline plan");
  flowkv_segment runs[FLOWKV_INLINE_RUNS_BLOCK_MAJOR];
  int64_t k = 0;
  const int rc = flowkv_plan(src_ids, dst_ids, n_blocks, src->num_blocks, dst->num_blocks, runs,
                             cap, &k);
  if (rc == FLOWKV_ECAP) {
    *n_runs = k;
    return fail(FLOWKV_ECAP, "%lld runs: at most %lld travel in the kernel arguments between "
                "these pools", (long long)k, (long long)cap);
  }
  if (rc) return rc;
  // *n_runs is an output: written on success only (and on ECAP above)
  const int rl = flowkv_transfer_inline(src, dst, runs, k, n_blocks, cfg, hip_stream);
  if (rl == FLOWKV_OK) *n_runs = k;
  return rl;
}
