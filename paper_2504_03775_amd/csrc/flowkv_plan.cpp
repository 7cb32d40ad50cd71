// Bidirectional segment alignment (FlowKV, arXiv 2504.03775, section 3.3 and
// the Figure 3 caption).  The sender's and the receiver's block lists of a
// request are walked together; a run continues while both step by +1, and
// each maximal run becomes one flowkv_segment.  One pass to validate, one to
// count (so ECAP can report the exact need), one to write: O(n) per request.
#include <cstddef>
#include <cstdint>
#include <vector>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

namespace {

// One bit per pool block; set bits are cleared again by the caller so the
// bitmap can be reused without an O(pool) wipe.
struct Bitmap {
  std::vector<uint64_t> w;
  void size_for(int32_t n) {
    size_t words = (size_t(n) + 63) / 64;
    if (w.size() < words) w.resize(words, 0);
  }
  bool test_set(int32_t i) {
    uint64_t m = 1ull << (i & 63);
    bool was = w[size_t(i) >> 6] & m;
    w[size_t(i) >> 6] |= m;
    return was;
  }
  void clear(int32_t i) { w[size_t(i) >> 6] &= ~(1ull << (i & 63)); }
};

thread_local Bitmap t_src_seen, t_dst_seen;

int check_range(const int32_t* ids, int64_t lo, int64_t hi, int32_t pool, const char* side) {
  for (int64_t i = lo; i < hi; ++i)
    if (ids[i] < 0 || ids[i] >= pool)
      return fail(FLOWKV_ERANGE, "%s block %d at position %lld outside [0, %d)", side, ids[i],
                  (long long)i, pool);
  return FLOWKV_OK;
}

// Mark ids[lo, hi) in `seen`; EDUP on a repeat.  Bits set before a failure
// are cleared before returning.
int mark_unique(Bitmap& seen, const int32_t* ids, int64_t lo, int64_t hi, const char* side) {
  for (int64_t i = lo; i < hi; ++i) {
    if (seen.test_set(ids[i])) {
      for (int64_t j = lo; j < i; ++j) seen.clear(ids[j]);
      return fail(FLOWKV_EDUP, "%s block %d repeated (position %lld)", side, ids[i],
                  (long long)i);
    }
  }
  return FLOWKV_OK;
}

void unmark(Bitmap& seen, const int32_t* ids, int64_t lo, int64_t hi) {
  for (int64_t i = lo; i < hi; ++i) seen.clear(ids[i]);
}

inline bool breaks(const int32_t* S, const int32_t* D, int64_t i) {
  return S[i] != S[i - 1] + 1 || D[i] != D[i - 1] + 1;
}

int plan_impl(int32_t n_req, const int64_t* offsets, const int32_t* S, const int32_t* D,
              int32_t src_pool, int32_t dst_pool, flowkv_segment* out, int64_t cap,
              int64_t* n_out) {
  if (!n_out) return fail(FLOWKV_EINVAL, "NULL n_out");
  if (n_req < 0) return fail(FLOWKV_EINVAL, "negative request count %d", n_req);
  if (src_pool < 0 || dst_pool < 0) return fail(FLOWKV_EINVAL, "negative pool size");
  if (cap < 0) return fail(FLOWKV_EINVAL, "negative capacity");
  if (n_req > 0 && !offsets) return fail(FLOWKV_EINVAL, "NULL offsets");
  if (n_req > 0 && offsets[0] != 0) return fail(FLOWKV_EINVAL, "offsets[0] must be 0");
  for (int32_t r = 0; r < n_req; ++r)
    if (offsets[r + 1] < offsets[r]) return fail(FLOWKV_EINVAL, "offsets decrease at %d", r);
  const int64_t total = n_req > 0 ? offsets[n_req] : 0;
  if (total > INT32_MAX) return fail(FLOWKV_EINVAL, "more than 2^31-1 blocks in one plan");
  if (total > 0 && (!S || !D)) return fail(FLOWKV_EINVAL, "NULL block list");

  int rc = check_range(S, 0, total, src_pool, "sender");
  if (!rc) rc = check_range(D, 0, total, dst_pool, "receiver");
  if (rc) return rc;

  // receiver IDs: distinct across the whole batch; sender IDs: within a request
  t_dst_seen.size_for(dst_pool);
  t_src_seen.size_for(src_pool);
  rc = mark_unique(t_dst_seen, D, 0, total, "receiver");
  if (rc) return rc;
  for (int32_t r = 0; r < n_req && !rc; ++r) {
    rc = mark_unique(t_src_seen, S, offsets[r], offsets[r + 1], "sender");
    if (!rc) unmark(t_src_seen, S, offsets[r], offsets[r + 1]);
  }
  unmark(t_dst_seen, D, 0, total);
  if (rc) return rc;

  int64_t need = 0;
  for (int32_t r = 0; r < n_req; ++r)
    for (int64_t i = offsets[r]; i < offsets[r + 1]; ++i)
      need += (i == offsets[r] || breaks(S, D, i)) ? 1 : 0;
  if (need > cap) {
    *n_out = need;
    return fail(FLOWKV_ECAP, "%lld segments need room, capacity %lld", (long long)need,
                (long long)cap);
  }
  if (need > 0 && !out) return fail(FLOWKV_EINVAL, "NULL output segments");

  int64_t k = 0;
  for (int32_t r = 0; r < n_req; ++r) {
    for (int64_t i = offsets[r]; i < offsets[r + 1]; ++i) {
      if (i == offsets[r] || breaks(S, D, i)) {
        out[k].src_block = S[i];
        out[k].dst_block = D[i];
        out[k].n_blocks = 0;
        out[k].first = int32_t(i);
        ++k;
      }
      ++out[k - 1].n_blocks;
    }
  }
  *n_out = k;
  return ok();
}

}  // namespace

extern "C" int flowkv_plan(const int32_t* src_ids, const int32_t* dst_ids, int32_t n_blocks,
                           int32_t src_pool_blocks, int32_t dst_pool_blocks,
                           flowkv_segment* out, int64_t cap, int64_t* n_out) {
  if (n_blocks < 0) return fail(FLOWKV_EINVAL, "negative block count %d", n_blocks);
  const int64_t offsets[2] = {0, n_blocks};
  return flowkv::guarded([&] {
    return plan_impl(1, offsets, src_ids, dst_ids, src_pool_blocks, dst_pool_blocks, out, cap,
                     n_out);
  });
}

extern "C" int flowkv_plan_batch(int32_t n_req, const int64_t* offsets, const int32_t* src_ids,
                                 const int32_t* dst_ids, int32_t src_pool_blocks,
                                 int32_t dst_pool_blocks, flowkv_segment* out, int64_t cap,
                                 int64_t* n_out) {
  return flowkv::guarded([&] {
    return plan_impl(n_req, offsets, src_ids, dst_ids, src_pool_blocks, dst_pool_blocks, out,
                     cap, n_out);
  });
}
