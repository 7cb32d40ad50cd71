// Bidirectional segment alignment (FlowKV, arXiv 2504.03775, section 3.3 and
// the Figure 3 caption).  The sender's and the receiver's block lists of a
// request are walked together; a run continues while both step by +1, and
// each maximal run becomes one flowkv_segment.  Passes to validate, then one
// to write (preceded by one to count when the output may be too small, so
// ECAP can report the exact need): O(n) per request.
#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <vector>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

namespace {

// One bit per pool block; set bits are cleared again by the caller so the
// bitmap can be reused without an O(pool) wipe.  Block lists are mostly runs
// of consecutive IDs, so bits are tested, set and cleared a run at a time,
// with word masks: per ID, a read-modify-write of the same word would chain
// every ID of a run through one memory location.
struct Bitmap {
  std::vector<uint64_t> w;
  void size_for(int32_t n) {
    size_t words = (size_t(n) + 63) / 64;
    if (w.size() < words) w.resize(words, 0);
  }
  bool test(int32_t i) const { return (w[size_t(i) >> 6] >> (i & 63)) & 1; }
  // f(word index, mask) over the words of bits [a, b), a < b
  template <class F>
  static void words(int32_t a, int32_t b, F f) {
    const size_t wa = size_t(a) >> 6, wb = size_t(b - 1) >> 6;
    const uint64_t head = ~0ull << (a & 63), tail = ~0ull >> (63 - ((b - 1) & 63));
    if (wa == wb) {
      f(wa, head & tail);
      return;
    }
    f(wa, head);
    for (size_t i = wa + 1; i < wb; ++i) f(i, ~0ull);
    f(wb, tail);
  }
  bool any(int32_t a, int32_t b) const {
    uint64_t hit = 0;
    words(a, b, [&](size_t i, uint64_t m) { hit |= w[i] & m; });
    return hit != 0;
  }
  void set(int32_t a, int32_t b) {
    words(a, b, [&](size_t i, uint64_t m) { w[i] |= m; });
  }
  void clear(int32_t a, int32_t b) {
    words(a, b, [&](size_t i, uint64_t m) { w[i] &= ~m; });
  }
};

// A run of IDs [lo, hi) as marked in a bitmap.
struct IdRun {
  int32_t lo, hi;
};

thread_local Bitmap t_src_seen, t_dst_seen;
thread_local std::vector<IdRun> t_src_runs, t_dst_runs;

int check_range(const int32_t* ids, int64_t lo, int64_t hi, int32_t pool, const char* side) {
  for (int64_t i = lo; i < hi; ++i)
    if (ids[i] < 0 || ids[i] >= pool)
      return fail(FLOWKV_ERANGE, "%s block %d at position %lld outside [0, %d)", side, ids[i],
                  (long long)i, pool);
  return FLOWKV_OK;
}

// End of the maximal +1 run of ids that starts at position i (< hi).
inline int64_t run_end(const int32_t* ids, int64_t i, int64_t hi) {
  int64_t j = i + 1;
  while (j < hi && ids[j] == ids[j - 1] + 1) ++j;
  return j;
}

// Clear the bits of the recorded runs and forget them.
void unmark(Bitmap& seen, std::vector<IdRun>& runs) {
  for (const IdRun& r : runs) seen.clear(r.lo, r.hi);
  runs.clear();
}

// Mark ids[lo, hi) (all inside the pool) in `seen`, recording each run in
// `runs` (empty on entry, with room for hi - lo entries, so nothing allocates
// while bits are set); EDUP on a repeat, naming the first position whose ID
// appeared earlier.  A run's IDs are distinct, so a repeat is a run meeting
// bits already set.  Bits set before a failure are cleared before returning.
int mark_unique(Bitmap& seen, std::vector<IdRun>& runs, const int32_t* ids, int64_t lo,
                int64_t hi, const char* side) {
  for (int64_t i = lo; i < hi;) {
    const int64_t j = run_end(ids, i, hi);
    const int32_t a = ids[i], b = ids[i] + int32_t(j - i);
    if (seen.any(a, b)) {
      int64_t k = i;
      while (!seen.test(ids[k])) ++k;
      unmark(seen, runs);
      return fail(FLOWKV_EDUP, "%s block %d repeated (position %lld)", side, ids[k],
                  (long long)k);
    }
    seen.set(a, b);
    runs.push_back({a, b});
    i = j;
  }
  return FLOWKV_OK;
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

  // receiver IDs: distinct across the whole batch; sender IDs: within a
  // request.  Everything that allocates happens before the first bit is set.
  t_dst_seen.size_for(dst_pool);
  t_src_seen.size_for(src_pool);
  int64_t longest = 0;
  for (int32_t r = 0; r < n_req; ++r) longest = std::max(longest, offsets[r + 1] - offsets[r]);
  t_dst_runs.clear();
  t_src_runs.clear();
  t_dst_runs.reserve(size_t(total));
  t_src_runs.reserve(size_t(longest));
  rc = mark_unique(t_dst_seen, t_dst_runs, D, 0, total, "receiver");
  if (rc) return rc;
  for (int32_t r = 0; r < n_req && !rc; ++r) {
    rc = mark_unique(t_src_seen, t_src_runs, S, offsets[r], offsets[r + 1], "sender");
    if (!rc) unmark(t_src_seen, t_src_runs);
  }
  unmark(t_dst_seen, t_dst_runs);
  if (rc) return rc;

  // a plan has at most one record per block: with room for that many the
  // records are written in the counting pass; otherwise they are counted
  // first, so that ECAP leaves the output untouched
  if (cap < total) {
    int64_t need = 0;
    for (int32_t r = 0; r < n_req; ++r)
      for (int64_t i = offsets[r]; i < offsets[r + 1]; ++i)
        need += (i == offsets[r] || breaks(S, D, i)) ? 1 : 0;
    if (need > cap) {
      *n_out = need;
      return fail(FLOWKV_ECAP, "%lld segments need room, capacity %lld", (long long)need,
                  (long long)cap);
    }
  }
  if (total > 0 && !out) return fail(FLOWKV_EINVAL, "NULL output segments");

  // the records, then their lengths: a run ends where the next record starts
  // (runs never span requests, and an empty request adds no record), the
  // last one at the plan's end
  int64_t k = 0;
  for (int32_t r = 0; r < n_req; ++r) {
    for (int64_t i = offsets[r]; i < offsets[r + 1]; ++i) {
      if (i == offsets[r] || breaks(S, D, i)) {
        out[k].src_block = S[i];
        out[k].dst_block = D[i];
        out[k].first = int32_t(i);
        ++k;
      }
    }
  }
  for (int64_t j = 0; j < k; ++j)
    out[j].n_blocks = int32_t((j + 1 < k ? int64_t(out[j + 1].first) : total) - out[j].first);
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
