// Contiguity-aware paged-block allocator (FlowKV, arXiv 2504.03775, section
// 3.3, allocator paragraph): free blocks are kept as maximal free runs, a
// request is placed in as few runs as possible with the least waste, and
// released blocks merge with free neighbours.
//
// Free runs live in two ordered indexes: by (length, start) for best-fit and
// longest-run queries, and by start for neighbour merging.  Every operation is
// O(k log F) for k runs touched and F free runs; the O(P) work happens only at
// creation.  The FIFO policies are the naive free lists used to build
// fragmented comparison tables.
#include <algorithm>
#include <climits>
#include <cstdint>
#include <deque>
#include <iterator>
#include <map>
#include <new>
#include <set>
#include <utility>
#include <vector>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

struct flowkv_allocator {
  int32_t num_blocks = 0;
  int32_t policy = FLOWKV_POLICY_SEGMENT;
  int64_t free_blocks = 0;
  std::vector<uint8_t> used;  // 1 = in use (2: seen while a list is being checked)

  // FLOWKV_POLICY_SEGMENT
  std::map<int32_t, int32_t> by_start;            // start -> length
  std::set<std::pair<int32_t, int32_t>> by_len;   // (length, start)

  // FIFO policies
  std::deque<int32_t> fifo;

  void insert_run(int32_t start, int32_t len) {
    by_start.emplace(start, len);
    by_len.emplace(len, start);
  }
  void erase_run(int32_t start, int32_t len) {
    by_start.erase(start);
    by_len.erase({len, start});
  }

  // Insert the free run [start, start+len), merging with free neighbours.
  void release_run(int32_t start, int32_t len) {
    auto next = by_start.find(start + len);
    if (next != by_start.end()) {
      int32_t nl = next->second;
      erase_run(start + len, nl);
      len += nl;
    }
    auto it = by_start.lower_bound(start);
    if (it != by_start.begin()) {
      auto prev = std::prev(it);
      if (prev->first + prev->second == start) {
        int32_t ps = prev->first, pl = prev->second;
        erase_run(ps, pl);
        start = ps;
        len += pl;
      }
    }
    insert_run(start, len);
  }

  // Remove [a, b) (all free) from the run that contains it.
  void claim_range(int32_t a, int32_t b) {
    auto it = std::prev(by_start.upper_bound(a));
    int32_t s = it->first, l = it->second;
    erase_run(s, l);
    if (a > s) insert_run(s, a - s);
    if (s + l > b) insert_run(b, s + l - b);
  }
};

namespace {

uint64_t splitmix64_next(uint64_t& state) {
  state += 0x9E3779B97F4A7C15ull;
  uint64_t z = state;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Check ids[0..n): all in range (first, so ERANGE wins over EDUP), pairwise
// distinct, and each in use (want_used) or free (!want_used).  The state
// check marks each ID as seen in this list (used = 2) and undoes the marks
// before returning, so nothing changes and no sorted copy is needed.
int check_ids(flowkv_allocator* a, const int32_t* ids, int32_t n, bool want_used) {
  if (n < 0) return fail(FLOWKV_EINVAL, "negative block count %d", n);
  if (n > 0 && !ids) return fail(FLOWKV_EINVAL, "NULL block list");
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= a->num_blocks)
      return fail(FLOWKV_ERANGE, "block %d outside [0, %d)", ids[i], a->num_blocks);
  const uint8_t want = want_used ? 1 : 0;
  int rc = FLOWKV_OK;
  int32_t i = 0;
  for (; i < n; ++i) {
    uint8_t& u = a->used[ids[i]];
    if (u == 2) {
      rc = fail(FLOWKV_EDUP, "block %d listed twice", ids[i]);
      break;
    }
    if (u != want) {
      rc = fail(FLOWKV_EDUP, "block %d is %s", ids[i],
                want_used ? "already free" : "already in use");
      break;
    }
    u = 2;
  }
  for (int32_t j = 0; j < i; ++j) a->used[ids[j]] = want;
  return rc;
}

// Call f(start, end) for each maximal run of consecutive IDs (each one more
// than the last) of ids[0..n), in list order.
template <class F>
void for_each_run(const int32_t* ids, int32_t n, F f) {
  int32_t i = 0;
  while (i < n) {
    int32_t j = i + 1;
    while (j < n && ids[j] == ids[j - 1] + 1) ++j;
    f(ids[i], ids[j - 1] + 1);
    i = j;
  }
}

}  // namespace

extern "C" int flowkv_allocator_create(int32_t num_blocks, int32_t policy, uint64_t seed,
                                       flowkv_allocator** out) {
  if (!out) return fail(FLOWKV_EINVAL, "NULL output handle");
  if (num_blocks < 0) return fail(FLOWKV_EINVAL, "negative pool size %d", num_blocks);
  if (policy != FLOWKV_POLICY_SEGMENT && policy != FLOWKV_POLICY_FIFO_SORTED &&
      policy != FLOWKV_POLICY_FIFO_SHUFFLED)
    return fail(FLOWKV_EINVAL, "unknown allocator policy %d", policy);
  auto* a = new (std::nothrow) flowkv_allocator();
  if (!a) return fail(FLOWKV_ENOMEM, "out of host memory");
  try {
    a->num_blocks = num_blocks;
    a->policy = policy;
    a->free_blocks = num_blocks;
    a->used.assign(num_blocks, 0);
    if (policy == FLOWKV_POLICY_SEGMENT) {
      if (num_blocks > 0) a->insert_run(0, num_blocks);
    } else {
      std::vector<int32_t> ids(num_blocks);
      for (int32_t i = 0; i < num_blocks; ++i) ids[i] = i;
      if (policy == FLOWKV_POLICY_FIFO_SHUFFLED) {
        uint64_t st = seed;
        for (int64_t i = int64_t(num_blocks) - 1; i >= 1; --i) {
          uint64_t j = splitmix64_next(st) % uint64_t(i + 1);
          std::swap(ids[i], ids[j]);
        }
      }
      a->fifo.assign(ids.begin(), ids.end());
    }
  } catch (const std::bad_alloc&) {
    delete a;
    return fail(FLOWKV_ENOMEM, "out of host memory");
  }
  *out = a;
  return ok();
}

extern "C" void flowkv_allocator_destroy(flowkv_allocator* a) { delete a; }

namespace {

int alloc_impl(flowkv_allocator* a, int32_t n, int32_t* out_ids) {
  if (!a) return fail(FLOWKV_EINVAL, "NULL allocator");
  if (n < 0) return fail(FLOWKV_EINVAL, "negative block count %d", n);
  if (n > 0 && !out_ids) return fail(FLOWKV_EINVAL, "NULL output list");
  if (n > a->free_blocks)
    return fail(FLOWKV_ENOSPC, "%d blocks asked, %lld free", n, (long long)a->free_blocks);
  if (a->policy != FLOWKV_POLICY_SEGMENT) {
    for (int32_t i = 0; i < n; ++i) {
      out_ids[i] = a->fifo.front();
      a->fifo.pop_front();
      a->used[out_ids[i]] = 1;
    }
    a->free_blocks -= n;
    return ok();
  }
  int32_t need = n, pos = 0;
  while (need > 0) {
    // best fit: the shortest run holding `need`, lowest start among equals
    auto fit = a->by_len.lower_bound({need, INT32_MIN});
    if (fit != a->by_len.end()) {
      int32_t len = fit->first, start = fit->second;
      a->erase_run(start, len);
      if (len > need) a->insert_run(start + need, len - need);
      for (int32_t i = 0; i < need; ++i) out_ids[pos++] = start + i;
      need = 0;
    } else {
      // nothing holds the rest: take the longest run whole (lowest start)
      int32_t len = std::prev(a->by_len.end())->first;
      int32_t start = a->by_len.lower_bound({len, INT32_MIN})->second;
      a->erase_run(start, len);
      for (int32_t i = 0; i < len; ++i) out_ids[pos++] = start + i;
      need -= len;
    }
  }
  for (int32_t i = 0; i < n; ++i) a->used[out_ids[i]] = 1;
  a->free_blocks -= n;
  return ok();
}

// Freed runs merge with free neighbours on both sides, so releasing them in
// list order leaves the same maximal free runs as any other order.
int free_impl(flowkv_allocator* a, const int32_t* ids, int32_t n) {
  if (!a) return fail(FLOWKV_EINVAL, "NULL allocator");
  int rc = check_ids(a, ids, n, /*want_used=*/true);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i) a->used[ids[i]] = 0;
  a->free_blocks += n;
  if (a->policy == FLOWKV_POLICY_SEGMENT)
    for_each_run(ids, n, [&](int32_t lo, int32_t hi) { a->release_run(lo, hi - lo); });
  else
    for (int32_t i = 0; i < n; ++i) a->fifo.push_back(ids[i]);
  return ok();
}

// A run of consecutive free IDs lies inside one maximal free run, also after
// other runs of the same list were claimed.
int mark_used_impl(flowkv_allocator* a, const int32_t* ids, int32_t n) {
  if (!a) return fail(FLOWKV_EINVAL, "NULL allocator");
  int rc = check_ids(a, ids, n, /*want_used=*/false);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i) a->used[ids[i]] = 1;
  a->free_blocks -= n;
  if (a->policy == FLOWKV_POLICY_SEGMENT) {
    for_each_run(ids, n, [&](int32_t lo, int32_t hi) { a->claim_range(lo, hi); });
  } else {
    std::deque<int32_t> kept;
    for (int32_t b : a->fifo)
      if (!a->used[b]) kept.push_back(b);
    a->fifo.swap(kept);
  }
  return ok();
}

}  // namespace

extern "C" int flowkv_alloc(flowkv_allocator* a, int32_t n, int32_t* out_ids) {
  return flowkv::guarded([&] { return alloc_impl(a, n, out_ids); });
}

extern "C" int flowkv_free(flowkv_allocator* a, const int32_t* ids, int32_t n) {
  return flowkv::guarded([&] { return free_impl(a, ids, n); });
}

extern "C" int flowkv_mark_used(flowkv_allocator* a, const int32_t* ids, int32_t n) {
  return flowkv::guarded([&] { return mark_used_impl(a, ids, n); });
}

extern "C" int flowkv_allocator_stats(const flowkv_allocator* a, flowkv_alloc_stats* out) {
  if (!a || !out) return fail(FLOWKV_EINVAL, "NULL argument");
  flowkv_alloc_stats st{a->free_blocks, 0, 0};
  if (a->policy == FLOWKV_POLICY_SEGMENT) {
    st.free_segments = int64_t(a->by_start.size());
    st.largest_free = a->by_len.empty() ? 0 : std::prev(a->by_len.end())->first;
  } else {
    int64_t run = 0;
    for (int32_t b = 0; b < a->num_blocks; ++b) {
      if (a->used[b]) {
        run = 0;
        continue;
      }
      if (run == 0) ++st.free_segments;
      ++run;
      st.largest_free = std::max(st.largest_free, run);
    }
  }
  *out = st;
  return ok();
}
