// Host-side stress driver for the allocator, planner and scheduler of libflowkv, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitizers.py (CPU only).
//
// It runs seeded random alloc / free / mark_used streams on every policy and
// checks, after every call, the invariants the C ABI promises: no block handed
// out twice, free + held = pool size, stats agree with a recount, failed calls
// change nothing.  It plans random block lists (single and batch) and checks
// that the runs reassemble both lists, are maximal, and that `first` tiles
// the plan; it calls every entry point with every kind of bad argument.
// Exit status 0 = all checks passed.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "flowkv.h"

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      std::exit(1);                                                          \
    }                                                                        \
  } while (0)

namespace {

struct Model {
  int32_t P;
  std::vector<uint8_t> held;  // 1 = handed out or marked
};

void recount(const flowkv_allocator* a, const Model& m) {
  flowkv_alloc_stats st{};
  CHECK(flowkv_allocator_stats(a, &st) == FLOWKV_OK);
  int64_t free_blocks = 0, runs = 0, longest = 0, cur = 0;
  for (int32_t b = 0; b < m.P; ++b) {
    if (m.held[b]) {
      cur = 0;
      continue;
    }
    ++free_blocks;
    if (cur == 0) ++runs;
    ++cur;
    if (cur > longest) longest = cur;
  }
  CHECK(st.free_blocks == free_blocks);
  CHECK(st.free_segments == runs);
  CHECK(st.largest_free == longest);
}

void allocator_stream(int policy, uint64_t seed) {
  std::mt19937_64 rng(seed);
  const int32_t P = int32_t(1 + rng() % 400);
  flowkv_allocator* a = nullptr;
  CHECK(flowkv_allocator_create(P, policy, seed, &a) == FLOWKV_OK && a);
  Model m{P, std::vector<uint8_t>(P, 0)};
  std::vector<std::vector<int32_t>> live;
  // pre-occupancy
  {
    std::vector<int32_t> pre;
    for (int32_t b = 0; b < P; ++b)
      if (rng() % 4 == 0) pre.push_back(b);
    std::shuffle(pre.begin(), pre.end(), rng);
    CHECK(flowkv_mark_used(a, pre.data(), int32_t(pre.size())) == FLOWKV_OK);
    for (int32_t b : pre) m.held[b] = 1;
  }
  recount(a, m);
  for (int step = 0; step < 300; ++step) {
    const int kind = int(rng() % 10);
    if (kind < 4 && !live.empty()) {
      const size_t i = rng() % live.size();
      CHECK(flowkv_free(a, live[i].data(), int32_t(live[i].size())) == FLOWKV_OK);
      for (int32_t b : live[i]) m.held[b] = 0;
      live.erase(live.begin() + long(i));
    } else if (kind < 8) {
      const int32_t n = int32_t(rng() % (P / 3 + 2));
      std::vector<int32_t> ids(size_t(n) + 1, -7);
      int64_t free_now = 0;
      for (uint8_t h : m.held) free_now += !h;
      const int rc = flowkv_alloc(a, n, ids.data());
      if (n > free_now) {
        CHECK(rc == FLOWKV_ENOSPC);
        CHECK(ids[0] == -7 || n == 0);
      } else {
        CHECK(rc == FLOWKV_OK);
        CHECK(ids[size_t(n)] == -7);  // nothing written past n
        ids.resize(size_t(n));
        for (int32_t b : ids) {
          CHECK(b >= 0 && b < P);
          CHECK(!m.held[b]);
          m.held[b] = 1;
        }
        live.push_back(ids);
      }
    } else {
      // rejected calls must change nothing
      std::vector<int32_t> bad;
      switch (rng() % 4) {
        case 0: bad = {P}; break;                           // out of range
        case 1: bad = {-1}; break;                          // out of range
        case 2: {                                           // freeing a free block
          for (int32_t b = 0; b < P; ++b)
            if (!m.held[b]) {
              bad = {b};
              break;
            }
          break;
        }
        default:                                            // repeated ID
          if (!live.empty() && !live[0].empty()) bad = {live[0][0], live[0][0]};
      }
      if (!bad.empty()) {
        const int rc = flowkv_free(a, bad.data(), int32_t(bad.size()));
        CHECK(rc == FLOWKV_ERANGE || rc == FLOWKV_EDUP);
      }
    }
    recount(a, m);
  }
  flowkv_allocator_destroy(a);
}

void plan_cases(uint64_t seed) {
  std::mt19937_64 rng(seed);
  const int32_t P = int32_t(1 + rng() % 300);
  const int n_req = int(1 + rng() % 5);
  std::vector<int32_t> perm_s(P), perm_d(P);
  for (int32_t i = 0; i < P; ++i) perm_s[i] = perm_d[i] = i;
  std::shuffle(perm_s.begin(), perm_s.end(), rng);
  std::shuffle(perm_d.begin(), perm_d.end(), rng);
  // sort stretches so contiguous runs appear
  for (int32_t i = 0; i + 8 < P; i += 9)
    if (rng() % 2) {
      std::sort(perm_s.begin() + i, perm_s.begin() + i + 8);
      std::sort(perm_d.begin() + i, perm_d.begin() + i + 8);
    }
  const int32_t total = int32_t(rng() % (P + 1));
  std::vector<int64_t> off(size_t(n_req) + 1, 0);
  for (int r = 1; r < n_req; ++r) off[size_t(r)] = int64_t(rng() % (total + 1));
  off[size_t(n_req)] = total;
  std::sort(off.begin(), off.end());
  std::vector<flowkv_segment> out(size_t(total) + 1);
  int64_t k = -1;
  CHECK(flowkv_plan_batch(n_req, off.data(), perm_s.data(), perm_d.data(), P, P, out.data(),
                          int64_t(out.size()), &k) == FLOWKV_OK);
  // reassemble, check maximality, request boundaries and `first`
  int64_t pos = 0;
  for (int64_t j = 0; j < k; ++j) {
    const flowkv_segment& s = out[size_t(j)];
    CHECK(s.n_blocks >= 1);
    CHECK(s.first == pos);
    for (int32_t q = 0; q < s.n_blocks; ++q) {
      CHECK(perm_s[size_t(pos + q)] == s.src_block + q);
      CHECK(perm_d[size_t(pos + q)] == s.dst_block + q);
    }
    const int64_t next = pos + s.n_blocks;
    bool boundary = next == total;
    for (int r = 1; r <= n_req; ++r) boundary |= off[size_t(r)] == next;
    if (!boundary)  // a run ends inside a request only where a list breaks
      CHECK(perm_s[size_t(next)] != s.src_block + s.n_blocks ||
            perm_d[size_t(next)] != s.dst_block + s.n_blocks);
    pos = next;
  }
  CHECK(pos == total);
  // ECAP reports the exact need and writes nothing
  if (k > 1) {
    int64_t need = -1;
    std::vector<flowkv_segment> small(1, flowkv_segment{-9, -9, -9, -9});
    CHECK(flowkv_plan_batch(n_req, off.data(), perm_s.data(), perm_d.data(), P, P, small.data(),
                            1, &need) == FLOWKV_ECAP);
    CHECK(need == k && small[0].src_block == -9);
  }
}

void bad_arguments() {
  int64_t n = 0;
  flowkv_segment seg{};
  const int32_t ids[2] = {0, 0};
  const int32_t other[2] = {0, 1};
  CHECK(flowkv_plan(nullptr, nullptr, 0, 4, 4, nullptr, 0, &n) == FLOWKV_OK && n == 0);
  CHECK(flowkv_plan(ids, other, 2, 4, 4, &seg, 1, nullptr) == FLOWKV_EINVAL);
  CHECK(flowkv_plan(nullptr, other, 1, 4, 4, &seg, 1, &n) == FLOWKV_EINVAL);
  CHECK(flowkv_plan(ids, other, -1, 4, 4, &seg, 1, &n) == FLOWKV_EINVAL);
  CHECK(flowkv_plan(ids, other, 2, 4, 4, &seg, 2, &n) == FLOWKV_EDUP);
  CHECK(flowkv_plan(other, ids, 2, 4, 4, &seg, 2, &n) == FLOWKV_EDUP);
  CHECK(flowkv_plan(other, other, 2, 1, 4, &seg, 2, &n) == FLOWKV_ERANGE);
  CHECK(flowkv_plan(other, other, 2, 4, 4, &seg, -1, &n) == FLOWKV_EINVAL);
  const int64_t bad_off[3] = {0, 2, 1};
  CHECK(flowkv_plan_batch(2, bad_off, other, other, 4, 4, &seg, 2, &n) == FLOWKV_EINVAL);
  CHECK(flowkv_plan_batch(-1, bad_off, other, other, 4, 4, &seg, 2, &n) == FLOWKV_EINVAL);
  CHECK(flowkv_plan_batch(1, nullptr, other, other, 4, 4, &seg, 2, &n) == FLOWKV_EINVAL);
  flowkv_allocator* a = nullptr;
  CHECK(flowkv_allocator_create(-1, 0, 0, &a) == FLOWKV_EINVAL && !a);
  CHECK(flowkv_allocator_create(4, 9, 0, &a) == FLOWKV_EINVAL && !a);
  CHECK(flowkv_allocator_create(4, 0, 0, nullptr) == FLOWKV_EINVAL);
  CHECK(flowkv_allocator_create(0, 0, 0, &a) == FLOWKV_OK && a);
  int32_t out = -3;
  CHECK(flowkv_alloc(a, 1, &out) == FLOWKV_ENOSPC && out == -3);
  CHECK(flowkv_alloc(a, 0, nullptr) == FLOWKV_OK);
  CHECK(flowkv_alloc(nullptr, 1, &out) == FLOWKV_EINVAL);
  CHECK(flowkv_free(a, nullptr, 1) == FLOWKV_EINVAL);
  CHECK(flowkv_mark_used(a, nullptr, -2) == FLOWKV_EINVAL);
  CHECK(flowkv_allocator_stats(a, nullptr) == FLOWKV_EINVAL);
  flowkv_allocator_destroy(a);
  flowkv_allocator_destroy(nullptr);
  for (int c = -7; c <= 1; ++c) CHECK(flowkv_strerror(c) != nullptr);
  CHECK(flowkv_last_error() != nullptr);
}

// Load-aware scheduler: random parameters, status streams and role changes;
// after every evaluation the result must be well formed (scenario in range,
// idle nodes ascending, in range and of the role that is not asked for, the
// node scores finite) and every route must name nodes of the right role.
void sched_stream(uint64_t seed) {
  std::mt19937_64 rng(seed);
  std::uniform_real_distribution<double> u01(0.0, 1.0);
  flowkv_sched_params p{};
  p.window = 1 + int32_t(rng() % 8);
  p.scale_after = 1 + int32_t(rng() % 3);
  for (double& x : p.scale) x = 0.5 + 8.0 * u01(rng);
  for (double& x : p.w_prefill) x = u01(rng);
  for (double& x : p.w_decode) x = u01(rng);
  p.eps_p_low = 0.1 + u01(rng);
  p.eps_d_low = 0.1 + u01(rng);
  p.eps_p_high = p.eps_p_low * (1.0 + 2.0 * u01(rng));
  p.eps_d_high = p.eps_d_low * (1.0 + 2.0 * u01(rng));
  p.idle_threshold = 0.5 * u01(rng);
  const int32_t n = 1 + int32_t(rng() % 24);
  std::vector<int32_t> roles(n);
  for (auto& r : roles) r = int32_t(rng() % 2);
  flowkv_sched* s = nullptr;
  CHECK(flowkv_sched_create(&p, n, roles.data(), &s) == FLOWKV_OK && s);
  flowkv_sched_result res{};
  std::vector<int32_t> idle(n, -7);
  std::vector<double> scores(2 * size_t(n));
  CHECK(flowkv_sched_evaluate(s, &res, idle.data(), scores.data()) == FLOWKV_EINVAL);
  std::vector<double> st(size_t(n) * FLOWKV_SCHED_INDICATORS);
  double level = 0.1 + 2.0 * u01(rng);
  for (int step = 0; step < 80; ++step) {
    level *= 0.7 + 0.7 * u01(rng);
    for (double& x : st) x = level * 8.0 * u01(rng);
    CHECK(flowkv_sched_observe(s, st.data()) == FLOWKV_OK);
    if (rng() % 8 == 0) {
      const int32_t i = int32_t(rng() % n), role = int32_t(rng() % 2);
      CHECK(flowkv_sched_set_role(s, i, role) == FLOWKV_OK);
      roles[i] = role;
    }
    CHECK(flowkv_sched_evaluate(s, &res, idle.data(), scores.data()) == FLOWKV_OK);
    CHECK(res.scenario >= FLOWKV_SCENARIO_NORMAL && res.scenario <= FLOWKV_SCENARIO_EXTREME);
    CHECK(res.n_idle >= 0 && res.n_idle <= n);
    if (res.scenario != FLOWKV_SCENARIO_IMBALANCED) CHECK(res.n_idle == 0 && res.switch_to == -1);
    for (int32_t k = 0; k < res.n_idle; ++k) {
      CHECK(idle[k] >= 0 && idle[k] < n && roles[idle[k]] != res.switch_to);
      if (k) CHECK(idle[k] > idle[k - 1]);
    }
    for (double x : scores) CHECK(x == x && x >= 0.0);
    // evaluating without the optional outputs gives the same result
    flowkv_sched_result again{};
    CHECK(flowkv_sched_observe(s, st.data()) == FLOWKV_OK);
    CHECK(flowkv_sched_evaluate(s, &again, nullptr, nullptr) == FLOWKV_OK);
    CHECK(again.n_idle >= 0 && again.n_idle <= n);
  }
  std::vector<int64_t> hit(n), queued(n), free_b(n);
  std::vector<double> rate(n), spb(size_t(n) * n), lat(size_t(n) * n);
  for (int k = 0; k < 200; ++k) {
    const int64_t prompt = int64_t(rng() % 30000), kv = int64_t(rng() % (int64_t(1) << 33));
    for (int32_t i = 0; i < n; ++i) {
      hit[i] = int64_t(rng() % 40000);
      queued[i] = int64_t(rng() % 100000);
      rate[i] = (rng() % 4) ? 1000.0 + 10000.0 * u01(rng) : 0.0;
      free_b[i] = (rng() % 3) ? kv + int64_t(rng() % 1000) : kv - 1;
    }
    for (double& x : spb) x = 1e-10 + 1e-9 * u01(rng);
    for (double& x : lat) x = 1e-3 * u01(rng);
    int32_t pn = -5, dn = -5;
    CHECK(flowkv_sched_route(s, prompt, hit.data(), queued.data(), rate.data(), kv, spb.data(),
                             lat.data(), free_b.data(), &pn, &dn) == FLOWKV_OK);
    CHECK(pn == -1 || (pn >= 0 && pn < n && roles[pn] == FLOWKV_ROLE_PREFILL && rate[pn] > 0));
    if (pn < 0) CHECK(dn == -1);
    CHECK(dn == -1 || (dn >= 0 && dn < n && roles[dn] == FLOWKV_ROLE_DECODE && free_b[dn] >= kv));
  }
  // bad arguments
  int32_t pn, dn;
  CHECK(flowkv_sched_route(s, -1, hit.data(), queued.data(), rate.data(), 1, spb.data(),
                           lat.data(), free_b.data(), &pn, &dn) == FLOWKV_EINVAL);
  CHECK(flowkv_sched_route(s, 1, nullptr, queued.data(), rate.data(), 1, spb.data(), lat.data(),
                           free_b.data(), &pn, &dn) == FLOWKV_EINVAL);
  CHECK(flowkv_sched_set_role(s, n, 0) == FLOWKV_ERANGE);
  CHECK(flowkv_sched_set_role(s, -1, 0) == FLOWKV_ERANGE);
  CHECK(flowkv_sched_set_role(s, 0, 3) == FLOWKV_EINVAL);
  CHECK(flowkv_sched_set_role(nullptr, 0, 0) == FLOWKV_EINVAL);
  CHECK(flowkv_sched_observe(s, nullptr) == FLOWKV_EINVAL);
  CHECK(flowkv_sched_evaluate(s, nullptr, nullptr, nullptr) == FLOWKV_EINVAL);
  flowkv_sched_destroy(s);
  flowkv_sched_destroy(nullptr);
  flowkv_sched* t = nullptr;
  CHECK(flowkv_sched_create(nullptr, 1, roles.data(), &t) == FLOWKV_EINVAL && !t);
  CHECK(flowkv_sched_create(&p, 0, roles.data(), &t) == FLOWKV_EINVAL && !t);
  flowkv_sched_params q = p;
  q.window = FLOWKV_SCHED_MAX_WINDOW + 1;
  CHECK(flowkv_sched_create(&q, 1, roles.data(), &t) == FLOWKV_EINVAL && !t);
  q = p;
  q.eps_d_high = q.eps_d_low / 2;
  CHECK(flowkv_sched_create(&q, 1, roles.data(), &t) == FLOWKV_EINVAL && !t);
  int32_t bad_role = 9;
  CHECK(flowkv_sched_create(&p, 1, &bad_role, &t) == FLOWKV_EINVAL && !t);
}

}  // namespace

int main(int argc, char** argv) {
  const int rounds = argc > 1 ? std::atoi(argv[1]) : 200;
  bad_arguments();
  for (int r = 0; r < rounds; ++r) {
    for (int policy = 0; policy < 3; ++policy) allocator_stream(policy, uint64_t(r) * 7 + policy);
    plan_cases(uint64_t(r) * 13 + 5);
    sched_stream(uint64_t(r) * 17 + 3);
  }
  std::printf("host_check: %d rounds ok\n", rounds);
  return 0;
}
