// Load-aware scheduler: FlowKV (arXiv 2504.03775), section 3.4 and Appendix A
// (Algorithm 1 and the node status indicators).  Host code; the arithmetic is
// IEEE double in the order the header states, so its results are exact
// functions of the inputs.
#include <cmath>
#include <cstdint>
#include <new>
#include <vector>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

namespace {

constexpr int kInd = FLOWKV_SCHED_INDICATORS;
constexpr int kTerms = FLOWKV_SCHED_TERMS;
// the indicators each role's score reads, in the order of its weights
constexpr int kPrefillTerms[kTerms] = {0, 1, 2, 3, 8, 9, 10, 11};
constexpr int kDecodeTerms[kTerms] = {4, 5, 6, 7, 8, 9, 10, 11};

bool valid_role(int32_t r) {
  return r == FLOWKV_ROLE_PREFILL || r == FLOWKV_ROLE_DECODE || r == FLOWKV_ROLE_OFFLINE;
}

}  // namespace

struct flowkv_sched {
  flowkv_sched_params p;
  int32_t n;
  std::vector<int32_t> roles;
  // per node a ring of `window` samples of 12 indicators; the oldest sample
  // sits at `head`, and `count` samples are valid (the same for every node)
  std::vector<double> ring;
  int32_t head = 0, count = 0;
  int32_t extreme_run = 0;     // consecutive overload evaluations
  int32_t low_run = 0;         // consecutive low-load evaluations
  std::vector<double> scores;  // scratch: (C_i^p, C_i^d) per node
};

extern "C" int flowkv_sched_create(const flowkv_sched_params* params, int32_t n_nodes,
                                   const int32_t* roles, flowkv_sched** out) {
  if (!params || !roles || !out) return fail(FLOWKV_EINVAL, "NULL argument");
  const flowkv_sched_params& p = *params;
  if (n_nodes < 1 || n_nodes > (1 << 20))
    return fail(FLOWKV_EINVAL, "n_nodes %d: need 1..2^20", n_nodes);
  if (p.window < 1 || p.window > FLOWKV_SCHED_MAX_WINDOW)
    return fail(FLOWKV_EINVAL, "window %d: need 1..%d", p.window, FLOWKV_SCHED_MAX_WINDOW);
  if (p.scale_after < 1) return fail(FLOWKV_EINVAL, "scale_after %d: need >= 1", p.scale_after);
  for (int k = 0; k < kInd; ++k)
    if (!(p.scale[k] > 0) || !std::isfinite(p.scale[k]))
      return fail(FLOWKV_EINVAL, "scale[%d] must be positive and finite", k);
  for (int t = 0; t < kTerms; ++t)
    if (!std::isfinite(p.w_prefill[t]) || !std::isfinite(p.w_decode[t]))
      return fail(FLOWKV_EINVAL, "weight %d not finite", t);
  if (!(p.eps_p_low > 0 && p.eps_p_low <= p.eps_p_high && p.eps_d_low > 0 &&
        p.eps_d_low <= p.eps_d_high) ||
      !std::isfinite(p.eps_p_high) || !std::isfinite(p.eps_d_high) ||
      std::isnan(p.idle_threshold))
    return fail(FLOWKV_EINVAL, "thresholds need 0 < low <= high, finite");
  if (!(p.eps_p_min >= 0 && p.eps_p_min <= p.eps_p_low && p.eps_d_min >= 0 &&
        p.eps_d_min <= p.eps_d_low))
    return fail(FLOWKV_EINVAL, "low-load thresholds need 0 <= min <= low");
  for (int32_t i = 0; i < n_nodes; ++i)
    if (!valid_role(roles[i])) return fail(FLOWKV_EINVAL, "role of node %d is %d", i, roles[i]);
  flowkv_sched* s = new (std::nothrow) flowkv_sched;
  if (!s) return fail(FLOWKV_ENOMEM, "out of host memory");
  try {
    s->p = p;
    s->n = n_nodes;
    s->roles.assign(roles, roles + n_nodes);
    s->ring.assign(size_t(n_nodes) * p.window * kInd, 0.0);
    s->scores.assign(size_t(n_nodes) * 2, 0.0);
  } catch (const std::bad_alloc&) {
    delete s;
    return fail(FLOWKV_ENOMEM, "out of host memory");
  }
  *out = s;
  return ok();
}

extern "C" void flowkv_sched_destroy(flowkv_sched* s) { delete s; }

extern "C" int flowkv_sched_set_role(flowkv_sched* s, int32_t node, int32_t role) {
  if (!s) return fail(FLOWKV_EINVAL, "NULL scheduler");
  if (node < 0 || node >= s->n) return fail(FLOWKV_ERANGE, "node %d of %d", node, s->n);
  if (!valid_role(role)) return fail(FLOWKV_EINVAL, "role %d", role);
  s->roles[node] = role;
  return ok();
}

extern "C" int flowkv_sched_observe(flowkv_sched* s, const double* status) {
  if (!s || !status) return fail(FLOWKV_EINVAL, "NULL argument");
  const int32_t W = s->p.window;
  // the slot after the newest; when the window is full it is the oldest
  const int32_t slot = (s->head + s->count) % W;
  for (int32_t i = 0; i < s->n; ++i) {
    double* dst = &s->ring[(size_t(i) * W + slot) * kInd];
    for (int k = 0; k < kInd; ++k) dst[k] = status[size_t(i) * kInd + k];
  }
  if (s->count < W)
    ++s->count;
  else
    s->head = (s->head + 1) % W;
  return ok();
}

extern "C" int flowkv_sched_evaluate(flowkv_sched* s, flowkv_sched_result* res,
                                     int32_t* idle_nodes, double* node_scores) {
  if (!s || !res) return fail(FLOWKV_EINVAL, "NULL argument");
  if (s->count == 0) return fail(FLOWKV_EINVAL, "no status observed yet");
  const flowkv_sched_params& p = s->p;
  const int32_t W = p.window;
  // per node: window means (oldest sample first), normalised, then the two
  // weighted sums term by term
  for (int32_t i = 0; i < s->n; ++i) {
    double acc[kInd] = {};
    const double* node = &s->ring[size_t(i) * W * kInd];
    for (int32_t j = 0, slot = s->head; j < s->count; ++j, slot = slot + 1 == W ? 0 : slot + 1) {
      const double* x = node + size_t(slot) * kInd;
      for (int k = 0; k < kInd; ++k) acc[k] += x[k];
    }
    double norm[kInd];
    for (int k = 0; k < kInd; ++k) norm[k] = acc[k] / double(s->count) / p.scale[k];
    double cp = 0.0, cd = 0.0;
    for (int t = 0; t < kTerms; ++t) cp += p.w_prefill[t] * norm[kPrefillTerms[t]];
    for (int t = 0; t < kTerms; ++t) cd += p.w_decode[t] * norm[kDecodeTerms[t]];
    s->scores[2 * size_t(i)] = cp;
    s->scores[2 * size_t(i) + 1] = cd;
  }
  double sp = 0.0, sd = 0.0;
  int32_t np = 0, nd = 0;
  for (int32_t i = 0; i < s->n; ++i) {
    if (s->roles[i] == FLOWKV_ROLE_PREFILL) {
      sp += s->scores[2 * size_t(i)];
      ++np;
    } else if (s->roles[i] == FLOWKV_ROLE_DECODE) {
      sd += s->scores[2 * size_t(i) + 1];
      ++nd;
    }
  }
  flowkv_sched_result r{};
  r.c_prefill = np ? sp / double(np) : 0.0;
  r.c_decode = nd ? sd / double(nd) : 0.0;
  r.switch_to = -1;
  int32_t n_idle = 0;
  if (std::fabs(r.c_prefill) < p.eps_p_min && std::fabs(r.c_decode) < p.eps_d_min) {
    // low load: the extreme scenario's other side; once it has lasted, each
    // role with more than one node may give one up
    r.scenario = FLOWKV_SCENARIO_LOW_LOAD;
    s->extreme_run = 0;
    if (++s->low_run >= p.scale_after) {
      r.scale_prefill = np > 1 ? -1 : 0;
      r.scale_decode = nd > 1 ? -1 : 0;
      s->low_run = 0;
    }
  } else if (std::fabs(r.c_prefill) <= p.eps_p_low && std::fabs(r.c_decode) <= p.eps_d_low) {
    r.scenario = FLOWKV_SCENARIO_NORMAL;
    s->extreme_run = 0;
    s->low_run = 0;
  } else if (std::fabs(r.c_prefill) <= p.eps_p_high && std::fabs(r.c_decode) <= p.eps_d_high) {
    r.scenario = FLOWKV_SCENARIO_IMBALANCED;
    s->extreme_run = 0;
    s->low_run = 0;
    const int32_t busier = r.c_prefill / p.eps_p_low >= r.c_decode / p.eps_d_low
                               ? FLOWKV_ROLE_PREFILL
                               : FLOWKV_ROLE_DECODE;
    r.switch_to = busier;
    for (int32_t i = 0; i < s->n; ++i) {
      const int32_t role = s->roles[i];
      if (role != busier && role != FLOWKV_ROLE_OFFLINE &&
          s->scores[2 * size_t(i) + role] < p.idle_threshold) {
        if (idle_nodes) idle_nodes[n_idle] = i;
        ++n_idle;
      }
    }
  } else {
    r.scenario = FLOWKV_SCENARIO_EXTREME;
    s->low_run = 0;
    if (++s->extreme_run >= p.scale_after) {
      r.scale_prefill = std::fabs(r.c_prefill) > p.eps_p_high;
      r.scale_decode = std::fabs(r.c_decode) > p.eps_d_high;
      s->extreme_run = 0;
    }
  }
  r.n_idle = n_idle;
  if (node_scores)
    for (size_t k = 0; k < size_t(s->n) * 2; ++k) node_scores[k] = s->scores[k];
  *res = r;
  return ok();
}

extern "C" int flowkv_sched_route(const flowkv_sched* s, int64_t prompt_tokens,
                                  const int64_t* prefix_hit, const int64_t* queued_tokens,
                                  const double* prefill_rate, int64_t kv_bytes,
                                  const double* xfer_sec_per_byte, const double* xfer_latency,
                                  const int64_t* free_bytes, int32_t* prefill_node,
                                  int32_t* decode_node) {
  if (!s || !prefix_hit || !queued_tokens || !prefill_rate || !xfer_sec_per_byte ||
      !xfer_latency || !free_bytes || !prefill_node || !decode_node)
    return fail(FLOWKV_EINVAL, "NULL argument");
  if (prompt_tokens < 0 || kv_bytes < 0) return fail(FLOWKV_EINVAL, "negative sizes");
  const int32_t n = s->n;
  int32_t best_p = -1;
  double best_t = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    if (s->roles[i] != FLOWKV_ROLE_PREFILL || !(prefill_rate[i] > 0)) continue;
    const int64_t hit = prefix_hit[i] < prompt_tokens ? prefix_hit[i] : prompt_tokens;
    const double t = double(queued_tokens[i] + (prompt_tokens - hit)) / prefill_rate[i];
    if (best_p < 0 || t < best_t) {
      best_p = i;
      best_t = t;
    }
  }
  int32_t best_d = -1;
  if (best_p >= 0) {
    double best_l = 0.0;
    for (int32_t j = 0; j < n; ++j) {
      if (s->roles[j] != FLOWKV_ROLE_DECODE || free_bytes[j] < kv_bytes) continue;
      const size_t e = size_t(best_p) * n + j;
      const double lat = xfer_latency[e] + double(kv_bytes) * xfer_sec_per_byte[e];
      if (best_d < 0 || lat < best_l) {
        best_d = j;
        best_l = lat;
      }
    }
  }
  *prefill_node = best_p;
  *decode_node = best_d;
  return ok();
}
