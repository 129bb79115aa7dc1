// Mixed-precision bit allocation (Section 3.3) on the host: the memory budget
// (S_low, B_base, the B_delta releases, B_total), size-tiered upgrades in
// descending sensitivity under the budget constraint, and the three back-off
// rules.  Sizes are int64 counts of 1/64-bit units, so every fit decision is
// an exact comparison.  Rule 2 keeps the upgraded tensors in a max-heap by
// (parameters, sensitivity rank); the freeable totals of rules 2 and 3 are
// kept incrementally, so a plan costs O(n log n).
#include <math.h>

#include <algorithm>
#include <queue>
#include <tuple>
#include <vector>

#include "internal.h"

namespace {

moeq_status bad(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  moeq::vset_error(MOEQ_ERR_INVALID_ARG, fmt, ap);
  va_end(ap);
  return MOEQ_ERR_INVALID_ARG;
}

constexpr int64_t kUnitsPerByte = 8 * 64;
constexpr double kUnitsPerGB = 64.0 * 8e9;

void partition_order(int n_layers, std::vector<int32_t>& out) {
  out.clear();
  std::vector<std::pair<int, int>> level{{0, n_layers}}, next;
  while (!level.empty()) {
    next.clear();
    for (const auto& iv : level) {
      const int lo = iv.first, hi = iv.second;
      if (lo >= hi) continue;
      const int mid = hi - lo == 1 ? lo : (lo + hi + 1) / 2;
      out.push_back(mid);
      next.push_back({lo, mid});
      next.push_back({mid + 1, hi});
    }
    level.swap(next);
  }
}

moeq_status check_params(const moeq_plan_params* p) {
  if (!p) return bad("plan params are NULL");
  if (p->n_levels < 3 || p->n_levels > MOEQ_PLAN_MAX_LEVELS)
    return bad("n_levels %d outside 3..%d", p->n_levels, MOEQ_PLAN_MAX_LEVELS);
  for (int i = 0; i < p->n_levels; ++i) {
    if (p->width64[i] < 1 || p->width64[i] > 4096) return bad("width64[%d] = %d outside 1..4096", i, p->width64[i]);
    if (i && p->width64[i] <= p->width64[i - 1]) return bad("width64 must be strictly increasing (level %d)", i);
  }
  if (!(0 <= p->low_prime && p->low_prime < p->low && p->low < p->floor && p->floor <= p->medium_level &&
        p->medium_level <= p->small_level && p->small_level < p->n_levels))
    return bad("levels must satisfy low_prime < low < floor <= medium_level <= small_level < n_levels");
  if (p->small_params < 1 || p->medium_params < p->small_params)
    return bad("need 1 <= small_params <= medium_params");
  if (p->m_limit_bytes > (1ull << 50)) return bad("m_limit_bytes above 2^50");
  if (p->n_moe_layers < 0 || p->n_moe_layers > 4096) return bad("n_moe_layers %d outside 0..4096", p->n_moe_layers);
  return MOEQ_OK;
}

}  // namespace

extern "C" {

moeq_status moeq_sensitivity(int32_t n, double ppl_low, const double* ppl_high, const int64_t* params,
                             const int64_t* layer_params, double* sens) {
  if (n < 0) return bad("n %d is negative", n);
  if (n > 0 && (!ppl_high || !params || !layer_params || !sens))
    return bad("ppl_high, params, layer_params and sens must not be NULL");
  if (!isfinite(ppl_low)) return bad("ppl_low is not finite");
  for (int t = 0; t < n; ++t) {
    if (!isfinite(ppl_high[t])) return bad("ppl_high[%d] is not finite", t);
    if (params[t] < 1 || layer_params[t] < params[t])
      return bad("tensor %d: need 1 <= params <= layer_params", t);
  }
  for (int t = 0; t < n; ++t) {
    const double rho = (double)params[t] / (double)layer_params[t];
    sens[t] = (ppl_low - ppl_high[t]) / rho;
  }
  return MOEQ_OK;
}

moeq_status moeq_layer_order(int32_t n_layers, int32_t* order) {
  if (n_layers < 1 || n_layers > 4096) return bad("n_layers %d outside 1..4096", n_layers);
  if (!order) return bad("order is NULL");
  std::vector<int32_t> o;
  partition_order(n_layers, o);
  std::copy(o.begin(), o.end(), order);
  return MOEQ_OK;
}

moeq_status moeq_plan_bits(const moeq_plan_params* p, int32_t n, const int64_t* params, const double* sens,
                           const int32_t* kind, const int32_t* layer, int32_t* level, moeq_plan_report* report) {
  moeq_status st = check_params(p);
  if (st != MOEQ_OK) return st;
  if (n < 1 || n > (1 << 20)) return bad("n %d outside 1..2^20", n);
  if (!params || !sens || !kind || !level) return bad("params, sens, kind and level must not be NULL");
  int64_t total_params = 0;
  bool any_routed = false;
  for (int t = 0; t < n; ++t) {
    if (params[t] < 1 || params[t] > (int64_t(1) << 45)) return bad("params[%d] outside 1..2^45", t);
    total_params += params[t];
    if (total_params > (int64_t(1) << 45)) return bad("the parameter total exceeds 2^45");
    if (!isfinite(sens[t])) return bad("sens[%d] is not finite", t);
    if (kind[t] < MOEQ_TENSOR_OTHER || kind[t] > MOEQ_TENSOR_ROUTED_DOWN) return bad("kind[%d] = %d", t, kind[t]);
    any_routed |= kind[t] != MOEQ_TENSOR_OTHER;
  }
  if (any_routed) {
    if (!layer) return bad("layer is NULL but routed tensors are present");
    for (int t = 0; t < n; ++t)
      if (kind[t] != MOEQ_TENSOR_OTHER && (layer[t] < 0 || layer[t] >= p->n_moe_layers))
        return bad("routed tensor %d has layer %d outside 0..n_moe_layers-1", t, layer[t]);
  }

  const int32_t* w = p->width64;
  const int low = p->low, lowp = p->low_prime, floor_lv = p->floor;
  auto extra = [&](int t, int lv) { return params[t] * (int64_t)(w[lv] - w[low]); };

  for (int t = 0; t < n; ++t) level[t] = low;
  int64_t s_low = 0;
  for (int t = 0; t < n; ++t) s_low += params[t] * (int64_t)w[low];
  const int64_t b_base = (int64_t)p->m_limit_bytes * kUnitsPerByte - s_low;
  int64_t released = 0, used = 0;
  int n_rule2 = 0, n_rule3 = 0, n_up = 0;

  // rule 3's queue: (pass, layer position, kind, index); pass 0 = gate/up, 1 = down
  std::vector<int32_t> pos_of(p->n_moe_layers > 0 ? p->n_moe_layers : 1, 0);
  if (p->n_moe_layers > 0) {
    std::vector<int32_t> o;
    partition_order(p->n_moe_layers, o);
    for (int i = 0; i < (int)o.size(); ++i) pos_of[o[i]] = i;
  }
  std::vector<std::tuple<int, int, int, int>> keyed;
  for (int t = 0; t < n; ++t)
    if (kind[t] != MOEQ_TENSOR_OTHER)
      keyed.emplace_back(kind[t] == MOEQ_TENSOR_ROUTED_DOWN, pos_of[layer[t]], kind[t], t);
  std::sort(keyed.begin(), keyed.end());
  size_t qi = 0;
  int64_t rule3_left = 0;
  for (const auto& k : keyed) rule3_left += params[std::get<3>(k)] * (int64_t)(w[low] - w[lowp]);
  auto rule3 = [&]() {
    const int t = std::get<3>(keyed[qi++]);
    const int64_t d = params[t] * (int64_t)(w[low] - w[lowp]);
    released += d;
    rule3_left -= d;
    level[t] = lowp;
    ++n_rule3;
  };
  while (used > b_base + released && qi < keyed.size()) rule3();

  // upgrade candidates in descending sensitivity
  std::vector<int32_t> cand, target(n, -1);
  for (int t = 0; t < n; ++t) {
    if (kind[t] != MOEQ_TENSOR_OTHER) continue;
    if (params[t] < p->small_params)
      target[t] = p->small_level;
    else if (params[t] <= p->medium_params)
      target[t] = p->medium_level;
    else
      continue;
    cand.push_back(t);
  }
  std::sort(cand.begin(), cand.end(), [&](int a, int b) { return sens[a] > sens[b] || (sens[a] == sens[b] && a < b); });
  std::vector<int32_t> rank(n, 0);
  for (int i = 0; i < (int)cand.size(); ++i) rank[cand[i]] = i;

  // rule 2's heap: upgraded tensors still above the floor
  std::priority_queue<std::tuple<int64_t, int32_t, int32_t>> heap;
  int64_t rule2_left = 0;  // sum over upgraded tensors of what lowering them to the floor frees
  for (const int t : cand) {
    const int tgt = target[t];
    const int lowest = std::max(tgt - 2, floor_lv);
    int placed = -1;
    for (int lv = tgt; lv >= lowest; --lv)
      if (used + extra(t, lv) <= b_base + released) {
        placed = lv;
        break;
      }
    if (placed < 0) {
      const int64_t need = used + extra(t, lowest) - (b_base + released);
      if (need > rule2_left + rule3_left) continue;
      while (used + extra(t, lowest) > b_base + released) {
        if (!heap.empty()) {
          const int u = std::get<2>(heap.top());
          heap.pop();
          const int64_t d = params[u] * (int64_t)(w[level[u]] - w[level[u] - 1]);
          --level[u];
          used -= d;
          rule2_left -= d;
          ++n_rule2;
          if (level[u] > floor_lv) heap.emplace(params[u], rank[u], u);
        } else {
          rule3();
        }
      }
      placed = lowest;
    }
    level[t] = placed;
    used += extra(t, placed);
    rule2_left += params[t] * (int64_t)(w[placed] - w[floor_lv]);
    ++n_up;
    if (placed > floor_lv) heap.emplace(params[t], rank[t], t);
  }

  if (report) {
    report->s_low_gb = (double)s_low / kUnitsPerGB;
    report->b_base_gb = (double)b_base / kUnitsPerGB;
    report->b_delta_gb = (double)released / kUnitsPerGB;
    report->b_total_gb = (double)(b_base + released) / kUnitsPerGB;
    report->upgrade_gb = (double)used / kUnitsPerGB;
    report->total_gb = (double)(s_low - released + used) / kUnitsPerGB;
    report->n_upgraded = n_up;
    report->n_rule2 = n_rule2;
    report->n_rule3 = n_rule3;
    report->feasible = used <= b_base + released;
  }
  return MOEQ_OK;
}

}  // extern "C"
