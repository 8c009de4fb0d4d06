// Host-side throughput cost model and routing of trajectories to rollout
// instances (the coordinator's use of this path's cost).
//
// Per-decode-step latency of an instance is charged as attention linear in
// its KV-cache size plus a matrix-multiplication term that is memory bound
// for few running trajectories and compute bound for many, plus a constant;
// throughput is running trajectories over that latency (App. B.1). Routing a
// trajectory to an instance changes that throughput by a marginal gain, and
// the routing strategy walks candidate instances from the oldest model
// version upward, taking the first version group whose best gain reaches a
// fraction mu of the gain on an idle instance (Sec. 5.3; App. D). The rule is
// stated in sf_decode_attn.h next to sf_route.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "sf_internal.h"

namespace {

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

bool valid_model(const sf_cost_model* m) {
  return m && finite_nonneg(m->k1) && finite_nonneg(m->k2) && finite_nonneg(m->k3) && finite_nonneg(m->k4) &&
         finite_nonneg(m->k5) && !std::isnan(m->kv_budget);
}

double step_latency(const sf_cost_model* m, int64_t n, double kv) {
  return m->k1 * kv + std::max(m->k2, m->k3 * double(n)) + m->k4;
}

double throughput(const sf_cost_model* m, int64_t n, double kv) {
  return n == 0 ? 0.0 : double(n) / step_latency(m, n, kv);
}

// The instance after a trajectory of this length is routed to it: it runs
// if it fits the KV budget and nothing waits, else it waits.
sf_instance_state routed(const sf_cost_model* m, sf_instance_state s, double length) {
  const double grown = s.kv_cache + m->k5 * length;
  if (grown <= m->kv_budget && s.num_waiting == 0) {
    s.num_running += 1;
    s.kv_cache = grown;
  } else {
    s.num_waiting += 1;
  }
  return s;
}

double gain(const sf_cost_model* m, const sf_instance_state& s, double length) {
  const sf_instance_state t = routed(m, s, length);
  return throughput(m, t.num_running, t.kv_cache) - throughput(m, s.num_running, s.kv_cache);
}

}  // namespace

extern "C" double sf_cost_throughput(const sf_cost_model* m, const sf_instance_state* s) {
  if (!valid_model(m) || !s || s->num_running < 0) return NAN;
  return throughput(m, s->num_running, s->kv_cache);
}

extern "C" double sf_cost_marginal_gain(const sf_cost_model* m, const sf_instance_state* s, double length) {
  if (!valid_model(m) || !s || s->num_running < 0 || s->num_waiting < 0 || !finite_nonneg(length)) return NAN;
  return gain(m, *s, length);
}

extern "C" double sf_cost_ideal_gain(const sf_cost_model* m, double length) {
  if (!valid_model(m) || !finite_nonneg(length)) return NAN;
  return 1.0 / step_latency(m, 1, m->k5 * length);
}

extern "C" sf_status sf_route(const sf_cost_model* m, double mu, int32_t min_initial_version,
                              sf_instance_state* inst, int32_t num_inst, const sf_trajectory* trajs,
                              int32_t num_trajs, int32_t* target, int32_t* num_routed) {
  if (!valid_model(m) || !std::isfinite(mu) || num_inst < 0 || num_trajs < 0 || !num_routed)
    return SF_ERR_INVALID_ARG;
  if ((num_inst > 0 && !inst) || (num_trajs > 0 && (!trajs || !target))) return SF_ERR_INVALID_ARG;
  for (int32_t i = 0; i < num_inst; ++i)
    if (inst[i].num_running < 0 || inst[i].num_waiting < 0 || !std::isfinite(inst[i].kv_cache))
      return SF_ERR_INVALID_ARG;
  for (int32_t j = 0; j < num_trajs; ++j)
    if (!finite_nonneg(trajs[j].length)) return SF_ERR_INVALID_ARG;

  *num_routed = 0;
  for (int32_t j = 0; j < num_trajs; ++j) target[j] = -1;
  // Queues: by trajectory version, oldest first; initial trajectories last;
  // arrival order inside a queue.
  std::vector<int32_t> order(static_cast<size_t>(num_trajs));
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
    const bool ix = trajs[x].version < 0, iy = trajs[y].version < 0;
    if (ix != iy) return iy;
    return !ix && trajs[x].version < trajs[y].version;
  });
  std::vector<int32_t> cands, versions;
  for (int32_t pos = 0; pos < num_trajs; ++pos) {
    const sf_trajectory& t = trajs[order[size_t(pos)]];
    cands.clear();
    for (int32_t i = 0; i < num_inst; ++i) {
      const bool ok = t.version < 0 ? inst[i].version >= min_initial_version : inst[i].version >= t.version;
      if (ok) cands.push_back(i);
    }
    if (cands.empty()) break;  // this queue stops, and with it every later one
    versions.clear();
    for (int32_t i : cands) versions.push_back(inst[i].version);
    std::sort(versions.begin(), versions.end());
    versions.erase(std::unique(versions.begin(), versions.end()), versions.end());
    const double threshold = mu * sf_cost_ideal_gain(m, t.length);
    int32_t selected = -1;
    for (int32_t v : versions) {
      int32_t best = -1;
      double best_gain = -INFINITY;
      for (int32_t i : cands) {
        if (inst[i].version != v) continue;
        const double g = gain(m, inst[i], t.length);
        if (g > best_gain) {
          best_gain = g;
          best = i;
        }
      }
      if (best_gain >= threshold) {
        selected = best;
        break;
      }
    }
    if (selected < 0) break;  // withheld: routing stops until the load changes
    target[order[size_t(pos)]] = selected;
    inst[selected] = routed(m, inst[selected], t.length);
    ++*num_routed;
  }
  return SF_OK;
}
