// Out-of-order agent scheduler: the controller of AI Metropolis (§3.1-§3.5,
// Algorithm 3) on the host.
//
// State: every agent's position, completed steps and whether it waits, runs
// (its cluster was handed out) or is done.  Readiness is recomputed from that
// state whenever it changed (an acknowledged cluster) and a cluster is asked
// for, which gives the same clusters as the paper's incremental dependency
// graph (§3.4):
//  - with moves bounded by max_vel, an agent that is not blocked stays so
//    while the agents behind it advance (each advance lowers the blocking
//    distance by max_vel and the distance by at most max_vel);
//  - a waiting cluster never gains members: an agent arriving at its step
//    within the coupling distance was, one step earlier, within the blocking
//    distance of those members, so their cluster was not ready.
// Cost: O(n^2) distance tests per recomputation (about a millisecond at 1000
// agents), far below an LLM call.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <map>
#include <new>
#include <numeric>
#include <unordered_map>
#include <utility>
#include <vector>

#include "../../include/metro_sched.h"
#include "errors.h"

namespace {

constexpr int32_t kWaiting = 0, kRunning = 1, kDone = 2;

}  // namespace

struct metro_sched {
  metro_sched_config cfg{};
  std::vector<int32_t> x, y, step, state;
  struct Cluster {
    int32_t step;
    std::vector<int32_t> members;
  };
  std::unordered_map<int32_t, Cluster> running;  // handed out, not yet acknowledged
  int32_t next_id = 0;
  // ready clusters not handed out yet, keyed (step, lowest member id)
  std::map<std::pair<int32_t, int32_t>, std::vector<int32_t>> ready;
  bool dirty = true;

  // dist(a, b) <= thr in the configured metric; thr >= 0
  bool within(int32_t xa, int32_t ya, int32_t xb, int32_t yb, double thr) const {
    const double dx = std::abs(static_cast<double>(xa) - xb), dy = std::abs(static_cast<double>(ya) - yb);
    if (cfg.metric == METRO_DIST_CHEBYSHEV) return std::max(dx, dy) <= thr;
    return dx * dx + dy * dy <= thr * thr;
  }

  // §3.3: A at step s_A is blocked by B at s_B < s_A when
  // dist(A, B) <= (s_A - s_B + 1) * max_vel + radius_p
  bool blocked(int32_t a) const {
    const int32_t n = cfg.n_agents;
    for (int32_t b = 0; b < n; ++b) {
      if (step[b] >= step[a]) continue;
      const double thr = static_cast<double>(step[a] - step[b] + 1) * cfg.max_vel + cfg.radius_p;
      if (within(x[a], y[a], x[b], y[b], thr)) return true;
    }
    return false;
  }

  void recompute() {
    ready.clear();
    dirty = false;
    const int32_t n = cfg.n_agents;
    if (cfg.sync) {
      // Algorithm 1: one cluster of every agent once all have finished the step
      if (!running.empty()) return;
      std::vector<int32_t> all;
      for (int32_t a = 0; a < n; ++a)
        if (state[a] == kWaiting) all.push_back(a);
      if (!all.empty()) ready.emplace(std::make_pair(step[all[0]], all[0]), std::move(all));
      return;
    }
    // connected components of the coupled relation among waiting agents:
    // same step and dist <= radius_p + max_vel (§3.3)
    std::vector<int32_t> parent(n);
    std::iota(parent.begin(), parent.end(), 0);
    auto root = [&](int32_t a) {
      while (parent[a] != a) a = parent[a] = parent[parent[a]];
      return a;
    };
    const double couple = static_cast<double>(cfg.max_vel) + cfg.radius_p;
    for (int32_t a = 0; a < n; ++a) {
      if (state[a] != kWaiting) continue;
      for (int32_t b = a + 1; b < n; ++b) {
        if (state[b] != kWaiting || step[b] != step[a]) continue;
        if (within(x[a], y[a], x[b], y[b], couple)) {
          const int32_t ra = root(a), rb = root(b);
          if (ra != rb) parent[std::max(ra, rb)] = std::min(ra, rb);
        }
      }
    }
    // a component is ready when none of its members is blocked (§3.4)
    std::map<int32_t, std::vector<int32_t>> comps;
    for (int32_t a = 0; a < n; ++a)
      if (state[a] == kWaiting) comps[root(a)].push_back(a);
    for (auto& kv : comps) {
      bool ok = true;
      for (int32_t a : kv.second)
        if (blocked(a)) {
          ok = false;
          break;
        }
      if (ok) ready.emplace(std::make_pair(step[kv.second[0]], kv.second[0]), std::move(kv.second));
    }
  }
};

extern "C" {

metro_status metro_sched_create(const metro_sched_config* cfg, const int32_t* xy, metro_sched** out) {
  metro::clear_error();
  if (!cfg || !xy || !out) return metro::report(METRO_E_INVAL, "sched: NULL argument");
  if (cfg->n_agents <= 0 || cfg->target_step <= 0 || !(cfg->radius_p >= 0.f) || !(cfg->max_vel >= 0.f) ||
      !std::isfinite(cfg->radius_p) || !std::isfinite(cfg->max_vel) ||
      (cfg->metric != METRO_DIST_CHEBYSHEV && cfg->metric != METRO_DIST_EUCLIDEAN) || (cfg->sync != 0 && cfg->sync != 1))
    return metro::report(METRO_E_INVAL, "sched: bad config");
  metro_sched* s = new (std::nothrow) metro_sched;
  if (!s) return metro::report(METRO_E_NOMEM, "sched: allocation failed");
  s->cfg = *cfg;
  const int32_t n = cfg->n_agents;
  try {
    s->x.resize(n);
    s->y.resize(n);
    s->step.assign(n, 0);
    s->state.assign(n, kWaiting);
  } catch (...) {
    delete s;
    return metro::report(METRO_E_NOMEM, "sched: allocation failed");
  }
  for (int32_t a = 0; a < n; ++a) {
    s->x[a] = xy[2 * a];
    s->y[a] = xy[2 * a + 1];
  }
  *out = s;
  return METRO_OK;
}

void metro_sched_destroy(metro_sched* s) { delete s; }

metro_status metro_sched_next(metro_sched* s, int32_t* cluster, int32_t* step, int32_t* agents, int32_t cap,
                              int32_t* n_out) {
  metro::clear_error();
  if (!s || !cluster || !step || !n_out || (cap > 0 && !agents)) return metro::report(METRO_E_INVAL, "sched: NULL argument");
  *n_out = 0;
  *cluster = -1;
  *step = -1;
  if (s->dirty) s->recompute();
  if (s->ready.empty()) return METRO_OK;
  auto it = s->ready.begin();
  const std::vector<int32_t>& m = it->second;
  if (static_cast<int64_t>(m.size()) > cap)
    return metro::report(METRO_E_CAPACITY, "sched: cluster of %zu agents > cap %d", m.size(), cap);
  const int32_t id = s->next_id++;
  for (size_t j = 0; j < m.size(); ++j) {
    agents[j] = m[j];
    s->state[m[j]] = kRunning;
  }
  *cluster = id;
  *step = it->first.first;
  *n_out = static_cast<int32_t>(m.size());
  s->running.emplace(id, metro_sched::Cluster{it->first.first, m});
  s->ready.erase(it);
  return METRO_OK;
}

metro_status metro_sched_ack(metro_sched* s, int32_t cluster, const int32_t* xy) {
  metro::clear_error();
  if (!s || !xy) return metro::report(METRO_E_INVAL, "sched: NULL argument");
  auto it = s->running.find(cluster);
  if (it == s->running.end()) return metro::report(METRO_E_INVAL, "sched: cluster %d is not running", cluster);
  const std::vector<int32_t>& m = it->second.members;
  for (size_t j = 0; j < m.size(); ++j) {
    const int32_t a = m[j];
    if (!s->within(s->x[a], s->y[a], xy[2 * j], xy[2 * j + 1], s->cfg.max_vel))
      return metro::report(METRO_E_INVAL, "sched: agent %d moves farther than max_vel", a);
  }
  for (size_t j = 0; j < m.size(); ++j) {
    const int32_t a = m[j];
    s->x[a] = xy[2 * j];
    s->y[a] = xy[2 * j + 1];
    s->step[a] += 1;
    s->state[a] = s->step[a] >= s->cfg.target_step ? kDone : kWaiting;
  }
  s->running.erase(it);
  s->dirty = true;
  return METRO_OK;
}

metro_status metro_sched_state(const metro_sched* s, int32_t* steps, int32_t* xy, int32_t* state, int32_t* running,
                               int32_t* done) {
  metro::clear_error();
  if (!s) return metro::report(METRO_E_INVAL, "sched: NULL argument");
  const int32_t n = s->cfg.n_agents;
  bool all_done = true;
  for (int32_t a = 0; a < n; ++a) {
    if (steps) steps[a] = s->step[a];
    if (xy) {
      xy[2 * a] = s->x[a];
      xy[2 * a + 1] = s->y[a];
    }
    if (state) state[a] = s->state[a];
    all_done = all_done && s->state[a] == kDone;
  }
  if (running) *running = static_cast<int32_t>(s->running.size());
  if (done) *done = all_done ? 1 : 0;
  return METRO_OK;
}

}  // extern "C"
