// The playout-slack controller (host code): service credit, tiers, dispatch
// order and Bi-Modal Pareto Routing.  Plain computation on caller arrays; see ardit_control.h for the
// rules and their sources in the paper.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "ardit.h"
#include "ardit_control.h"

namespace ardit {
// error reporting shared with the rest of the library (api.cpp)
int set_error(int status, const char* msg);
int host_failure();
}  // namespace ardit

namespace {

using ardit::host_failure;
using ardit::set_error;

bool is_fin(double x) { return std::isfinite(x); }

// quality mode / speed recovery over the frontier (ties as documented)
int bmpr(const ardit_fidelity* c, int nf, const int32_t* f, double floor_q, double budget,
         int32_t* cfg, int32_t* mode) {
  int best = -1;
  for (int k = 0; k < nf; ++k) {
    const int i = f[k];
    if (!(c[i].quality >= floor_q) || !(c[i].latency_ms <= budget)) continue;
    if (best < 0 || c[i].quality > c[best].quality ||
        (c[i].quality == c[best].quality &&
         (c[i].latency_ms < c[best].latency_ms ||
          (c[i].latency_ms == c[best].latency_ms && i < best))))
      best = i;
  }
  if (best >= 0) {
    *cfg = best;
    *mode = ARDIT_BMPR_QUALITY;
    return ARDIT_OK;
  }
  for (int k = 0; k < nf; ++k) {
    const int i = f[k];
    if (!(c[i].quality >= floor_q)) continue;
    if (best < 0 || c[i].latency_ms < c[best].latency_ms ||
        (c[i].latency_ms == c[best].latency_ms &&
         (c[i].quality > c[best].quality || (c[i].quality == c[best].quality && i < best))))
      best = i;
  }
  if (best < 0) return set_error(ARDIT_ECAPACITY, "no frontier point reaches the quality floor");
  *cfg = best;
  *mode = ARDIT_BMPR_SPEED_RECOVERY;
  return ARDIT_OK;
}

int check_frontier(int32_t n_cfgs, const ardit_fidelity* cfgs, int32_t nf, const int32_t* f) {
  if (n_cfgs < 1 || !cfgs) return set_error(ARDIT_EINVAL, "no configurations");
  if (nf < 1 || !f) return set_error(ARDIT_EINVAL, "empty frontier");
  for (int k = 0; k < nf; ++k)
    if (f[k] < 0 || f[k] >= n_cfgs) return set_error(ARDIT_EINVAL, "frontier index out of range");
  for (int i = 0; i < n_cfgs; ++i)
    if (!is_fin(cfgs[i].latency_ms) || !is_fin(cfgs[i].quality))
      return set_error(ARDIT_EINVAL, "non-finite latency or quality");
  return ARDIT_OK;
}

}  // namespace

extern "C" {

int ardit_pareto_frontier(int32_t n, const ardit_fidelity* cfgs, int32_t* frontier,
                          int32_t* n_frontier, double* q_floor) try {
  if (n < 1 || !cfgs || !frontier || !n_frontier || !q_floor)
    return set_error(ARDIT_EINVAL, "pareto_frontier: empty set or NULL pointer");
  for (int i = 0; i < n; ++i)
    if (!is_fin(cfgs[i].latency_ms) || !is_fin(cfgs[i].quality))
      return set_error(ARDIT_EINVAL, "pareto_frontier: non-finite latency or quality");
  // sort by latency ascending, quality descending, index; a point survives
  // when its quality beats every strictly faster point and it ties the best
  // of its own latency
  std::vector<int> ord(n);
  for (int i = 0; i < n; ++i) ord[i] = i;
  std::sort(ord.begin(), ord.end(), [&](int a, int b) {
    if (cfgs[a].latency_ms != cfgs[b].latency_ms) return cfgs[a].latency_ms < cfgs[b].latency_ms;
    if (cfgs[a].quality != cfgs[b].quality) return cfgs[a].quality > cfgs[b].quality;
    return a < b;
  });
  int m = 0;
  double best_faster = -INFINITY;
  for (int s = 0; s < n;) {
    int e = s;
    while (e < n && cfgs[ord[e]].latency_ms == cfgs[ord[s]].latency_ms) ++e;
    const double top = cfgs[ord[s]].quality;   // the group's best (sorted)
    for (int k = s; k < e && cfgs[ord[k]].quality == top; ++k)
      if (top > best_faster) frontier[m++] = ord[k];
    best_faster = std::max(best_faster, top);
    s = e;
  }
  std::vector<double> q(n);
  for (int i = 0; i < n; ++i) q[i] = cfgs[i].quality;
  std::sort(q.begin(), q.end());
  *q_floor = (n % 2) ? q[n / 2] : 0.5 * (q[n / 2 - 1] + q[n / 2]);
  *n_frontier = m;
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_bmpr_select(int32_t n_cfgs, const ardit_fidelity* cfgs, int32_t n_frontier,
                      const int32_t* frontier, double q_floor, double budget_ms, int32_t* cfg,
                      int32_t* mode) try {
  int s = check_frontier(n_cfgs, cfgs, n_frontier, frontier);
  if (s != ARDIT_OK) return s;
  if (!cfg || !mode) return set_error(ARDIT_EINVAL, "bmpr_select: NULL output");
  if (std::isnan(q_floor) || std::isnan(budget_ms))
    return set_error(ARDIT_EINVAL, "bmpr_select: NaN floor or budget");
  int32_t c = 0, md = 0;
  s = bmpr(cfgs, n_frontier, frontier, q_floor, budget_ms, &c, &md);
  if (s != ARDIT_OK) return s;
  *cfg = c;
  *mode = md;
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_control_tick(int32_t n_workers, int32_t n_cfgs, const ardit_fidelity* cfgs,
                       int32_t n_frontier, const int32_t* frontier, double q_floor,
                       int32_t n_streams, const ardit_stream_state* st,
                       ardit_stream_decision* out) try {
  if (n_streams < 0 || (n_streams > 0 && (!st || !out)))
    return set_error(ARDIT_EINVAL, "control_tick: NULL argument");
  int s = check_frontier(n_cfgs, cfgs, n_frontier, frontier);
  if (s != ARDIT_OK) return s;
  const int W = n_workers;
  if (W < 1 || std::isnan(q_floor)) return set_error(ARDIT_EINVAL, "control_tick: malformed parameters");
  for (int i = 0; i < n_streams; ++i) {
    if (st[i].worker < 0 || st[i].worker >= W)
      return set_error(ARDIT_EINVAL, "control_tick: worker out of range");
    if (!is_fin(st[i].slack_ms) || !is_fin(st[i].remaining_ms))
      return set_error(ARDIT_EINVAL, "control_tick: non-finite stream state");
  }
  std::vector<ardit_stream_decision> d(n_streams);
  // 1. fidelity, credit, tier
  for (int i = 0; i < n_streams; ++i) {
    ardit_stream_decision& o = d[i];
    s = bmpr(cfgs, n_frontier, frontier, q_floor, st[i].slack_ms - st[i].remaining_ms, &o.cfg,
             &o.mode);
    if (s != ARDIT_OK) return s;
    const double T = cfgs[o.cfg].latency_ms;
    o.credit_ms = st[i].slack_ms - (st[i].remaining_ms + T);
    o.tier = o.credit_ms < 2.0 * T ? ARDIT_URGENT
             : o.credit_ms > 4.0 * T ? ARDIT_RELAXED : ARDIT_NORMAL;
    o.queue_pos = 0;
  }
  // 2. streams per worker in dispatch order (credit, then index)
  std::vector<std::vector<int>> on(W);
  for (int i = 0; i < n_streams; ++i) on[st[i].worker].push_back(i);
  for (int w = 0; w < W; ++w) {
    std::sort(on[w].begin(), on[w].end(), [&](int a, int b) {
      return d[a].credit_ms != d[b].credit_ms ? d[a].credit_ms < d[b].credit_ms : a < b;
    });
    for (size_t k = 0; k < on[w].size(); ++k) d[on[w][k]].queue_pos = static_cast<int32_t>(k);
  }
  std::copy(d.begin(), d.end(), out);
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

}  // extern "C"
