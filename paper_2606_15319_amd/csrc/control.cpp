// The playout-slack controller (host code): service credit, tiers, dispatch
// order, re-homing, elastic-SP donors, eviction, admission and Bi-Modal Pareto
// Routing.  Plain computation on caller arrays; see ardit_control.h for the
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

int ardit_control_tick(const ardit_ctl_params* p, int32_t n_cfgs, const ardit_fidelity* cfgs,
                       int32_t n_frontier, const int32_t* frontier, double q_floor,
                       int32_t n_streams, const ardit_stream_state* st,
                       ardit_stream_decision* out) try {
  if (!p || !st || !out || n_streams < 0) return set_error(ARDIT_EINVAL, "control_tick: NULL argument");
  int s = check_frontier(n_cfgs, cfgs, n_frontier, frontier);
  if (s != ARDIT_OK) return s;
  const int W = p->n_workers;
  if (W < 1 || p->gpus_per_node < 1 || p->cap_send < 0 || p->cap_recv < 0 ||
      !is_fin(p->now_ms) || std::isnan(p->cooldown_ms) || std::isnan(q_floor))
    return set_error(ARDIT_EINVAL, "control_tick: malformed parameters");
  for (int i = 0; i < n_streams; ++i) {
    if (st[i].worker < 0 || st[i].worker >= W || st[i].sp_donor < -1 || st[i].sp_donor >= W)
      return set_error(ARDIT_EINVAL, "control_tick: worker or donor out of range");
    if (!is_fin(st[i].slack_ms) || !is_fin(st[i].remaining_ms) ||
        std::isnan(st[i].cooldown_until_ms))
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
    o.rehome_to = -1;
    o.sp_donor = -1;
    o.cooldown_until_ms = st[i].cooldown_until_ms;
  }
  // streams per worker, in dispatch order (credit, then index)
  std::vector<std::vector<int>> on(W);
  for (int i = 0; i < n_streams; ++i) on[st[i].worker].push_back(i);
  for (int w = 0; w < W; ++w) {
    std::sort(on[w].begin(), on[w].end(), [&](int a, int b) {
      return d[a].credit_ms != d[b].credit_ms ? d[a].credit_ms < d[b].credit_ms : a < b;
    });
    for (size_t k = 0; k < on[w].size(); ++k) d[on[w][k]].queue_pos = static_cast<int32_t>(k);
  }
  // 3. re-homing
  std::vector<int> n_urgent(W, 0);
  std::vector<char> relaxed(W, 1);
  for (int i = 0; i < n_streams; ++i) {
    if (d[i].tier == ARDIT_URGENT) ++n_urgent[st[i].worker];
    if (d[i].tier != ARDIT_RELAXED) relaxed[st[i].worker] = 0;
  }
  std::vector<int> senders, receivers;
  for (int w = 0; w < W; ++w) {
    if (n_urgent[w] >= 2) senders.push_back(w);
    if (relaxed[w]) receivers.push_back(w);
  }
  std::sort(senders.begin(), senders.end(), [&](int a, int b) {
    return n_urgent[a] != n_urgent[b] ? n_urgent[a] > n_urgent[b] : a < b;
  });
  const int g = p->gpus_per_node;
  std::vector<int> sent(W, 0), recv(W, 0);
  std::vector<char> moved(n_streams, 0);
  for (int src : senders) {
    std::vector<int> dsts = receivers;
    std::stable_sort(dsts.begin(), dsts.end(), [&](int a, int b) {
      return (a / g != src / g) < (b / g != src / g);
    });
    for (int dst : dsts) {
      if (sent[src] >= p->cap_send || recv[dst] >= p->cap_recv) continue;
      int pick = -1;
      for (int i : on[src]) {   // dispatch order: the first eligible has the lowest credit
        if (d[i].tier == ARDIT_URGENT && !moved[i] && st[i].cooldown_until_ms <= p->now_ms &&
            st[i].sp_donor < 0) {
          pick = i;
          break;
        }
      }
      if (pick < 0) continue;
      d[pick].rehome_to = dst;
      d[pick].cooldown_until_ms = p->now_ms + p->cooldown_ms;
      moved[pick] = 1;
      ++sent[src];
      ++recv[dst];
    }
  }
  // 4. elastic SP
  std::vector<char> busy(W, 0);
  for (int i = 0; i < n_streams; ++i) {
    if (st[i].sp_donor < 0) continue;
    if (d[i].credit_ms >= 2.0 * cfgs[d[i].cfg].latency_ms) continue;   // recovered: released
    d[i].sp_donor = st[i].sp_donor;
    busy[st[i].sp_donor] = 1;
  }
  std::vector<double> wcredit(W, INFINITY);
  for (int i = 0; i < n_streams; ++i)
    wcredit[st[i].worker] = std::min(wcredit[st[i].worker], d[i].credit_ms);
  std::vector<int> need;
  for (int i = 0; i < n_streams; ++i)
    if (d[i].credit_ms < 0.0 && d[i].sp_donor < 0 && d[i].rehome_to < 0) need.push_back(i);
  std::sort(need.begin(), need.end(), [&](int a, int b) {
    return d[a].credit_ms != d[b].credit_ms ? d[a].credit_ms < d[b].credit_ms : a < b;
  });
  for (int i : need) {
    const int w = st[i].worker;
    int donor = -1;
    for (int c = 0; c < W; ++c) {
      if (c == w || busy[c] || !relaxed[c] || recv[c] != 0 || c / g != w / g) continue;
      if (donor < 0 || wcredit[c] > wcredit[donor]) donor = c;   // ties keep the lower id
    }
    if (donor < 0) continue;
    d[i].sp_donor = donor;
    busy[donor] = 1;
  }
  std::copy(d.begin(), d.end(), out);
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_evict_for(int32_t n, const double* credits, const int32_t* resident_pages,
                    int32_t requester, int64_t free_pages, int64_t need_pages, int32_t* evict,
                    int32_t* n_evict) try {
  if (n < 0 || (n > 0 && (!credits || !resident_pages)) || !evict || !n_evict)
    return set_error(ARDIT_EINVAL, "evict_for: NULL argument");
  for (int i = 0; i < n; ++i)
    if (std::isnan(credits[i]) || resident_pages[i] < 0)
      return set_error(ARDIT_EINVAL, "evict_for: NaN credit or negative page count");
  std::vector<int> ord;
  for (int i = 0; i < n; ++i)
    if (i != requester && resident_pages[i] > 0) ord.push_back(i);
  std::sort(ord.begin(), ord.end(), [&](int a, int b) {
    return credits[a] != credits[b] ? credits[a] > credits[b] : a > b;
  });
  int m = 0;
  int64_t free_now = free_pages;
  std::vector<int32_t> chosen;
  for (int i : ord) {
    if (free_now >= need_pages) break;
    chosen.push_back(i);
    free_now += resident_pages[i];
    ++m;
  }
  if (free_now < need_pages)
    return set_error(ARDIT_ECAPACITY, "evict_for: the pool cannot hold the requested pages");
  std::copy(chosen.begin(), chosen.end(), evict);
  *n_evict = m;
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_admit(int32_t n_workers, const int32_t* streams_per_worker, double first_chunk_ms,
                int32_t* home, double* slack_ms) try {
  if (n_workers < 1 || !streams_per_worker || !home || !slack_ms || !is_fin(first_chunk_ms))
    return set_error(ARDIT_EINVAL, "admit: malformed argument");
  int best = 0;
  for (int w = 1; w < n_workers; ++w)
    if (streams_per_worker[w] < streams_per_worker[best]) best = w;
  *home = best;
  *slack_ms = 4.0 * first_chunk_ms;
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

}  // extern "C"
