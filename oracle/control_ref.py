"""Reference of the playout-slack controller -- TEST INFRASTRUCTURE ONLY.

Plain Python definitions of the control plane's decisions, taken from the
paper in its order: service credit (Section 3.1, its equation), the three
urgency tiers and the dispatch order (Section 4.1), credit-aware eviction
(Section 4.1), bipartite re-homing planning (Section 4.2 and its algorithm;
caps, cooldown and node preference from Appendix C.2), the elastic-SP donor
choice and release (Section 4.3, Appendix C.3), admission (Section 3.3), the
tick's order of decisions (Appendix C.1), and
Bi-Modal Pareto Routing over the profiled frontier with the median quality
as floor (Section 5.2, Appendix A).  Times are milliseconds in double
precision; every decision is an integer or an order, so the product must
match it exactly.

Readings where the paper is silent:
  - the budget B of BMPR is the slack left when the next chunk can start,
    P - R: a configuration with latency <= B keeps the credit >= 0;
  - ties: the frontier keeps points with identical (L, Q) (neither dominates);
    quality mode prefers higher quality, then lower latency, then the lower
    configuration index; speed-recovery prefers lower latency, then higher
    quality, then the lower index; queues order by credit, then stream id;
  - a worker is a re-homing sender when it holds at least two URGENT streams
    (an urgent stream is queued behind another), senders go by URGENT count
    (descending) then id; receivers are workers with no URGENT or NORMAL
    stream (idle workers included), same node first, then by id; a stream
    already in an SP2 group or in cooldown is not moved;
  - a worker's credit (donor choice) is the lowest credit of its streams, +inf
    when idle; streams with negative credit get donors in ascending credit
    order, one donor per stream, a donor lends to one stream, never to a
    stream on itself, and a re-homing receiver of the same tick is not a
    donor; a donor is released when its stream's credit reaches the NORMAL
    tier (C >= 2T);
  - eviction frees the highest-credit resident streams other than the
    requester, one at a time (ties to the higher stream id, the later
    admitted), until the requester's pages fit.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

URGENT, NORMAL, RELAXED = 0, 1, 2
QUALITY_MODE, SPEED_RECOVERY = 0, 1


def service_credit(slack_ms: float, remaining_ms: float, next_chunk_ms: float) -> float:
    """C = P - (R + T)."""
    return slack_ms - (remaining_ms + next_chunk_ms)


def tier(credit: float, next_chunk_ms: float) -> int:
    """URGENT below 2T, RELAXED above 4T, NORMAL in between (both ends)."""
    if credit < 2.0 * next_chunk_ms:
        return URGENT
    if credit > 4.0 * next_chunk_ms:
        return RELAXED
    return NORMAL


def dominates(a, b) -> bool:
    """a = (L, Q) dominates b: no slower, no worse, strictly better in one."""
    return a[0] <= b[0] and a[1] >= b[1] and (a[0] < b[0] or a[1] > b[1])


def pareto_frontier(latency, quality):
    """Indices of the non-dominated configurations, by latency ascending (then
    quality descending, then index)."""
    n = len(latency)
    pts = [(float(latency[i]), float(quality[i])) for i in range(n)]
    keep = [i for i in range(n) if not any(dominates(pts[j], pts[i]) for j in range(n))]
    return sorted(keep, key=lambda i: (pts[i][0], -pts[i][1], i))


def quality_floor(quality) -> float:
    """Median quality over all candidates (mean of the middle two for an even count)."""
    q = sorted(float(v) for v in quality)
    n = len(q)
    return q[n // 2] if n % 2 else 0.5 * (q[n // 2 - 1] + q[n // 2])


def bmpr_select(frontier, latency, quality, q_floor: float, budget_ms: float):
    """(configuration index, mode).  Quality mode: the highest-quality frontier
    point with L <= B and Q >= floor; else speed recovery: the fastest
    frontier point with Q >= floor."""
    ok = [i for i in frontier if quality[i] >= q_floor]
    fit = [i for i in ok if latency[i] <= budget_ms]
    if fit:
        return min(fit, key=lambda i: (-quality[i], latency[i], i)), QUALITY_MODE
    return min(ok, key=lambda i: (latency[i], -quality[i], i)), SPEED_RECOVERY


def choose_home(streams_per_worker) -> int:
    """Admission: the worker with the fewest streams (lowest id on ties)."""
    return min(range(len(streams_per_worker)), key=lambda w: (streams_per_worker[w], w))


def initial_slack(first_chunk_ms: float) -> float:
    """Admission: the TTFC budget, 4x the estimated first-chunk time."""
    return 4.0 * first_chunk_ms


@dataclass
class Stream:
    worker: int
    slack_ms: float
    remaining_ms: float = 0.0
    cooldown_until_ms: float = -math.inf
    sp_donor: int = -1


@dataclass
class Params:
    n_workers: int
    gpus_per_node: int = 8
    cap_send: int = 2
    cap_recv: int = 1
    cooldown_ms: float = 60000.0
    now_ms: float = 0.0


@dataclass
class Decision:
    cfg: int = -1
    mode: int = QUALITY_MODE
    credit_ms: float = 0.0
    tier: int = NORMAL
    queue_pos: int = 0
    rehome_to: int = -1
    sp_donor: int = -1
    cooldown_until_ms: float = -math.inf


def control_tick(p: Params, latency, quality, frontier, q_floor: float, streams):
    """One control tick (the appendix's workflow): per stream BMPR, credit and
    tier under the selected configuration; dispatch order per worker;
    re-homing plan; elastic-SP donors.  Returns one Decision per stream."""
    out = []
    for s in streams:
        d = Decision()
        d.cfg, d.mode = bmpr_select(frontier, latency, quality, q_floor,
                                    s.slack_ms - s.remaining_ms)
        T = float(latency[d.cfg])
        d.credit_ms = service_credit(s.slack_ms, s.remaining_ms, T)
        d.tier = tier(d.credit_ms, T)
        d.cooldown_until_ms = s.cooldown_until_ms
        out.append(d)
    W = p.n_workers
    on = [[i for i in range(len(streams)) if streams[i].worker == w] for w in range(W)]
    # dispatch order: ascending credit, then stream id
    for w in range(W):
        for pos, i in enumerate(sorted(on[w], key=lambda i: (out[i].credit_ms, i))):
            out[i].queue_pos = pos
    # re-homing
    n_urgent = [sum(1 for i in on[w] if out[i].tier == URGENT) for w in range(W)]
    senders = sorted([w for w in range(W) if n_urgent[w] >= 2], key=lambda w: (-n_urgent[w], w))
    receivers = [w for w in range(W) if all(out[i].tier == RELAXED for i in on[w])]
    sent = [0] * W
    recv = [0] * W
    moved = set()
    node = lambda w: w // p.gpus_per_node   # noqa: E731
    for src in senders:
        for dst in sorted(receivers, key=lambda w: (node(w) != node(src), w)):
            if sent[src] < p.cap_send and recv[dst] < p.cap_recv:
                cand = [i for i in on[src] if out[i].tier == URGENT and i not in moved
                        and streams[i].cooldown_until_ms <= p.now_ms and streams[i].sp_donor < 0]
                if not cand:
                    continue
                s = min(cand, key=lambda i: (out[i].credit_ms, i))
                out[s].rehome_to = dst
                out[s].cooldown_until_ms = p.now_ms + p.cooldown_ms
                moved.add(s)
                sent[src] += 1
                recv[dst] += 1
    # elastic SP: keep or release the current donors, then lend new ones
    busy = set()
    for i, s in enumerate(streams):
        if s.sp_donor >= 0:
            if out[i].credit_ms >= 2.0 * float(latency[out[i].cfg]):
                out[i].sp_donor = -1            # recovered to NORMAL: release
            else:
                out[i].sp_donor = s.sp_donor
                busy.add(s.sp_donor)
    wcredit = [min((out[i].credit_ms for i in on[w]), default=math.inf) for w in range(W)]
    relaxed = [w for w in range(W) if all(out[i].tier == RELAXED for i in on[w])
               and recv[w] == 0]
    need = sorted([i for i in range(len(streams)) if out[i].credit_ms < 0.0
                   and out[i].sp_donor < 0 and out[i].rehome_to < 0],
                  key=lambda i: (out[i].credit_ms, i))
    for i in need:
        w = streams[i].worker
        cands = [d for d in relaxed if d != w and d not in busy and node(d) == node(w)]
        if not cands:
            continue
        donor = max(cands, key=lambda d: (wcredit[d], -d))
        out[i].sp_donor = donor
        busy.add(donor)
    return out


def evict_for(credits, resident_pages, requester: int, free_pages: int, need_pages: int):
    """Streams to evict (in order) so that need_pages fit: the highest-credit
    residents other than the requester first (ties to the higher id).  Returns
    None when even evicting every other resident leaves too few pages."""
    order = sorted([i for i in range(len(credits)) if i != requester and resident_pages[i] > 0],
                   key=lambda i: (-credits[i], -i))
    out = []
    for i in order:
        if free_pages >= need_pages:
            break
        out.append(i)
        free_pages += resident_pages[i]
    return out if free_pages >= need_pages else None
