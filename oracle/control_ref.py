"""Reference of the playout-slack controller -- TEST INFRASTRUCTURE ONLY.

Plain Python definitions of the control plane's decisions that pick each
stream's next configuration and its place in the queue, taken from the paper
in its order: service credit (Section 3.1, its equation), the three urgency
tiers and the credit-ordered dispatch (Section 4.1), the tick's order of
decisions (Appendix C.1), and Bi-Modal Pareto Routing over the profiled
frontier with the median quality as floor (Section 5.2, Appendix A).  Times
are milliseconds in double precision; every decision is an integer or an
order, so the product must match it exactly.

Readings where the paper is silent:
  - the budget B of BMPR is the slack left when the next chunk can start,
    P - R: a configuration with latency <= B keeps the credit >= 0;
  - ties: the frontier keeps points with identical (L, Q) (neither dominates);
    quality mode prefers higher quality, then lower latency, then the lower
    configuration index; speed-recovery prefers lower latency, then higher
    quality, then the lower index; queues order by credit, then stream id.
"""
from __future__ import annotations

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


@dataclass
class Stream:
    worker: int
    slack_ms: float
    remaining_ms: float = 0.0


@dataclass
class Decision:
    cfg: int = -1
    mode: int = QUALITY_MODE
    credit_ms: float = 0.0
    tier: int = NORMAL
    queue_pos: int = 0


def control_tick(n_workers: int, latency, quality, frontier, q_floor: float, streams):
    """One control tick (the appendix's workflow, its first two decisions): per
    stream BMPR, credit and tier under the selected configuration; dispatch
    order per worker.  Returns one Decision per stream."""
    out = []
    for s in streams:
        d = Decision()
        d.cfg, d.mode = bmpr_select(frontier, latency, quality, q_floor,
                                    s.slack_ms - s.remaining_ms)
        T = float(latency[d.cfg])
        d.credit_ms = service_credit(s.slack_ms, s.remaining_ms, T)
        d.tier = tier(d.credit_ms, T)
        out.append(d)
    on = [[i for i in range(len(streams)) if streams[i].worker == w] for w in range(n_workers)]
    # dispatch order: ascending credit, then stream id
    for w in range(n_workers):
        for pos, i in enumerate(sorted(on[w], key=lambda i: (out[i].credit_ms, i))):
            out[i].queue_pos = pos
    return out
