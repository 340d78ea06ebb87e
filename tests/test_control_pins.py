"""CPU pins of the controller oracle (oracle/control_ref.py) against hand-worked
cases of the paper's rules and against independent formulations: the credit
equation (Section 3.1), tier bounds (Section 4.1), the Pareto frontier
(Section 5.2) against a sort-and-sweep construction, the median floor, both
BMPR modes, and a worked control tick (configuration, credit, tier and the
credit-ordered dispatch of Section 4.1)."""
import math

import numpy as np

from oracle import control_ref as K


def test_credit_and_tier_bounds():
    assert K.service_credit(3000.0, 500.0, 800.0) == 1700.0
    T = 250.0
    assert K.tier(2 * T - 1e-9, T) == K.URGENT
    assert K.tier(2 * T, T) == K.NORMAL          # both ends of NORMAL are closed
    assert K.tier(4 * T, T) == K.NORMAL
    assert K.tier(4 * T + 1e-9, T) == K.RELAXED
    assert K.tier(-1.0, T) == K.URGENT


def _sweep_frontier(L, Q):
    """Independent construction: sort by latency ascending and quality
    descending; a point is non-dominated iff its quality beats every strictly
    faster point's and it is not beaten by an equally fast one."""
    n = len(L)
    keep = []
    best_faster = -math.inf          # best quality among strictly faster points
    i = 0
    order = sorted(range(n), key=lambda k: (L[k], -Q[k]))
    while i < n:
        j = i
        while j < n and L[order[j]] == L[order[i]]:
            j += 1
        group = order[i:j]
        top = max(Q[k] for k in group)
        for k in group:
            if Q[k] == top and Q[k] > best_faster:
                keep.append(k)
        best_faster = max(best_faster, top)
        i = j
    return sorted(keep, key=lambda k: (L[k], -Q[k], k))


def test_frontier_worked_example_and_sweep():
    # A(10,5) B(20,7) C(15,4) dominated by A, D(20,6) by B, E = A duplicated, F(30,7) by B
    L = [10, 20, 15, 20, 10, 30]
    Q = [5, 7, 4, 6, 5, 7]
    assert K.pareto_frontier(L, Q) == [0, 4, 1]
    rng = np.random.default_rng(5)
    for _ in range(200):
        n = int(rng.integers(1, 40))
        L = list(rng.integers(1, 12, size=n).astype(float))   # many ties on purpose
        Q = list(rng.integers(1, 8, size=n).astype(float))
        assert K.pareto_frontier(L, Q) == _sweep_frontier(L, Q)


def test_quality_floor_is_the_median():
    assert K.quality_floor([4, 1, 3, 2]) == 2.5
    assert K.quality_floor([5, 1, 3]) == 3
    rng = np.random.default_rng(6)
    q = rng.standard_normal(90)
    assert K.quality_floor(q) == float(np.median(q))


def test_bmpr_modes():
    L = [50.0, 80.0, 120.0, 200.0]
    Q = [70.0, 75.0, 80.0, 82.0]
    F = K.pareto_frontier(L, Q)
    floor = 74.0
    assert K.bmpr_select(F, L, Q, floor, 130.0) == (2, K.QUALITY_MODE)
    assert K.bmpr_select(F, L, Q, floor, 1000.0) == (3, K.QUALITY_MODE)
    assert K.bmpr_select(F, L, Q, floor, 80.0) == (1, K.QUALITY_MODE)
    # nothing within 60 ms clears the floor: the fastest point above it, not the 50 ms one
    assert K.bmpr_select(F, L, Q, floor, 60.0) == (1, K.SPEED_RECOVERY)
    assert K.bmpr_select(F, L, Q, floor, -5.0) == (1, K.SPEED_RECOVERY)
    # never below the floor, whatever the budget
    for b in np.linspace(-100, 300, 41):
        c, _ = K.bmpr_select(F, L, Q, floor, float(b))
        assert Q[c] >= floor


def test_worked_tick():
    """Three configurations: A (100 ms, Q 80), B (200 ms, Q 90), C (50 ms, Q 60);
    floor = median 80.  Stream budgets P - R pick B when >= 200, A when in
    [100, 200), and speed recovery (A, the fastest at the floor) below 100;
    credit and tier follow, and each worker's queue runs by credit."""
    lat, qual = [100.0, 200.0, 50.0], [80.0, 90.0, 60.0]
    F = K.pareto_frontier(lat, qual)
    assert F == [2, 0, 1] and K.quality_floor(qual) == 80.0
    st = [K.Stream(0, 1500.0), K.Stream(0, 180.0, 30.0), K.Stream(1, 90.0),
          K.Stream(0, 700.0, 100.0), K.Stream(1, 450.0)]
    d = K.control_tick(2, lat, qual, F, 80.0, st)
    assert [x.cfg for x in d] == [1, 0, 0, 1, 1]
    assert [x.mode for x in d] == [K.QUALITY_MODE, K.QUALITY_MODE, K.SPEED_RECOVERY,
                                   K.QUALITY_MODE, K.QUALITY_MODE]
    assert [x.credit_ms for x in d] == [1300.0, 50.0, -10.0, 400.0, 250.0]
    assert [x.tier for x in d] == [K.RELAXED, K.URGENT, K.URGENT, K.NORMAL, K.URGENT]
    # worker 0: credits 1300, 50, 400 -> order 1, 3, 0; worker 1: -10, 250 -> 2, 4
    assert [x.queue_pos for x in d] == [2, 0, 0, 1, 1]
    # equal credits keep the stream order
    d = K.control_tick(1, lat, qual, F, 80.0, [K.Stream(0, 300.0), K.Stream(0, 300.0)])
    assert [x.queue_pos for x in d] == [0, 1]
