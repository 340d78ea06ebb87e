"""CPU pins of the controller oracle (oracle/control_ref.py) against hand-worked
cases of the paper's rules and against independent formulations: the credit
equation (Section 3.1), tier bounds (Section 4.1), the Pareto frontier
(Section 5.2) against a sort-and-sweep construction, the median floor, both
BMPR modes, the re-homing example of Section 4.2 (two RELAXED workers, one
with queued URGENT streams) with its caps, cooldown and node preference
(Appendix C.2), elastic-SP donor choice and release (Section 4.3, Appendix
C.3), credit-aware eviction (Section 4.1) and admission (Section 3.3)."""
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


def _tick(streams, latency, quality, **kw):
    F = K.pareto_frontier(latency, quality)
    return K.control_tick(K.Params(**kw), latency, quality, F, K.quality_floor(quality), streams)


def test_rehoming_example_and_caps():
    # one configuration of 100 ms: tiers by slack alone (URGENT < 300, RELAXED > 500)
    lat, qual = [100.0], [1.0]
    st = [K.Stream(0, 900.0), K.Stream(1, 800.0),                    # W0, W1: RELAXED
          K.Stream(2, 150.0), K.Stream(2, 120.0), K.Stream(2, 250.0),  # W2: three URGENT
          K.Stream(3, 1000.0)]                                        # W3: RELAXED
    d = _tick(st, lat, qual, n_workers=4, now_ms=5000.0)
    assert [x.tier for x in d] == [K.RELAXED, K.RELAXED, K.URGENT, K.URGENT, K.URGENT, K.RELAXED]
    # W2 sends its two lowest-credit URGENT streams (cap 2), one per receiver (cap 1)
    assert [x.rehome_to for x in d] == [-1, -1, 1, 0, -1, -1]
    assert d[3].cooldown_until_ms == 65000.0 and d[2].cooldown_until_ms == 65000.0
    # dispatch order on W2: lowest credit first
    assert [d[i].queue_pos for i in (2, 3, 4)] == [1, 0, 2]
    # the lowest-credit stream in cooldown stays; the next one goes
    st[3].cooldown_until_ms = 30000.0
    d = _tick(st, lat, qual, n_workers=4, now_ms=5000.0)
    assert [x.rehome_to for x in d] == [-1, -1, 0, -1, 1, -1]
    # receivers on the sender's node come first: sender W9 (node 1) picks W8, then W0
    st = [K.Stream(0, 900.0), K.Stream(8, 900.0), K.Stream(9, 100.0), K.Stream(9, 110.0),
          K.Stream(9, 120.0)]
    d = _tick(st, lat, qual, n_workers=10, gpus_per_node=8)
    assert [x.rehome_to for x in d][2:] == [8, 0, -1]
    # one URGENT stream alone is not congestion: nothing moves
    d = _tick([K.Stream(0, 100.0), K.Stream(1, 900.0)], lat, qual, n_workers=2)
    assert [x.rehome_to for x in d] == [-1, -1]


def test_elastic_sp_donor_and_release():
    lat, qual = [100.0], [1.0]
    # stream 0 on W0 will miss its window (C = 50 - 100 < 0); W1 and W2 are
    # RELAXED on the same node, W2 idle (+inf credit), W9 RELAXED on another node
    st = [K.Stream(0, 50.0), K.Stream(1, 600.0), K.Stream(9, 5000.0)]
    d = _tick(st, lat, qual, n_workers=10)
    assert d[0].sp_donor == 2 and d[0].tier == K.URGENT
    # without same-node RELAXED workers there is no donor
    st2 = [K.Stream(0, 50.0), K.Stream(1, 50.0), K.Stream(9, 5000.0)]
    d = _tick(st2, lat, qual, n_workers=10, gpus_per_node=2)
    assert d[0].sp_donor == -1 and d[1].sp_donor == -1
    # a donor is kept while the stream stays below NORMAL and released at C >= 2T
    st[0].sp_donor = 2
    st[0].slack_ms = 250.0                   # C = 150 < 200: keep
    assert _tick(st, lat, qual, n_workers=10)[0].sp_donor == 2
    st[0].slack_ms = 300.0                   # C = 200 = 2T: NORMAL, release
    assert _tick(st, lat, qual, n_workers=10)[0].sp_donor == -1


def test_credit_aware_eviction():
    credits = [500.0, -20.0, 900.0, 300.0]
    pages = [6, 6, 6, 6]
    # stream 1 (the most urgent) needs 9 pages with 2 free: evict 2 (900), then 0 (500)
    assert K.evict_for(credits, pages, 1, 2, 9) == [2, 0]
    assert K.evict_for(credits, pages, 1, 9, 9) == []
    assert K.evict_for(credits, pages, 1, 0, 40) is None
    # ties go to the later stream
    assert K.evict_for([1.0, 1.0, 0.0], [3, 3, 3], 2, 0, 3) == [1]


def test_admission():
    assert K.choose_home([3, 1, 1, 2]) == 1
    assert K.initial_slack(250.0) == 1000.0
