"""The controller in libardit (include/ardit_control.h, host code, no GPU)
against the controller oracle, decision for decision, on seeded random
cluster states: frontier and floor, BMPR choices, whole control ticks
(configuration, credit, tier, dispatch order); plus the host-side
rejections."""
import math

import numpy as np
import pytest

from oracle import control_ref as K

A = pytest.importorskip("paper_2606_15319_amd.ardit",
                        reason="libardit.so not built (python -m paper_2606_15319_amd.build)")


def _space(rng, n, tie_heavy):
    """n configurations of the paper's knob space with random (L, Q)."""
    cfgs = []
    for i in range(n):
        S = int(rng.choice([2, 3, 4]))
        rho = float(rng.choice([0.0, 0.6, 0.7, 0.8, 0.9]))
        W = int(rng.choice([1, 3, 7]))
        Q = int(rng.integers(0, 2))
        if tie_heavy:
            lat = float(rng.integers(5, 15)) * 20.0
            qual = float(rng.integers(70, 80))
        else:
            lat = float(rng.uniform(50, 300))
            qual = float(rng.uniform(70, 85))
        cfgs.append((S, rho, W, Q, lat, qual))
    return cfgs


@pytest.mark.parametrize("seed", range(6))
def test_frontier_floor_and_bmpr_match_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    for trial in range(30):
        cfgs = _space(rng, int(rng.integers(1, 91)), tie_heavy=trial % 2 == 0)
        L = [c[4] for c in cfgs]
        Q = [c[5] for c in cfgs]
        f, fl = A.ardit_pareto_frontier(cfgs)
        assert f == K.pareto_frontier(L, Q)
        assert fl == K.quality_floor(Q)
        for b in list(rng.uniform(-50, 400, size=8)) + L[:4]:
            assert A.ardit_bmpr_select(cfgs, f, fl, b) == K.bmpr_select(f, L, Q, fl, b)


def _cluster(rng, n_workers, n_streams):
    streams = []
    for _ in range(n_streams):
        w = int(rng.integers(0, n_workers))
        slack = float(rng.choice([rng.uniform(-400, 3500), rng.integers(-4, 30) * 50.0]))
        rem = float(rng.choice([0.0, rng.uniform(0, 400)]))
        streams.append((w, slack, rem))
    return streams


@pytest.mark.parametrize("seed", range(8))
def test_control_tick_matches_oracle(seed):
    rng = np.random.default_rng(200 + seed)
    for trial in range(25):
        cfgs = _space(rng, int(rng.integers(1, 91)), tie_heavy=trial % 3 == 0)
        L = [c[4] for c in cfgs]
        Q = [c[5] for c in cfgs]
        F = K.pareto_frontier(L, Q)
        fl = K.quality_floor(Q)
        W = int(rng.integers(1, 20))
        streams = _cluster(rng, W, int(rng.integers(0, 60)))
        got = A.ardit_control_tick(W, cfgs, F, fl, streams)
        ref = K.control_tick(W, L, Q, F, fl, [K.Stream(*s) for s in streams])
        for i, (x, r) in enumerate(zip(got, ref)):
            assert (x.cfg, x.mode, x.tier, x.queue_pos) == (r.cfg, r.mode, r.tier, r.queue_pos), \
                (trial, i)
            assert x.credit_ms == r.credit_ms


def _status(fn, *a):
    with pytest.raises(A.ArditError) as e:
        fn(*a)
    return e.value.status


def test_controller_rejections():
    cfgs = [(4, 0.0, 7, 0, 200.0, 80.0), (2, 0.9, 1, 1, 60.0, 70.0)]
    f, fl = A.ardit_pareto_frontier(cfgs)
    assert _status(A.ardit_pareto_frontier, []) == -1
    assert _status(A.ardit_pareto_frontier, [(4, 0.0, 7, 0, float("nan"), 1.0)]) == -1
    assert _status(A.ardit_bmpr_select, cfgs, [], fl, 100.0) == -1
    assert _status(A.ardit_bmpr_select, cfgs, [5], fl, 100.0) == -1
    # a floor above every frontier point: nothing to route to
    assert _status(A.ardit_bmpr_select, cfgs, f, 99.0, 100.0) == -3
    assert _status(A.ardit_control_tick, 2, cfgs, f, fl, [(2, 100.0, 0.0)]) == -1
    assert _status(A.ardit_control_tick, 2, cfgs, f, fl, [(-1, 100.0, 0.0)]) == -1
    assert _status(A.ardit_control_tick, 2, cfgs, f, fl, [(0, math.inf, 0.0)]) == -1
    assert _status(A.ardit_control_tick, 2, cfgs, f, fl, [(0, 100.0, math.nan)]) == -1
    assert _status(A.ardit_control_tick, 0, cfgs, f, fl, []) == -1
    assert A.ardit_control_tick(2, cfgs, f, fl, []) == []


def test_profiler_space_is_the_papers():
    """The profiler enumerates the 90 configurations of the paper's knob
    product (golden settings, Appendix A), the reference first, with S
    timesteps spaced evenly from 1000."""
    import itertools
    import json
    import os
    from paper_2606_15319_amd import profiler as P
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_settings.json")))
    space = list(itertools.product(P.STEPS, P.SPARSITY, P.WINDOWS, P.QUANTS))
    assert len(space) == g["n_fidelity_configs"] == 90
    assert list(P.STEPS) == g["denoise_steps"] and list(P.SPARSITY) == g["sparsity"]
    assert list(P.WINDOWS) == g["kv_window_chunks"] and len(P.QUANTS) == len(g["quant_modes"])
    top = g["top_config"]
    assert P.REFERENCE == (top[0], top[1], top[2], g["quant_modes"].index(top[3]))
    assert P.timesteps(4) == [1000.0, 750.0, 500.0, 250.0] and P.timesteps(2) == [1000.0, 500.0]


def test_committed_profile_frontier_is_consistent():
    """The MI355X latency table under profiles/ covers the 90 configurations
    and its starred rows are exactly the frontier ardit_pareto_frontier
    builds from it (and the oracle's definition agrees)."""
    import itertools
    import os
    from paper_2606_15319_amd import profiler as P
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles",
                        "fidelity_block13b_latency.md")
    rows = P.read_profile(path)
    assert sorted((r[0], r[1], r[2], r[3]) for r in rows) == \
        sorted(itertools.product(P.STEPS, P.SPARSITY, P.WINDOWS, P.QUANTS))
    starred = []
    for line in open(path):
        if line.startswith("| ") and line.rstrip().endswith("| * |"):
            starred.append(line)
    f, fl = A.ardit_pareto_frontier(rows)
    assert len(f) == len(starred)
    assert f == K.pareto_frontier([r[4] for r in rows], [r[5] for r in rows])
    assert fl == K.quality_floor([r[5] for r in rows])
    # every starred row is a frontier row
    on = {(rows[i][0], rows[i][1], rows[i][2], rows[i][3]) for i in f}
    for line in starred:
        c = [x.strip() for x in line.strip().strip("|").split("|")]
        assert (int(c[0]), float(c[1]), int(c[2]), int(c[3] == "FP8")) in on
