"""Pins of the time-interval policy oracle (Sec. IV-A policy form, Alg. 1 interval lookup and idle
energy), on the CPU: hand-worked runs, the reduction to the per-pack evaluation, and an
independent recursive evaluation."""
import functools
import math

import numpy as np
import pytest

import oracle
import pins
from oracle import intervals
from paper_2607_12324_amd import synth


def golden_intervals():
    return pins.load_golden("handworked_intervals.json")


def test_handworked_intervals():
    d = golden_intervals()
    g = pins.graph_from_golden(pins.load_golden())
    for case in d["cases"]:
        T, E = intervals.eval_intervals(g, case["change_points"], [case["levels"]], d["idle_power"])
        if case["makespan"] is None:
            assert np.isnan(T[0]) and np.isnan(E[0]), case
        else:
            assert T[0] == case["makespan"] and E[0] == case["energy"], (case, T[0], E[0])


def recursive_eval(g, pts, row, idle):
    """The same quantities by memoised recursion over predecessors (no topological sort): a
    node's start is the largest finish among its predecessors, its level that of the interval
    holding the start."""
    preds = [[] for _ in range(g.num_nodes)]
    for s, t in zip(g.edge_src.tolist(), g.edge_dst.tolist()):
        preds[t].append(s)

    @functools.lru_cache(maxsize=None)
    def finish(v):
        start = max([finish(k)[0] for k in preds[v]] + [0.0])
        p = int(g.node_pack[v])
        if p < 0:
            return start + float(g.node_duration[v]), 0.0
        i = sum(1 for x in pts if x <= start)
        return start + float(g.pack_time[p, row[i]]), float(g.pack_energy[p, row[i]])

    T = max(finish(v)[0] for v in range(g.num_nodes))
    active = sum(finish(v)[1] for v in range(g.num_nodes))
    bounds = [0.0] + list(pts) + [math.inf]
    idle_e = sum(idle[row[i]] * max(0.0, min(T, bounds[i + 1]) - bounds[i]) for i in range(len(pts) + 1))
    return T, active + idle_e


@pytest.mark.parametrize("seed", range(4))
def test_intervals_match_recursive_definition(seed):
    rng = np.random.default_rng(300 + seed)
    for i in range(6):
        g = synth.random_dag(rng, int(rng.integers(2, 40)), float(rng.uniform(0.05, 0.3)), 0.7,
                             int(rng.integers(2, 6)))
        T0 = float(oracle.eval_batch(g, np.full((1, g.num_packs), g.num_levels - 1, np.uint8))[0][0])
        K = int(rng.integers(1, 7))
        pts = np.sort(rng.choice(np.arange(1, max(2, int(T0 * 16))), size=K - 1, replace=False)) / 16.0
        pts = [float(x) for x in pts]
        idle = [float(x) for x in np.round(rng.uniform(0, 1, g.num_levels) * 64) / 64]
        rows = rng.integers(0, g.num_levels, size=(5, K)).astype(np.uint8)
        T, E = intervals.eval_intervals(g, pts, rows, idle)
        for c in range(len(rows)):
            Tr, Er = recursive_eval(g, pts, [int(x) for x in rows[c]], idle)
            assert T[c] == Tr, (seed, i, c)
            assert abs(E[c] - Er) <= 1e-12 * max(1.0, abs(Er)), (seed, i, c)


@pytest.mark.parametrize("seed", range(3))
def test_one_interval_is_the_per_pack_evaluation(seed):
    """One interval (no change point) and idle power = static_power at every level: every pack
    runs at the row's one level and the idle term is static_power * makespan, so the result is
    the per-pack evaluation with that level everywhere; change points past every start leave
    the packs at the first interval's level and charge that level's idle power."""
    rng = np.random.default_rng(400 + seed)
    g = synth.random_dag(rng, 60, 0.08, 0.7, 5)
    P, F = g.num_packs, g.num_levels
    rows1 = np.arange(F, dtype=np.uint8)[:, None]
    T, E = intervals.eval_intervals(g, [], rows1, [g.static_power] * F)
    To, Eo = oracle.eval_batch(g, np.repeat(rows1, P, axis=1))
    assert np.array_equal(T, To)
    assert np.allclose(E, Eo, rtol=1e-12, atol=0)
    Tslow = float(oracle.eval_batch(g, np.zeros((1, P), np.uint8))[0][0])
    far = [Tslow + 1.0, Tslow + 2.0]
    idle = [0.125 * (f + 1) for f in range(F)]
    rows3 = np.stack([np.arange(F), (np.arange(F) + 1) % F, (np.arange(F) + 2) % F], axis=1).astype(np.uint8)
    T3, E3 = intervals.eval_intervals(g, far, rows3, idle)
    assert np.array_equal(T3, To)
    ea = Eo - g.static_power * To
    assert np.allclose(E3, ea + np.asarray(idle) * To, rtol=1e-12, atol=0)


def test_interval_policy_rejects_bad_arguments():
    g = pins.graph_from_golden(pins.load_golden())
    for pts, idle in (([12.0, 12.0], [0.1, 0.1]), ([0.0], [0.1, 0.1]), ([float("nan")], [0.1, 0.1]),
                      ([12.0], [0.1]), ([12.0], [0.1, -1.0])):
        with pytest.raises(intervals.IntervalError):
            intervals.eval_intervals(g, pts, [[0] * (len(pts) + 1)], idle)
