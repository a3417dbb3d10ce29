"""Pins of the policy-search oracle (Alg. 2, one frequency interval per pack), on the CPU:
hand-worked runs, exactness of the dynamic program on chains (where the discretised makespan is
a sufficient state: a knapsack over the packs' durations), and invariants on DAGs."""
import json
import os

import numpy as np
import pytest

import pins
from oracle import dp
from oracle import eval_batch
from paper_2607_12324_amd import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def golden_dp():
    with open(os.path.join(HERE, "golden", "handworked_dp.json")) as f:
        return json.load(f)


def test_dp_handworked():
    g = pins.graph_from_golden(pins.load_golden())
    for case in golden_dp()["cases"]:
        r = dp.dp_search(g, case["latency_target"], case["quantum"], case["pack_order"])
        assert r.num_states == case["num_states"], case
        if case["levels"] is None:
            assert r.levels is None and np.isnan(r.energy) and np.isnan(r.makespan), case
        else:
            assert list(r.levels) == case["levels"], case
            assert r.energy == case["energy"] and r.makespan == case["makespan"], case


def random_chain(rng, P, F, fixed_every=0):
    """Packs 0..P-1 in one chain (a fixed node after every `fixed_every` packs), times on the
    grid and non-increasing in level, energies on a 2^-6 grid."""
    src, dst, pack, dur = [], [], [], []
    prev = None
    for p in range(P):
        v = len(pack)
        pack.append(p)
        dur.append(0.0)
        if prev is not None:
            src.append(prev)
            dst.append(v)
        prev = v
        if fixed_every and (p + 1) % fixed_every == 0:
            w = len(pack)
            pack.append(-1)
            dur.append(float(synth.quantize(rng.uniform(0.5, 5.0))))
            src.append(prev)
            dst.append(w)
            prev = w
    t = np.sort(synth.quantize(rng.uniform(1.0, 20.0, (P, F))), axis=1)[:, ::-1].astype(np.float32)
    e = np.round(rng.uniform(0.0, 8.0, (P, F)) * 64) / 64
    return synth.Graph("chain", len(pack), np.asarray(src, np.int32), np.asarray(dst, np.int32),
                       np.asarray(pack, np.int32), np.asarray(dur, np.float32), P, F,
                       np.ascontiguousarray(t), np.ascontiguousarray(e.astype(np.float32)), 0.25)


@pytest.mark.parametrize("seed", range(4))
def test_dp_is_exact_on_chains(seed):
    """On a chain the makespan is the sum of the durations, so a policy's future depends only on
    its makespan so far: with buckets of one grid step (each bucket one exact makespan) and
    times non-increasing in level, the dynamic program finds the least energy of the whole
    policy space that meets the target."""
    rng = np.random.default_rng(500 + seed)
    checked = 0
    for i in range(12):
        P, F = int(rng.integers(1, 6)), int(rng.integers(2, 4))
        g = random_chain(rng, P, F, fixed_every=int(rng.integers(0, 3)))
        T0, _ = eval_batch(g, np.full((1, P), F - 1, np.uint8))
        Tslow, _ = eval_batch(g, np.zeros((1, P), np.uint8))
        tgt = float(np.float32(T0[0] + rng.uniform(0.0, 1.0) * (Tslow[0] - T0[0])))
        r = dp.dp_search(g, tgt, synth.Q, rng.permutation(P))
        lv, E, T = dp.exhaustive_best(g, tgt)
        assert lv is not None and r.levels is not None
        assert r.energy == E, (seed, i)
        assert r.makespan <= tgt
        checked += 1
    assert checked == 12


@pytest.mark.parametrize("seed", range(4))
def test_dp_invariants_on_dags(seed):
    """On DAGs the discretised makespan is not a sufficient state, so the search is a heuristic:
    its policy meets the target and evaluates to the reported makespan and energy, its energy is
    at least the exhaustive optimum and at most that of the all-maximum policy when that one is
    feasible, and it finds nothing only when nothing is feasible."""
    rng = np.random.default_rng(600 + seed)
    for i in range(10):
        g = synth.random_dag(rng, int(rng.integers(3, 9)), float(rng.uniform(0.2, 0.6)), 0.7,
                             int(rng.integers(2, 4)))
        P, F = g.num_packs, g.num_levels
        if P == 0 or F ** P > 4096:
            continue
        T0, E0 = eval_batch(g, np.full((1, P), F - 1, np.uint8))
        tgt = float(np.float32(T0[0] * rng.uniform(0.95, 1.3)))
        q = float(2.0 ** int(rng.integers(-4, 3)))
        r = dp.dp_search(g, tgt, q)
        lv, E, _ = dp.exhaustive_best(g, tgt)
        if lv is None:
            assert r.levels is None and r.num_states == 0
            continue
        if np.float32(T0[0]) <= np.float32(tgt):
            assert r.levels is not None and r.energy <= float(np.float32(E0[0]))
        if r.levels is None:
            continue
        Tr, Er = eval_batch(g, r.levels[None, :])
        assert float(np.float32(Tr[0])) == r.makespan and float(np.float32(Er[0])) == r.energy
        assert r.makespan <= tgt and r.energy >= E


def test_dp_rejects_bad_arguments():
    g = pins.graph_from_golden(pins.load_golden())
    with pytest.raises(ValueError):
        dp.dp_search(g, 20.0, 1.0, [0, 0, 1])
    with pytest.raises(ValueError):
        dp.dp_search(g, 20.0, 0.0)
