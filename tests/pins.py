"""Pins for the CPU oracle: checks against what the paper and the mathematics fix, written
independently of the oracle's own code.

* A hand-worked example (tests/golden/handworked_fork_join.json), values derived by hand.
* Brute force over all source-to-sink paths on tiny DAGs: the makespan of Eq. 2 is the longest
  path, the slack of a node is the makespan minus the longest path through it, the depth of a
  node is the longest path to it counted in edges.
* Closed forms: a chain's makespan is its duration sum; disjoint chains give the largest sum.
* Invariants: slack >= 0 and = 0 along Alg. 1's critical-predecessor chain; lowering a pack's
  level never shortens the makespan (tables non-increasing in level, Sec. IV-D); the what-if
  identity of total float; the static-energy identity.
* Exhaustive selection over every policy of a small graph.

Each ``pin_*`` function raises AssertionError on a mismatch.  They are plain functions so that
tests/test_oracle_mutants.py can run them against copies of the oracle with planted mistakes.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle
from paper_2607_12324_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------- helpers

def graph_from_golden(d) -> synth.Graph:
    return synth.Graph(
        name="golden", num_nodes=len(d["node_pack"]),
        edge_src=np.asarray(d["edge_src"], dtype=np.int32),
        edge_dst=np.asarray(d["edge_dst"], dtype=np.int32),
        node_pack=np.asarray(d["node_pack"], dtype=np.int32),
        node_duration=np.asarray(d["node_duration"], dtype=np.float32),
        num_packs=len(d["pack_time"]), num_levels=int(d["num_levels"]),
        pack_time=np.asarray(d["pack_time"], dtype=np.float32),
        pack_energy=np.asarray(d["pack_energy"], dtype=np.float32),
        static_power=float(d["static_power"]))


def load_golden(name="handworked_fork_join.json"):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def all_paths(g):
    """Every source-to-sink path as a list of nodes (tiny graphs only)."""
    V = g.num_nodes
    succ = [[] for _ in range(V)]
    npred = [0] * V
    for a, b in zip(g.edge_src.tolist(), g.edge_dst.tolist()):
        if b not in succ[a]:
            succ[a].append(b)
            npred[b] += 1
    paths = []

    def walk(v, acc):
        acc.append(v)
        if not succ[v]:
            paths.append(list(acc))
        for u in succ[v]:
            walk(u, acc)
        acc.pop()

    for v in range(V):
        if npred[v] == 0:
            walk(v, [])
    return paths


def durations(g, row):
    """Per-node duration under one level row, float64."""
    d = np.asarray(g.node_duration, dtype=np.float64).copy()
    for v in range(g.num_nodes):
        p = int(g.node_pack[v])
        if p >= 0:
            d[v] = float(g.pack_time[p, int(row[p])])
    return d


def brute_makespan_and_slack(g, row, paths=None):
    paths = all_paths(g) if paths is None else paths
    d = durations(g, row)
    sums = [sum(d[v] for v in path) for path in paths]
    T = max(sums) if sums else 0.0
    through = np.full(g.num_nodes, -np.inf)
    for path, s in zip(paths, sums):
        for v in path:
            through[v] = max(through[v], s)
    return T, T - through


def brute_depth(g):
    depth = np.zeros(g.num_nodes, dtype=np.int64)
    for path in all_paths(g):
        for i, v in enumerate(path):
            depth[v] = max(depth[v], i)
    return depth


def with_duration(g, v, new_dur):
    d = g.node_duration.copy()
    d[v] = np.float32(new_dur)
    return synth.Graph(**{**g.__dict__, "node_duration": d})


def with_table_entry(g, p, lvl, new_t):
    t = g.pack_time.copy()
    t[p, lvl] = np.float32(new_t)
    return synth.Graph(**{**g.__dict__, "pack_time": t})


def tiny_dags(seed, count, on_grid=True):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        V = int(rng.integers(1, 10))
        F = int(rng.integers(1, 4))
        out.append(synth.random_dag(rng, V, float(rng.uniform(0.1, 0.6)),
                                    float(rng.uniform(0.3, 0.9)), F, on_grid=on_grid,
                                    name=f"tiny{i}"))
    return out


def random_rows(rng, g, n):
    if g.num_packs == 0:
        return np.zeros((n, 0), dtype=np.uint8)
    return rng.integers(0, g.num_levels, size=(n, g.num_packs), dtype=np.uint8)


# ----------------------------------------------------------------------------- pins

def pin_handworked():
    d = load_golden()
    g = graph_from_golden(d)
    rows = synth.exhaustive_policies(g.num_packs, g.num_levels, 0, 2 ** g.num_packs)
    T, E = oracle.eval_batch(g, rows)
    assert np.array_equal(T, np.asarray(d["makespan"])), (T, d["makespan"])
    assert np.array_equal(E, np.asarray(d["energy"])), (E, d["energy"])
    for c, expect in d["node_slack"].items():
        r = oracle.slack(g, rows[int(c)])
        assert np.array_equal(r.slack, np.asarray(expect)), (c, r.slack, expect)
    for s in d["selection"]:
        idx, feas, n = oracle.select(T, E, s["target"])
        assert idx == s["index"] and n == s["num_feasible"], (s, idx, n)
        assert np.array_equal(feas, T <= s["target"])
    r = oracle.slack(g, rows[-1])
    names = d["nodes"]
    v = int(np.argmax(r.eft))
    chain = []
    while v >= 0:
        chain.append(names[v])
        v = int(r.critical_pred[v])
    assert chain[::-1] == d["critical_path_all_max"], chain
    order, depth = oracle.topo_order(g.num_nodes, g.edge_src, g.edge_dst)
    assert order.tolist() == d["topo_order"] and depth.tolist() == d["depth"]


def pin_bruteforce_paths(seed=11, count=60, on_grid=True):
    """Makespan and slack against longest paths, on random tiny DAGs and random policies."""
    rng = np.random.default_rng(seed + 1)
    for g in tiny_dags(seed, count, on_grid):
        paths = all_paths(g)
        rows = random_rows(rng, g, 6)
        T, E = oracle.eval_batch(g, rows)
        for i, row in enumerate(rows):
            Tb, sb = brute_makespan_and_slack(g, row, paths)
            r = oracle.slack(g, row)
            if on_grid:
                assert T[i] == Tb and r.makespan == Tb, (g.name, T[i], Tb)
                assert np.array_equal(r.slack, sb), (g.name, r.slack, sb)
            else:
                assert abs(T[i] - Tb) <= 1e-12 * max(1.0, Tb), (g.name, T[i], Tb)
                assert np.allclose(r.slack, sb, rtol=0, atol=1e-9 * max(1.0, Tb)), (g.name, r.slack, sb)
            # energy: pack energies at the chosen levels plus static power times makespan
            e_sum = sum(float(g.pack_energy[p, row[p]]) for p in range(g.num_packs))
            assert abs(E[i] - (e_sum + float(np.float32(g.static_power)) * Tb)) <= 1e-12 * max(1.0, E[i])


def pin_topo_order(seed=5, count=60):
    for g in tiny_dags(seed, count):
        order, depth = oracle.topo_order(g.num_nodes, g.edge_src, g.edge_dst)
        assert sorted(order.tolist()) == list(range(g.num_nodes))
        pos = np.empty(g.num_nodes, dtype=np.int64)
        pos[order] = np.arange(g.num_nodes)
        assert np.all(pos[g.edge_src] < pos[g.edge_dst]) if g.num_edges else True
        assert np.array_equal(depth, brute_depth(g)), (g.name, depth, brute_depth(g))
        keys = [(int(depth[v]), int(v)) for v in order]
        assert keys == sorted(keys)


def pin_cycles():
    for src, dst in (([0], [0]), ([0, 1, 2], [1, 2, 0]), ([0, 1, 1], [1, 2, 0])):
        try:
            oracle.topo_order(3, np.asarray(src), np.asarray(dst))
        except oracle.OracleError:
            continue
        raise AssertionError(f"cycle not detected: {src}->{dst}")


def pin_closed_forms(seed=3):
    rng = np.random.default_rng(seed)
    for trial in range(20):
        # one chain in a shuffled id order: makespan = sum of durations
        n = int(rng.integers(1, 12))
        ids = rng.permutation(n)
        dur = synth.quantize(rng.uniform(0.5, 30.0, n))
        g = synth.Graph("chain", n, ids[:-1].astype(np.int32), ids[1:].astype(np.int32),
                        np.full(n, -1, np.int32), dur, 0, 1, np.zeros((0, 1), np.float32),
                        np.zeros((0, 1), np.float32), 0.0)
        T, _ = oracle.eval_batch(g, np.zeros((1, 0), np.uint8))
        assert T[0] == float(np.sum(dur.astype(np.float64)))
        # k disjoint chains: makespan = the largest chain sum
        k = int(rng.integers(1, 5))
        src, dst, durs, sums, base = [], [], [], [], 0
        for _ in range(k):
            m = int(rng.integers(1, 6))
            dd = synth.quantize(rng.uniform(0.5, 30.0, m))
            durs.append(dd)
            sums.append(float(np.sum(dd.astype(np.float64))))
            src += list(range(base, base + m - 1))
            dst += list(range(base + 1, base + m))
            base += m
        g = synth.Graph("chains", base, np.asarray(src, np.int32), np.asarray(dst, np.int32),
                        np.full(base, -1, np.int32), np.concatenate(durs), 0, 1,
                        np.zeros((0, 1), np.float32), np.zeros((0, 1), np.float32), 0.0)
        T, E = oracle.eval_batch(g, np.zeros((1, 0), np.uint8))
        assert T[0] == max(sums) and E[0] == 0.0


def pin_all_max_is_longest_path(seed=21, count=40):
    for g in tiny_dags(seed, count):
        row = np.full(g.num_packs, g.num_levels - 1, dtype=np.uint8)
        T, _ = oracle.eval_batch(g, row[None, :])
        Tb, _ = brute_makespan_and_slack(g, row)
        assert T[0] == Tb


def pin_invariants(g, rows, check_whatif=True):
    """Slack, monotonicity, what-if and energy identities on graph `g` (grid-exact data)."""
    sp = float(np.float32(g.static_power))
    for row in rows:
        r = oracle.slack(g, row)
        T = r.makespan
        assert np.all(r.slack >= 0), r.slack.min()
        # zero slack along the critical-predecessor chain from the latest-finishing node
        v = int(np.argmax(r.eft))
        assert r.eft[v] == T
        while v >= 0:
            assert r.slack[v] == 0.0, (v, r.slack[v])
            v = int(r.critical_pred[v])
        # energy identity, and linearity in the static power
        e_sum = sum(float(g.pack_energy[p, row[p]]) for p in range(g.num_packs))
        assert abs(r.energy - e_sum - sp * T) <= 1e-12 * max(1.0, r.energy)
        g0 = synth.Graph(**{**g.__dict__, "static_power": 0.0})
        _, E0 = oracle.eval_batch(g0, row[None, :])
        assert abs(r.energy - E0[0] - sp * T) <= 1e-12 * max(1.0, r.energy)
        # lowering any single pack's level never shortens the makespan
        lowered = []
        for p in range(g.num_packs):
            if row[p] > 0:
                rr = row.copy()
                rr[p] -= 1
                lowered.append(rr)
        if lowered:
            T2, _ = oracle.eval_batch(g, np.asarray(lowered))
            assert np.all(T2 >= T), (T2.min(), T)
        if not check_whatif:
            continue
        # what-if identity: stretching node v by delta <= slack(v) keeps T; beyond, T grows by
        # exactly delta - slack(v)
        for v in range(g.num_nodes):
            s = r.slack[v]
            p = int(g.node_pack[v])
            for delta in (s / 2, s, s + 1.0):
                delta = float(synth.quantize(delta)) if delta > 0 else 0.0
                if p < 0:
                    g2 = with_duration(g, v, float(g.node_duration[v]) + delta)
                else:
                    lvl = int(row[p])
                    g2 = with_table_entry(g, p, lvl, float(g.pack_time[p, lvl]) + delta)
                T2, _ = oracle.eval_batch(g2, row[None, :])
                expect = T + max(0.0, delta - s)
                assert T2[0] == expect, (v, s, delta, T2[0], expect)


def pin_invariants_tiny(seed=31, count=25):
    rng = np.random.default_rng(seed + 1)
    for g in tiny_dags(seed, count):
        pin_invariants(g, random_rows(rng, g, 3))


def pin_invariants_tiny_workload():
    g = synth.config_graph(1)
    rows = synth.config_policies(1, g, 0, 4 ** 8)
    rng = np.random.default_rng(2)
    pick = rows[rng.choice(rows.shape[0], 4, replace=False)]
    pin_invariants(g, np.concatenate([pick, rows[-1:]]))


def pin_exhaustive_selection(seed=41, count=20):
    """Exhaustive Eq. 4 optimum over every per-pack policy of small graphs."""
    rng = np.random.default_rng(seed)
    for g in tiny_dags(seed, count):
        if g.num_levels ** g.num_packs > 4096:
            continue
        rows = synth.exhaustive_policies(g.num_packs, g.num_levels, 0, g.num_levels ** g.num_packs)
        T, E = oracle.eval_batch(g, rows)
        paths = all_paths(g)
        Tb = np.asarray([brute_makespan_and_slack(g, r, paths)[0] for r in rows])
        assert np.array_equal(T, Tb)
        for ratio in (1.0, 1.05, 1.3, 0.9):
            target = float(np.float32(ratio * Tb.min()))
            idx, feas, n = oracle.select(T, E, target)
            ok = Tb <= target
            assert np.array_equal(feas, ok) and n == int(ok.sum())
            if not ok.any():
                assert idx == -1
                continue
            best = min((E[c], c) for c in np.nonzero(ok)[0])
            assert idx == best[1], (idx, best)
        _ = rng


def pin_select_edge_cases(seed=51):
    rng = np.random.default_rng(seed)
    idx, feas, n = oracle.select(np.zeros(0), np.zeros(0), 1.0)
    assert idx == -1 and n == 0 and feas.size == 0
    T = np.array([1.0, np.nan, 0.5, 2.0])
    E = np.array([3.0, 0.0, 3.0, 1.0])
    idx, feas, n = oracle.select(T, E, 1.0)
    assert idx == 0 and n == 2 and feas.tolist() == [True, False, True, False]
    for _ in range(20):
        B = int(rng.integers(1, 200))
        T = rng.integers(0, 10, B).astype(np.float64)
        E = rng.integers(0, 5, B).astype(np.float64)
        tgt = float(rng.integers(0, 10))
        idx, feas, n = oracle.select(T, E, tgt)
        cand = [(E[c], c) for c in range(B) if T[c] <= tgt]
        assert idx == (min(cand)[1] if cand else -1) and n == len(cand)


def pin_exhaustive_tiny_workload():
    """The tiny benchmark workload: all 4^8 policies against path enumeration."""
    g = synth.config_graph(1)
    rows = synth.config_policies(1, g)
    T, E = oracle.eval_batch(g, rows, nthreads=4)
    paths = all_paths(g)
    pk = np.asarray(g.node_pack)
    D = np.tile(g.node_duration.astype(np.float64), (rows.shape[0], 1))
    for v in range(g.num_nodes):
        if pk[v] >= 0:
            D[:, v] = g.pack_time[pk[v]].astype(np.float64)[rows[:, pk[v]]]
    Tb = np.max(np.stack([D[:, p].sum(axis=1) for p in paths]), axis=0)
    assert np.array_equal(T, Tb)
    T0 = Tb[-1]
    assert np.all(rows[-1] == g.num_levels - 1) and T0 == Tb.min()
    target = float(np.float32(1.05 * T0))
    idx, feas, n = oracle.select(T, E, target)
    ok = Tb <= target
    assert n == int(ok.sum()) and np.array_equal(feas, ok)
    ebf = np.sum(g.pack_energy.astype(np.float64)[np.arange(g.num_packs)[None, :], rows], axis=1) \
        + float(np.float32(g.static_power)) * Tb
    cand = np.nonzero(ok)[0]
    best = cand[np.lexsort((cand, ebf[cand]))[0]]
    assert idx == int(best), (idx, best)


def pin_invalid_level(seed=61):
    """A level byte >= F is not a policy: that candidate's makespan, energy and every slack
    value are NaN, it is never feasible and never selected; the other rows are unaffected."""
    rng = np.random.default_rng(seed)
    for g in tiny_dags(seed, 20):
        if g.num_packs == 0:
            continue
        rows = random_rows(rng, g, 5)
        good_T, good_E = oracle.eval_batch(g, rows)
        bad = rows.copy()
        bad[1, int(rng.integers(0, g.num_packs))] = g.num_levels + int(rng.integers(0, 256 - g.num_levels))
        bad[3, -1] = 255
        T, E = oracle.eval_batch(g, bad)
        assert np.isnan(T[1]) and np.isnan(E[1]) and np.isnan(T[3]) and np.isnan(E[3])
        keep = [0, 2, 4]
        assert np.array_equal(T[keep], good_T[keep]) and np.array_equal(E[keep], good_E[keep])
        r = oracle.slack(g, bad[1])
        assert np.isnan(r.makespan) and np.all(np.isnan(r.slack)) and np.all(np.isnan(r.lft))
        for pn in (False, True):
            Tb, Eb, Sb = oracle.slack_batch(g, bad, per_node=pn)
            assert np.all(np.isnan(Sb[[1, 3]])) and not np.any(np.isnan(Sb[keep]))
            assert np.isnan(Tb[1]) and np.isnan(Eb[3])
        idx, feas, n = oracle.select(T, E, float("inf"))
        assert not feas[1] and not feas[3] and n == 3 and idx in keep


def pin_critical_pred_ties():
    """Eq. 5 with equal completion times: the first maximal predecessor in the canonical order
    (depth, then id), which is not always the lowest id.  Nodes: 0 (1 us) -> 1 (4 us); 2 (5 us);
    1 and 2 -> 3.  C_1 = C_2 = 5; node 2 has depth 0 and node 1 depth 1, so 2 comes first."""
    g = synth.Graph("ties", 4, np.array([0, 1, 2], np.int32), np.array([1, 3, 3], np.int32),
                    np.full(4, -1, np.int32), np.array([1, 4, 5, 2], np.float32), 0, 1,
                    np.zeros((0, 1), np.float32), np.zeros((0, 1), np.float32), 0.0)
    r = oracle.slack(g, np.zeros(0, np.uint8))
    assert r.eft.tolist() == [1.0, 5.0, 5.0, 7.0]
    assert r.critical_pred.tolist() == [-1, 0, -1, 2], r.critical_pred
    # with unequal times the later one in the order can win
    g2 = synth.Graph(**{**g.__dict__, "node_duration": np.array([1, 4.5, 5, 2], np.float32)})
    assert oracle.slack(g2, np.zeros(0, np.uint8)).critical_pred.tolist() == [-1, 0, -1, 1]


def pin_slack_batch(seed=71, count=30):
    """The batched slack (by pack and by node) against longest paths through each node."""
    rng = np.random.default_rng(seed + 1)
    for g in tiny_dags(seed, count):
        paths = all_paths(g)
        rows = random_rows(rng, g, 5)
        T, E, SN = oracle.slack_batch(g, rows, per_node=True, nthreads=2)
        _, _, SP = oracle.slack_batch(g, rows, per_node=False)
        for i, row in enumerate(rows):
            Tb, sb = brute_makespan_and_slack(g, row, paths)
            assert T[i] == Tb and np.array_equal(SN[i], sb), (g.name, SN[i], sb)
            for v in range(g.num_nodes):
                p = int(g.node_pack[v])
                if p >= 0:
                    assert SP[i, p] == sb[v], (g.name, p, SP[i, p], sb[v])
        T1, E1 = oracle.eval_batch(g, rows)
        assert np.array_equal(T, T1) and np.array_equal(E, E1)


ALL_PINS = [pin_handworked, pin_bruteforce_paths, pin_topo_order, pin_cycles, pin_closed_forms,
            pin_all_max_is_longest_path, pin_invariants_tiny, pin_invariants_tiny_workload,
            pin_exhaustive_selection, pin_select_edge_cases, pin_exhaustive_tiny_workload,
            pin_invalid_level, pin_critical_pred_ties, pin_slack_batch]
