"""Pins of the packing oracle (Sec. IV-D: Eq. 5, rules 1-3, the contraction), on the CPU: the
hand-worked fixture, the all-maximum equality the rules are designed for, the relaxation bound
at any level vector, the singleton packing that keeps every edge, the granularity partition of a
chain, and planted mistakes that these pins must catch."""
import sys
import types

import numpy as np
import pytest

import oracle
import packing_cases as pc
from oracle import packing

pytestmark = pytest.mark.usefixtures("oracle_lib")


def _all_max(g):
    return np.full((1, int(g.num_packs)), int(g.num_levels) - 1, dtype=np.uint8)


def pin_handworked(pk=packing):
    d, g = pc.load_golden()
    eft, cpred, _, _ = pk.critical_links(g)
    assert eft.tolist() == d["all_max_completion"]
    assert cpred.tolist() == d["critical_pred"]
    for case in d["cases"]:
        grp, n = pk.pack_kernels(g, g.node_stream, case["max_pack_duration"])
        assert n == case["num_groups"] and grp.tolist() == case["groups"], case["why"]
    c = d["contracted"]
    pg = pk.contract(g, np.asarray(c["groups"]), 4)
    assert pg.packed_node.tolist() == c["packed_node"]
    assert [[a, b] for a, b in zip(pg.edge_src.tolist(), pg.edge_dst.tolist())] == c["edges"]
    assert pg.node_pack.tolist() == c["node_pack"]
    assert pg.pack_time.tolist() == c["pack_time"]
    assert oracle.eval_batch(pg, _all_max(pg))[0][0] == c["all_max_makespan"]
    u = d["unsafe"]
    bad = pk.contract(g, np.asarray(u["groups"]), 4)
    assert oracle.eval_batch(bad, _all_max(bad))[0][0] == u["all_max_makespan"], u["why"]


def pin_all_max_equality(pk=packing):
    """At the default frequency the packed graph keeps every completion time: the rules keep
    every critical dependency (Sec. IV-D)."""
    for name, g, lim in pc.random_cases():
        grp, n = pk.pack_kernels(g, g.node_stream, lim)
        pg = pk.contract(g, grp, n)
        r0 = oracle.slack(g, _all_max(g)[0])
        r1 = oracle.slack(pg, _all_max(pg)[0])
        assert r1.makespan == r0.makespan, name
        pkn = np.asarray(g.node_pack)
        last = {}
        for v in r0.eft.argsort(kind="stable"):
            if pkn[v] >= 0:
                last[int(grp[pkn[v]])] = v
        for v in range(g.num_nodes):
            if pkn[v] < 0:
                assert r1.eft[pg.packed_node[v]] == r0.eft[v], (name, v)
        for gid, v in last.items():
            assert r1.eft[pg.packed_node[v]] == r0.eft[v], (name, gid)


def pin_relaxation(pk=packing):
    """Any level vector, uniform within each pack: the packed graph drops constraints and keeps
    every duration sum, so its makespan never exceeds the per-kernel graph's."""
    rng = np.random.default_rng(5)
    for name, g, lim in pc.random_cases()[:14]:
        grp, n = pk.pack_kernels(g, g.node_stream, lim)
        pg = pk.contract(g, grp, n)
        rows = rng.integers(0, g.num_levels, (64, n)).astype(np.uint8)
        Tp, Ep = oracle.eval_batch(pg, rows)
        Tu, Eu = oracle.eval_batch(g, packing.expand_levels(grp, rows))
        assert (Tp <= Tu).all(), name
        dyn_p = Ep - g.static_power * Tp
        dyn_u = Eu - g.static_power * Tu
        assert np.allclose(dyn_p, dyn_u, rtol=1e-6), name


def pin_singletons_keep_graph(pk=packing):
    """A bound below every kernel's duration leaves each kernel alone: nothing is dropped, so
    makespan and energy equal the per-kernel graph's at every level vector."""
    rng = np.random.default_rng(9)
    for name, g, _ in pc.random_cases()[:12]:
        grp, n = pk.pack_kernels(g, g.node_stream, 0.01)
        assert n == g.num_packs and sorted(grp.tolist()) == list(range(n)), name
        pg = pk.contract(g, grp, n)
        assert pg.num_edges == len(set(zip(g.edge_src.tolist(), g.edge_dst.tolist()))), name
        rows = rng.integers(0, g.num_levels, (32, n)).astype(np.uint8)
        Tp, Ep = oracle.eval_batch(pg, rows)
        Tu, Eu = oracle.eval_batch(g, packing.expand_levels(grp, rows))
        assert (Tp == Tu).all() and np.allclose(Ep, Eu, rtol=1e-12), name


def pin_chain_granularity(pk=packing):
    """One stream, no other nodes: every dependency is on the stream, so rule 3 alone splits the
    chain.  Each pack of two or more kernels stays strictly below the bound, and each pack
    plus the next kernel would reach it."""
    for seed in range(6):
        g = pc.stream_dag(100 + seed, 60, 1, comm_p=0.0, cross_p=0.0, host=False)
        t = g.pack_time[:, -1].astype(np.float64)
        for lim in (10.0, 25.0, 80.0):
            grp, n = pk.pack_kernels(g, g.node_stream, lim)
            assert (np.diff(grp) >= 0).all() and grp[0] == 0 and grp[-1] == n - 1
            sums = np.bincount(grp, weights=t, minlength=n)
            sizes = np.bincount(grp, minlength=n)
            assert all(s < lim for s, c in zip(sums, sizes) if c > 1)
            starts = np.searchsorted(grp, np.arange(1, n))
            assert all(sums[i] + t[starts[i]] >= lim for i in range(n - 1))


ALL = [pin_handworked, pin_all_max_equality, pin_relaxation, pin_singletons_keep_graph,
       pin_chain_granularity]


@pytest.mark.parametrize("pin", ALL, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


MUTANTS = {
    "rule1_dropped": ("r1 = cpred[v] >= 0 and same_stream(v, int(cpred[v]))", "r1 = True"),
    "rule2_dropped": ("r2 = all(same_stream(k, u) for k in succs[u] if cpred[k] == u)", "r2 = True"),
    "rule3_inclusive": ("r3 = acc + t_v < limit", "r3 = acc + t_v <= limit"),
    "adjacency_dropped": ("adjacent = u in preds[v]", "adjacent = True"),
    "duration_not_accumulated": ("open_pack[s] = [gid, v, acc + t_v]", "open_pack[s] = [gid, v, t_v]"),
    "inner_out_edges_kept": ("if pk[a] >= 0 and a not in last:", "if False:"),
    "inner_in_edges_kept": ("if pk[b] >= 0 and b not in first:", "if False:"),
    "table_last_member_only": ("st += float(g.pack_time[int(pk[v]), f])",
                               "st = float(g.pack_time[int(pk[v]), f])"),
    "critical_pred_ignored": ("r2 = all(same_stream(k, u) for k in succs[u] if cpred[k] == u)",
                              "r2 = all(same_stream(k, u) for k in succs[u][:1])"),
}


def _mutant(name):
    old, new = MUTANTS[name]
    src = open(packing.__file__).read()
    assert src.count(old) == 1, name
    mod = types.ModuleType(f"oracle.packing_{name}")
    mod.__package__ = "oracle"
    sys.modules[mod.__name__] = mod
    try:
        exec(compile(src.replace(old, new), mod.__name__, "exec"), mod.__dict__)
    finally:
        del sys.modules[mod.__name__]
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name):
    mod = _mutant(name)
    caught = []
    for pin in ALL:
        try:
            pin(mod)
        except (AssertionError, packing.PackingError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin caught {name}"
