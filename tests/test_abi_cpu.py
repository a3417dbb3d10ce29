"""The C-ABI library on the CPU: exported symbols, host-side validation, graph analysis and the
canonical topological order (no device work)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import pins
from paper_2607_12324_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "emo.h")


@pytest.fixture(scope="module")
def emo():
    from paper_2607_12324_amd import emo as mod
    return mod


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(emo_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol(emo):
    names = declared_functions()
    assert set(names) == set(emo.ENTRY_POINTS)
    out = subprocess.run(["nm", "-D", "--defined-only", emo.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (emo_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        assert getattr(emo.lib, n) is not None


def test_status_strings(emo):
    for code, name in emo.STATUS_NAMES.items():
        assert emo.lib.emo_status_string(code).decode() == name


def _load(emo, g):
    return emo.EmoGraph(g, device=-1)


def _raises(emo, g, status):
    with pytest.raises(emo.EmoError) as ei:
        _load(emo, g)
    assert ei.value.status == status, str(ei.value)
    return str(ei.value)


def _base():
    return pins.graph_from_golden(pins.load_golden())


def _mod(g, **kw):
    return synth.Graph(**{**g.__dict__, **kw})


def test_validation_errors(emo):
    g = _base()
    INV, CYC = 1, 2
    _raises(emo, _mod(g, edge_dst=np.asarray([1, 2, 3, 9], np.int32)), INV)
    _raises(emo, _mod(g, edge_src=np.asarray([0, 0, 1, 3], np.int32)), CYC)  # 3 -> 3
    _raises(emo, _mod(g, edge_src=np.asarray([0, 0, 1, 2, 3], np.int32),
                      edge_dst=np.asarray([1, 2, 3, 3, 0], np.int32)), CYC)
    _raises(emo, _mod(g, node_pack=np.asarray([-1, 0, 0, 2], np.int32)), INV)   # duplicate
    _raises(emo, _mod(g, node_pack=np.asarray([-1, 0, 1, 5], np.int32)), INV)   # out of range
    _raises(emo, _mod(g, node_pack=np.asarray([-1, 0, 1, -1], np.int32)), INV)  # pack 2 unused
    _raises(emo, _mod(g, node_duration=np.asarray([-1, 0, 0, 0], np.float32)), INV)
    _raises(emo, _mod(g, node_duration=np.asarray([np.inf, 0, 0, 0], np.float32)), INV)
    t = g.pack_time.copy(); t[1, 0] = np.nan
    _raises(emo, _mod(g, pack_time=t), INV)
    e = g.pack_energy.copy(); e[2, 1] = -1
    _raises(emo, _mod(g, pack_energy=e), INV)
    _raises(emo, _mod(g, static_power=float("nan")), INV)
    _raises(emo, _mod(g, static_power=-0.5), INV)
    tt = np.zeros((3, 0), np.float32)
    _raises(emo, _mod(g, num_levels=0, pack_time=tt, pack_energy=tt), INV)
    big = np.zeros((3, 257), np.float32)
    _raises(emo, _mod(g, num_levels=257, pack_time=big, pack_energy=big), INV)


def test_host_only_graph_rejects_batch_calls(emo):
    gh = _load(emo, _base())
    st = emo.lib.emo_eval_policies(gh._h, None, 0, None, None, None)
    assert st == 5


def test_empty_and_degenerate_graphs_load(emo):
    z = np.zeros(0, np.int32)
    zf = np.zeros((0, 1), np.float32)
    empty = synth.Graph("empty", 0, z, z, z, np.zeros(0, np.float32), 0, 1, zf, zf, 0.0)
    gh = _load(emo, empty)
    assert gh.info()["num_nodes"] == 0
    order, depth = gh.topo_order()
    assert order.size == 0
    one = synth.Graph("one", 1, z, z, np.zeros(1, np.int32), np.zeros(1, np.float32), 1, 1,
                      np.ones((1, 1), np.float32), np.ones((1, 1), np.float32), 0.0)
    gh = _load(emo, one)
    inf = gh.info()
    assert inf["num_dynamic_nodes"] == 1 and inf["eval_slots"] == 0


def test_duplicate_edges_are_merged(emo):
    g = _base()
    g2 = _mod(g, edge_src=np.concatenate([g.edge_src, g.edge_src[:2]]),
              edge_dst=np.concatenate([g.edge_dst, g.edge_dst[:2]]))
    assert _load(emo, g2).info()["num_edges"] == g.num_edges


def _implied_edges(g) -> int:
    """Full transitive closure (Python integers as bit sets, filled in reverse topological
    order): counts merged edges u -> v such that another successor w of u reaches v."""
    V = g.num_nodes
    edges = sorted(set(zip(g.edge_src.tolist(), g.edge_dst.tolist())))
    succ = [[] for _ in range(V)]
    indeg = [0] * V
    for u, v in edges:
        succ[u].append(v)
        indeg[v] += 1
    order = [v for v in range(V) if indeg[v] == 0]
    for v in order:
        for w in succ[v]:
            indeg[w] -= 1
            if indeg[w] == 0:
                order.append(w)
    reach = [0] * V          # nodes reachable by one or more edges
    for u in reversed(order):
        r = 0
        for w in succ[u]:
            r |= (1 << w) | reach[w]
        reach[u] = r
    return sum(1 for u, v in edges if any(w != v and (reach[w] >> v) & 1 for w in succ[u]))


@pytest.mark.parametrize("seed", range(4))
def test_implied_edges_match_brute_force(emo, seed):
    """The loader skips exactly the edges implied by longer paths (transitive reduction) on
    graphs small enough for its search budget."""
    rng = np.random.default_rng(700 + seed)
    total = 0
    for i in range(12):
        V = int(rng.integers(2, 70))
        g = synth.random_dag(rng, V, float(rng.uniform(0.03, 0.4)), 0.6, 3)
        want = _implied_edges(g)
        assert _load(emo, g).info()["num_implied_edges"] == want
        total += want
    assert total > 0


def test_implied_edges_on_workloads(emo):
    """Cross-stream edges that span an all-stream synchronisation node are implied."""
    g = synth.config_graph(4)
    assert _load(emo, g).info()["num_implied_edges"] == _implied_edges(g)


def test_chain_detection(emo):
    """Chain lanes: the candidate-dependent nodes must form at most 64 disjoint chains."""
    expect = {1: 0, 2: 1, 3: 0, 4: 0, 5: 16}   # 2 cross edges / 1 stream / cross edges / syncs / 16 streams
    for k, lanes in expect.items():
        assert _load(emo, synth.config_graph(k)).info()["chain_lanes"] == lanes, k
    for S, lanes in ((1, 1), (3, 4), (17, 32), (64, 64), (65, 0)):
        g = synth.stream_graph(5, 20 * S, S, 4)
        assert _load(emo, g).info()["chain_lanes"] == lanes, S


def test_chain_windows(emo):
    """Window width of the windowed chain kernel: the widest of 256, 128, ..., 16 packs whose
    LDS working set fits (two level windows of 16 // chains groups of 64 candidates, two table
    windows, two step blocks, the slack tile) and whose copy takes at most 4 pieces of 16 bytes
    per thread (one piece for pack counts that are not multiples of 16, whose rows the kernel
    copies from the dwords around each piece); none with more than 16 chains, more than 128
    levels or a chain that goes back to an earlier window."""
    expect = {1: 0, 2: 16, 3: 0, 4: 0, 5: 256}
    for k, win in expect.items():
        assert _load(emo, synth.config_graph(k)).info()["chain_window"] == win, k
    for (P, S, F), win in (((8192, 16, 16), 256), ((4096, 3, 8), 64), ((8192, 9, 32), 64),
                           ((10000, 1, 16), 16), ((9008, 5, 16), 64), ((8304, 7, 8), 128),
                           ((4096, 2, 64), 32), ((4096, 16, 128), 32), ((9000, 5, 16), 64),
                           ((8301, 7, 8), 64),
                           ((8192, 17, 4), 0), ((4096, 2, 200), 0)):
        g = synth.stream_graph(7, P, S, F)
        assert _load(emo, g).info()["chain_window"] == win, (P, S, F)
    # one chain over 48 packs: in pack order it has windows 0, 1, 2; visiting packs 32..47
    # before 16..31 it goes back from window 2 to window 1
    for order, win in ((list(range(48)), 16), (list(range(16)) + list(range(32, 48)) + list(range(16, 32)), 0)):
        rng = np.random.default_rng(3)
        t = synth.quantize(rng.uniform(1.0, 9.0, (48, 2))).astype(np.float32)
        g = synth.Graph("one-chain", 48, np.arange(47, dtype=np.int32), np.arange(1, 48, dtype=np.int32),
                        np.asarray(order, np.int32), np.zeros(48, np.float32), 48, 2, t, 0.5 * t, 0.1)
        inf = _load(emo, g).info()
        assert inf["chain_lanes"] == 1 and inf["chain_window"] == win, order[:20]


def _cut_nodes(V, src, dst):
    """Nodes that every other node reaches or is reached from (the definition of a cut),
    by full reachability (Python integers as bit sets)."""
    succ = [[] for _ in range(V)]
    indeg = [0] * V
    for u, v in set(zip(src.tolist(), dst.tolist())):
        succ[u].append(v)
        indeg[v] += 1
    order = [v for v in range(V) if indeg[v] == 0]
    for v in order:
        for w in succ[v]:
            indeg[w] -= 1
            if indeg[w] == 0:
                order.append(w)
    down = [0] * V
    for u in reversed(order):
        for w in succ[u]:
            down[u] |= (1 << w) | down[w]
    up = [0] * V
    for v in range(V):
        r = down[v]
        while r:
            w = (r & -r).bit_length() - 1
            up[w] |= 1 << v
            r &= r - 1
    full = (1 << V) - 1
    return [c for c in range(V) if (down[c] | up[c] | (1 << c)) == full], up


def _expected_cut_segments(g, max_packs):
    """Segments of the cut-segment kernels from the definition: segment ends are cuts after a
    multiple of 32 packs (and the end of the graph); whole pieces are taken greedily while a
    segment holds at most max_packs packs; 0 when a piece is larger or there is one segment."""
    if g.num_packs % 32:
        return 0
    cuts, up = _cut_nodes(g.num_nodes, g.edge_src, g.edge_dst)
    packs = {int(v) for v in np.nonzero(g.node_pack >= 0)[0]}
    ends = set()
    for c in cuts:
        n = sum(1 for v in packs if (up[c] >> v) & 1) + (1 if c in packs else 0)
        if n % 32 == 0 and n > 0:
            ends.add(n)
    ends.add(g.num_packs)
    seg, last = [0], None
    for e in sorted(ends):
        if e - seg[-1] <= max_packs:
            last = e
            continue
        if last is None or last <= seg[-1] or e - last > max_packs:
            return 0
        seg.append(last)
        last = e
    seg.append(last)
    return len(seg) - 1 if len(seg) > 2 else 0


def test_cut_segments(emo):
    """Segments of the cut-segment kernels on the workloads and on packed graphs with periodic
    all-stream synchronisations: at most 256 packs (and 32 KB of (time, energy) table rows) per
    segment, ends after a multiple of 32 packs, packs visited in increasing id."""
    expect = {1: 0, 2: 0, 3: 0, 4: 16, 5: 0}
    for k, m in expect.items():
        info = _load(emo, synth.config_graph(k)).info()
        # every workload's times lie on the 2^-4 us grid with small enough sums
        assert info["cut_segments"] == m and info["exact_time_sums"] == 1, k
    for (P, S, F, se), m in (((1024, 8, 16, 256), 4), ((2048, 4, 8, 128), 8), ((1056, 8, 16, 256), 5),
                             ((960, 6, 5, 96), 5), ((1024, 4, 32, 128), 8), ((1024, 4, 32, 256), 0),
                             ((1000, 4, 16, 100), 0), ((1024, 4, 200, 128), 0), ((2048, 8, 16, 64), 8)):
        g = synth.packed_graph(11, P, S, F, sync_every=se, cross_p=0.05)
        assert _load(emo, g).info()["cut_segments"] == m, (P, S, F, se)
    g = synth.packed_graph(11, 1024, 8, 16, sync_every=256, cross_p=0.05, shuffle_pack_ids=True)
    assert _load(emo, g).info()["cut_segments"] == 0
    # the segments do not depend on the times; whether every time sum is exact does: times off a
    # common dyadic grid with a sum of largest durations of 2^24 grid units or more are not
    g = synth.packed_graph(11, 1024, 8, 16, sync_every=256, cross_p=0.05)
    info = _load(emo, g).info()
    assert info["cut_segments"] == 4 and info["exact_time_sums"] == 1
    for scale in (64.0, 8.0, 1.1):
        info = _load(emo, _mod(g, pack_time=(g.pack_time * scale).astype(np.float32))).info()
        assert info["cut_segments"] == 4 and info["exact_time_sums"] == (scale == 8.0), scale
    t = g.pack_time.copy()
    t[5, 3] += np.float32(2.0 ** -12)   # grid 2^-12: the sum bound becomes 4096 us
    info = _load(emo, _mod(g, pack_time=t)).info()
    assert info["cut_segments"] == 4 and info["exact_time_sums"] == 0


@pytest.mark.parametrize("seed", range(4))
def test_cut_segments_match_definition(emo, seed):
    """Cut detection (a linear scan of one topological order) against the definition by full
    reachability, through the segment count, on block graphs where some synchronisations are
    bypassed and some packs are cuts as well."""
    rng = np.random.default_rng(900 + seed)
    seen = set()
    for i in range(8):
        F = int(rng.choice([16, 32, 64]))   # at most 256, 128 or 64 packs per segment
        g = synth.block_graph(rng, int(rng.integers(2, 20)), float(rng.uniform(0.0, 0.5)), F)
        want = _expected_cut_segments(g, 4096 // F)
        assert _load(emo, g).info()["cut_segments"] == want, (seed, i, g.num_packs)
        seen.add(want > 0)
    assert seen == {True, False} or seed > 0


@pytest.mark.parametrize("seed", range(6))
def test_topo_order_matches_oracle_on_random_dags(emo, oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    for i in range(15):
        g = synth.random_dag(rng, int(rng.integers(1, 60)), float(rng.uniform(0.02, 0.3)),
                             float(rng.uniform(0.2, 0.9)), int(rng.integers(1, 5)))
        order, depth = _load(emo, g).topo_order()
        o2, d2 = oracle.topo_order(g.num_nodes, g.edge_src, g.edge_dst)
        assert np.array_equal(order, o2) and np.array_equal(depth, d2)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_topo_order_and_analysis_on_workloads(emo, oracle_lib, k):
    g = synth.config_graph(k)
    gh = _load(emo, g)
    order, depth = gh.topo_order()
    o2, d2 = oracle.topo_order(g.num_nodes, g.edge_src, g.edge_dst)
    assert np.array_equal(order, o2) and np.array_equal(depth, d2)
    inf = gh.info()
    assert inf["num_packs"] == g.num_packs and inf["num_levels"] == g.num_levels
    assert inf["pack_order_monotone"] == 1
    assert inf["max_depth"] == int(d2.max())
    # candidate-independent nodes: those with no pack ancestor (host launch chains)
    n_host_const = {1: 4, 2: 64, 3: 512, 4: 0, 5: 65536}[k]
    assert inf["num_dynamic_nodes"] == g.num_nodes - n_host_const
    # the finish time of the candidate-independent nodes is the host chain's total
    if n_host_const:
        host = np.nonzero(g.node_pack < 0)[0]
        assert inf["const_makespan"] == float(np.sum(g.node_duration[host].astype(np.float64)))


def test_one_hip_runtime_whatever_the_import_order():
    """Importing the binding before torch must not map a second HIP runtime: the library has
    to share torch's, or it sees no device."""
    import subprocess
    import sys
    code = ("from paper_2607_12324_amd import emo\nimport torch\n"
            "maps = [l.split()[-1] for l in open('/proc/self/maps') if 'amdhip64' in l]\n"
            "print(len(set(maps)))\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "1"
