"""The library's packing passes (host code: emo_pack_kernels, emo_contract_packs) against the
packing oracle, bit for bit, on the CPU: hand-worked fixture, seeded stream graphs, the workload
graphs (the 65,536-kernel one included) at several granularity bounds, edge cases and argument
errors."""
import math

import numpy as np
import pytest

import packing_cases as pc
from oracle import packing
from paper_2607_12324_amd import emo, synth

pytestmark = pytest.mark.usefixtures("oracle_lib")

FIELDS = ("edge_src", "edge_dst", "node_pack", "node_duration", "pack_time", "pack_energy",
          "packed_node")


def _bits(a):
    a = np.asarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


def _same(g, lim):
    go, no = packing.pack_kernels(g, g.node_stream, lim)
    gl, nl = emo.pack_kernels(g, g.node_stream, lim)
    assert nl == no and np.array_equal(gl, go)
    po = packing.contract(g, go, no)
    pl = emo.contract_packs(g, gl, nl)
    assert pl.num_nodes == po.num_nodes and pl.num_packs == po.num_packs
    for f in FIELDS:
        a, b = getattr(po, f), getattr(pl, f)
        assert a.shape == b.shape and np.array_equal(_bits(a), _bits(b)), f
    return gl, nl, pl


def test_handworked():
    d, g = pc.load_golden()
    for case in d["cases"]:
        grp, n = emo.pack_kernels(g, g.node_stream, case["max_pack_duration"])
        assert n == case["num_groups"] and grp.tolist() == case["groups"], case["why"]
    c = d["contracted"]
    pg = emo.contract_packs(g, c["groups"], 4)
    assert pg.packed_node.tolist() == c["packed_node"]
    assert [[a, b] for a, b in zip(pg.edge_src.tolist(), pg.edge_dst.tolist())] == c["edges"]
    assert pg.pack_time.tolist() == c["pack_time"]


@pytest.mark.parametrize("case", pc.random_cases(), ids=lambda c: f"{c[0]}-{c[2]:g}")
def test_parity(case):
    _, g, lim = case
    for bound in (lim, 12.5, math.inf, 0.01):
        _same(g, bound)


def test_unpacked_workload():
    """The 65,536-kernel per-kernel graph on 16 streams with its host launch chain."""
    g = synth.config_graph(5)
    for lim in (5000.0, 50.0):
        _same(g, lim)


def test_host_ahead_variant():
    """The same shape with launches far ahead of the kernels (1 us host nodes): kernels then
    wait on their stream and most merge."""
    g = synth._launch_graph(4, "streams-8192k-16s-F16-fast-host", P=8192, S=16, F=16,
                            packs_per_host=1, cross_p=0.0, n_cross_exact=None, median_us=8.0,
                            sigma=1.2)
    host = g.node_pack < 0
    g.node_duration[host] = synth.quantize(np.full(int(host.sum()), 0.25))
    grp, n, _ = _same(g, 5000.0)
    assert n < g.num_packs // 4


def test_edge_cases():
    empty = synth.Graph("empty", 0, np.zeros(0, np.int32), np.zeros(0, np.int32),
                        np.zeros(0, np.int32), np.zeros(0, np.float32), 0, 4,
                        np.zeros((0, 4), np.float32), np.zeros((0, 4), np.float32), 0.3,
                        node_stream=np.zeros(0, np.int32))
    grp, n = emo.pack_kernels(empty, empty.node_stream, 5000.0)
    assert n == 0 and grp.size == 0
    pg = emo.contract_packs(empty, grp, 0)
    assert pg.num_nodes == 0 and pg.num_edges == 0
    # host nodes only
    hosts = synth.Graph("hosts", 3, np.array([0, 1], np.int32), np.array([1, 2], np.int32),
                        np.full(3, -1, np.int32), np.ones(3, np.float32), 0, 2,
                        np.zeros((0, 2), np.float32), np.zeros((0, 2), np.float32), 0.3,
                        node_stream=np.full(3, -1, np.int32))
    assert emo.pack_kernels(hosts, hosts.node_stream, 5000.0)[1] == 0
    pg = emo.contract_packs(hosts, np.zeros(0, np.int32), 0)
    assert pg.num_nodes == 3 and pg.edge_src.tolist() == [0, 1]
    # duplicate edges are merged
    d, g = pc.load_golden()
    g2 = synth.Graph(g.name, g.num_nodes, np.concatenate([g.edge_src, g.edge_src[:3]]),
                     np.concatenate([g.edge_dst, g.edge_dst[:3]]), g.node_pack, g.node_duration,
                     g.num_packs, g.num_levels, g.pack_time, g.pack_energy, g.static_power,
                     node_stream=g.node_stream)
    _same(g2, 5000.0)


def test_errors():
    d, g = pc.load_golden()
    bad_stream = g.node_stream.copy()
    bad_stream[0] = -1
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.pack_kernels(g, bad_stream, 5000.0)
    for lim in (0.0, -1.0, float("nan")):
        with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
            emo.pack_kernels(g, g.node_stream, lim)
    cyc = synth.Graph(g.name, g.num_nodes, np.append(g.edge_src, 6).astype(np.int32),
                      np.append(g.edge_dst, 0).astype(np.int32), g.node_pack, g.node_duration,
                      g.num_packs, g.num_levels, g.pack_time, g.pack_energy, g.static_power,
                      node_stream=g.node_stream)
    with pytest.raises(emo.EmoError, match="CYCLE"):
        emo.pack_kernels(cyc, cyc.node_stream, 5000.0)
    with pytest.raises(emo.EmoError, match="CYCLE"):
        emo.contract_packs(cyc, [0, 1, 1, 2, 3], 4)
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.contract_packs(g, [0, 1, 1, 2, 4], 4)          # group out of range
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.contract_packs(g, [0, 1, 1, 3, 3], 4)          # group 2 empty
    twice = g.node_pack.copy()
    twice[6] = 0
    g3 = synth.Graph(g.name, g.num_nodes, g.edge_src, g.edge_dst, twice, g.node_duration,
                     g.num_packs, g.num_levels, g.pack_time, g.pack_energy, g.static_power)
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.pack_kernels(g3, g.node_stream, 5000.0)
