"""Shared inputs and pins of the packing tests (Sec. IV-D): the hand-worked fixture and seeded
per-kernel graphs with streams.  The generators hold no packing arithmetic."""
from __future__ import annotations

import json
import os

import numpy as np

from paper_2607_12324_amd import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def load_golden():
    with open(os.path.join(HERE, "golden", "handworked_packing.json")) as f:
        d = json.load(f)
    e = np.asarray(d["edges"], dtype=np.int32)
    g = synth.Graph(name="handworked-packing", num_nodes=len(d["node_pack"]),
                    edge_src=e[:, 0].copy(), edge_dst=e[:, 1].copy(),
                    node_pack=np.asarray(d["node_pack"], dtype=np.int32),
                    node_duration=np.asarray(d["node_duration"], dtype=np.float32),
                    num_packs=len(d["pack_time"]), num_levels=2,
                    pack_time=np.asarray(d["pack_time"], dtype=np.float32),
                    pack_energy=np.asarray(d["pack_energy"], dtype=np.float32),
                    static_power=float(d["static_power"]),
                    node_stream=np.asarray(d["node_stream"], dtype=np.int32))
    return d, g


def stream_dag(seed: int, kernels: int, streams: int, F: int = 4, comm_p: float = 0.15,
               cross_p: float = 0.2, host: bool = True, host_us: float = 2.0) -> synth.Graph:
    """Kernels (single-kernel packs) and communication nodes (fixed duration) in launch order on
    `streams` streams, each stream a chain in launch order; cross-stream edges from a random
    earlier node on another stream; optionally a host chain launching every kernel.  Durations
    on the 1/16 us grid."""
    rng = np.random.default_rng(seed)
    b = synth._Builder()
    last_on = {}
    prev_host = None
    t, e = synth.pack_tables(rng, kernels, F, 8.0, 1.0)
    fixed = []
    k = 0
    while k < kernels:
        s = int(rng.integers(0, streams))
        if rng.random() < comm_p:
            v = b.node(-1, s)
            fixed.append(float(synth.quantize(rng.lognormal(np.log(6.0), 1.0))))
        else:
            if host:
                h = b.node(-1, -1)
                fixed.append(float(synth.quantize(rng.lognormal(np.log(host_us), 0.5))))
                if prev_host is not None:
                    b.edge(prev_host, h)
                prev_host = h
            v = b.node(k, s)
            if host:
                b.edge(h, v)
            k += 1
        if s in last_on:
            b.edge(last_on[s], v)
        if rng.random() < cross_p:
            others = [u for u in range(v) if b.stream_of[u] >= 0 and b.stream_of[u] != s]
            if others:
                b.edge(int(others[int(rng.integers(0, len(others)))]), v)
        last_on[s] = v
    return synth._finish(b, f"streamdag-{seed}", np.asarray(fixed, dtype=np.float32), t, e)


def random_cases():
    """(name, graph, max_pack_duration) for the parity and invariant tests."""
    out = []
    for seed in range(12):
        S = 1 + seed % 4
        g = stream_dag(seed, 20 + 7 * seed, S, F=3 + seed % 3, host=seed % 3 != 0,
                       host_us=[0.5, 2.0, 20.0][seed % 3])
        out.append((g.name, g, [1e9, 40.0, 15.0][seed % 3]))
    for k in (1, 2, 3, 4):
        g = synth.config_graph(k)
        out.append((g.name, g, 5000.0))
    out.append(("launch-256k-4s", synth._launch_graph(11, "launch-256k-4s", P=256, S=4, F=8,
                                                      packs_per_host=1, cross_p=0.05,
                                                      n_cross_exact=None, median_us=50.0,
                                                      sigma=1.0), 300.0))
    return out
