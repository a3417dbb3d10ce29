"""Seeded synthetic inputs: execution graphs, pack tables and candidate policies.

The paper evaluates on traces of real training and inference jobs (Sec. V-A) that are not
available here, and publishes no graph statistics.  This module builds seeded stand-ins with
the structure those traces have in Sec. IV-B: host (runtime-API) nodes in a launch chain,
launch edges from host nodes to GPU packs, stream-order chains of packs, cross-stream event
edges and all-stream synchronisation nodes.  Durations follow the distributions of the five
benchmark workloads (tiny, inference-like, training-like, large packed, unpacked per-kernel).

This module holds none of the method's arithmetic: no finish time, makespan, energy total,
slack or selection is computed here.  Both the HIP path and the oracle consume what it makes.

Conventions
-----------
* Time unit: microseconds.  Every duration and every table time lies on the dyadic grid
  ``Q = 2**-4`` us (round half to even, at least one grid step), so sums of them stay exact in
  fp32 while path lengths stay below ``2**20`` us.
* Level ``j`` in ``[0, F)`` runs at frequency ratio ``r_j = 0.5 + 0.5*j/(F-1)``; level ``F-1`` is
  the maximum frequency (1800 MHz-like), level 0 is half of it (900 MHz-like), matching the
  900-1800 MHz range of the paper's random-policy experiment (Sec. V-B).
* Pack latency ``t[p][j] = t_max*(a/r_j + 1 - a)`` with ``a ~ U(0,1)`` the frequency-sensitive
  share; pack energy is the dynamic part ``e[p][j] = C_DYN * r_j**3 * t[p][j]`` of the power model
  ``P(f) = Ps + c*(f/f_max)**3``; the static part ``Ps`` is charged over the whole makespan
  through ``static_power``.
* Node ids follow launch order, so every generated edge goes from a lower to a higher id.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Iterator

import numpy as np

Q = 1.0 / 16.0            # duration grid (us)
STATIC_POWER = 0.3        # Ps, power units (P(f_max) = Ps + C_DYN = 1)
C_DYN = 0.7               # dynamic power coefficient c
POLICY_CHUNK = 1 << 16    # rows generated per independently seeded chunk


@dataclasses.dataclass
class Graph:
    """Plain arrays describing one execution graph and its pack tables."""
    name: str
    num_nodes: int
    edge_src: np.ndarray        # int32 [E]
    edge_dst: np.ndarray        # int32 [E]
    node_pack: np.ndarray       # int32 [V], pack id or -1
    node_duration: np.ndarray   # float32 [V], used where node_pack == -1
    num_packs: int
    num_levels: int
    pack_time: np.ndarray       # float32 [P, F]
    pack_energy: np.ndarray     # float32 [P, F]
    static_power: float
    node_stream: np.ndarray | None = None   # int32 [V], -1 for host/sync nodes (informational)

    @property
    def num_edges(self) -> int:
        return int(self.edge_src.shape[0])


@dataclasses.dataclass(frozen=True)
class ConfigSpec:
    index: int
    name: str
    num_candidates: int
    targets: tuple          # latency-target ratios relative to the all-max makespan
    seed: int               # graph and table seed
    policy_seed: int
    exhaustive: bool = False
    slack: bool = False     # the workload includes the backward slack pass for every candidate


CONFIGS = {
    1: ConfigSpec(1, "tiny-8p-2s-F4", 4 ** 8, (1.05,), 0, 1000, exhaustive=True, slack=True),
    2: ConfigSpec(2, "inference-64p-1s-F8", 1 << 20, (1.05, 1.02), 1, 1001, slack=True),
    3: ConfigSpec(3, "training-512p-4s-F16", 1 << 22, (1.02, 1.05), 2, 1002),
    4: ConfigSpec(4, "packed-4096p-8s-F16", 1 << 18, (1.05,), 3, 1003, slack=True),
    5: ConfigSpec(5, "unpacked-65536k-16s-F16", 1 << 14, (1.05,), 4, 1004, slack=True),
}


def quantize(x) -> np.ndarray:
    """Round to the Q grid (half to even), at least one grid step, as float32."""
    v = np.maximum(Q, np.round(np.asarray(x, dtype=np.float64) / Q) * Q)
    return v.astype(np.float32)


def level_ratios(num_levels: int) -> np.ndarray:
    if num_levels == 1:
        return np.ones(1)
    return 0.5 + 0.5 * np.arange(num_levels) / (num_levels - 1)


def pack_tables(rng: np.random.Generator, num_packs: int, num_levels: int,
                median_us: float, sigma: float):
    """Per-pack latency/energy tables, non-increasing in level (faster at higher level)."""
    t_max = rng.lognormal(math.log(median_us), sigma, num_packs)
    a = rng.random(num_packs)
    r = level_ratios(num_levels)
    t = quantize(t_max[:, None] * (a[:, None] / r[None, :] + 1.0 - a[:, None]))
    e = (C_DYN * (r[None, :] ** 3) * t.astype(np.float64)).astype(np.float32)
    return t, e


def host_durations(rng: np.random.Generator, n: int) -> np.ndarray:
    return quantize(rng.lognormal(math.log(10.0), 0.5, n))


class _Builder:
    def __init__(self):
        self.pack_of: list[int] = []
        self.stream_of: list[int] = []
        self.src: list[int] = []
        self.dst: list[int] = []

    def node(self, pack: int = -1, stream: int = -1) -> int:
        self.pack_of.append(pack)
        self.stream_of.append(stream)
        return len(self.pack_of) - 1

    def edge(self, a: int, b: int) -> None:
        self.src.append(a)
        self.dst.append(b)


def _cross_source(rng, pack_node, pack_stream, p, s):
    """Uniformly random earlier pack on another stream than `s`, or None."""
    earlier = np.nonzero(pack_stream[:p] != s)[0]
    if earlier.size == 0:
        return None
    return int(pack_node[int(earlier[rng.integers(0, earlier.size)])])


def _finish(b: _Builder, name, durations_fixed, t, e, static_power=STATIC_POWER) -> Graph:
    V = len(b.pack_of)
    node_pack = np.asarray(b.pack_of, dtype=np.int32)
    dur = np.zeros(V, dtype=np.float32)
    fixed = np.nonzero(node_pack < 0)[0]
    dur[fixed] = durations_fixed
    src = np.asarray(b.src, dtype=np.int32)
    dst = np.asarray(b.dst, dtype=np.int32)
    # drop duplicates (a cross edge may repeat a stream edge); keep first-seen order
    key = src.astype(np.int64) * V + dst
    _, first = np.unique(key, return_index=True)
    keep = np.sort(first)
    return Graph(name=name, num_nodes=V, edge_src=src[keep], edge_dst=dst[keep],
                 node_pack=node_pack, node_duration=dur, num_packs=int(t.shape[0]),
                 num_levels=int(t.shape[1]), pack_time=np.ascontiguousarray(t),
                 pack_energy=np.ascontiguousarray(e), static_power=float(static_power),
                 node_stream=np.asarray(b.stream_of, dtype=np.int32))


def _launch_graph(seed, name, P, S, F, packs_per_host, cross_p, n_cross_exact,
                  median_us, sigma, stream_mod=False) -> Graph:
    """Host launch chain H_0 -> H_1 -> ..., each H_h launching `packs_per_host` packs;
    stream-order chains; cross-stream edges."""
    rng = np.random.default_rng(seed)
    if stream_mod:
        pack_stream = np.arange(P) % S
    else:
        pack_stream = rng.integers(0, S, P)
    # cross edges: target pack -> source pack
    cross = {}
    if n_cross_exact is not None:
        cand = [p for p in range(P) if np.any(pack_stream[:p] != pack_stream[p])]
        targets = rng.choice(np.asarray(cand), size=n_cross_exact, replace=False)
        for p in sorted(int(x) for x in targets):
            cross[p] = None
    else:
        hit = rng.random(P) < cross_p
        for p in np.nonzero(hit)[0]:
            cross[int(p)] = None
    H = P // packs_per_host
    hdur = host_durations(rng, H)
    t, e = pack_tables(rng, P, F, median_us, sigma)

    b = _Builder()
    pack_node = np.zeros(P, dtype=np.int64)
    last_on_stream = {}
    prev_host = None
    p = 0
    for h in range(H):
        hn = b.node()
        if prev_host is not None:
            b.edge(prev_host, hn)
        prev_host = hn
        for _ in range(packs_per_host):
            s = int(pack_stream[p])
            pn = b.node(pack=p, stream=s)
            pack_node[p] = pn
            b.edge(hn, pn)
            if s in last_on_stream:
                b.edge(last_on_stream[s], pn)
            last_on_stream[s] = pn
            p += 1
    # cross-stream event edges, drawn after the structure so the draw order is fixed
    for p in sorted(cross):
        src = _cross_source(rng, pack_node, pack_stream, p, int(pack_stream[p]))
        if src is not None:
            b.edge(src, int(pack_node[p]))
    return _finish(b, name, hdur, t, e)


def _packed_graph(seed, name, P=4096, S=8, F=16, sync_every=256, cross_p=0.03) -> Graph:
    """Packs on S streams with periodic all-stream synchronisation nodes; no host nodes."""
    rng = np.random.default_rng(seed)
    pack_stream = rng.integers(0, S, P)
    hit = rng.random(P) < cross_p
    n_sync = P // sync_every
    sdur = host_durations(rng, n_sync)
    t, e = pack_tables(rng, P, F, 50.0, 1.0)

    b = _Builder()
    pack_node = np.zeros(P, dtype=np.int64)
    last_on_stream: dict = {}
    last_sync = None
    for p in range(P):
        s = int(pack_stream[p])
        pn = b.node(pack=p, stream=s)
        pack_node[p] = pn
        if last_on_stream.get(s) is not None:
            b.edge(last_on_stream[s], pn)
        elif last_sync is not None:
            b.edge(last_sync, pn)
        last_on_stream[s] = pn
        if (p + 1) % sync_every == 0:
            sn = b.node()
            for s2 in range(S):
                if last_on_stream.get(s2) is not None:
                    b.edge(last_on_stream[s2], sn)
                last_on_stream[s2] = None
            last_sync = sn
    for p in np.nonzero(hit)[0]:
        src = _cross_source(rng, pack_node, pack_stream, int(p), int(pack_stream[p]))
        if src is not None:
            b.edge(src, int(pack_node[p]))
    return _finish(b, name, sdur, t, e)


def packed_graph(seed: int, P: int, S: int, F: int, sync_every: int = 256,
                 cross_p: float = 0.03, shuffle_pack_ids: bool = False) -> Graph:
    """A graph shaped like the large packed workload at another size: P packs on S streams with
    periodic all-stream synchronisation nodes and random cross-stream edges.  With
    shuffle_pack_ids the pack numbering is a random permutation (tables permuted with it)."""
    g = _packed_graph(seed, f"packed-{P}p-{S}s-F{F}", P=P, S=S, F=F, sync_every=sync_every,
                      cross_p=cross_p)
    if not shuffle_pack_ids:
        return g
    perm = np.random.default_rng(seed + 1).permutation(P)     # old id -> new id
    node_pack = g.node_pack.copy()
    m = node_pack >= 0
    node_pack[m] = perm[node_pack[m]]
    t = np.empty_like(g.pack_time)
    e = np.empty_like(g.pack_energy)
    t[perm] = g.pack_time
    e[perm] = g.pack_energy
    return dataclasses.replace(g, name=g.name + "-shuffled", node_pack=node_pack.astype(np.int32),
                               pack_time=t, pack_energy=e)


def stream_graph(seed: int, P: int, S: int, F: int, median_us: float = 8.0,
                 sigma: float = 1.2) -> Graph:
    """A graph shaped like the unpacked per-kernel workload at another size: P kernels on S
    streams, each launched by a node of one host launch chain, no cross-stream edges."""
    return _launch_graph(seed, f"streams-{P}k-{S}s-F{F}", P=P, S=S, F=F, packs_per_host=1,
                         cross_p=0.0, n_cross_exact=None, median_us=median_us, sigma=sigma)


def block_graph(rng, nblk: int, bypass_p: float, F: int = 16) -> Graph:
    """Blocks of 32 packs (random edges from earlier to later packs of the block), each closed by
    a synchronisation node that waits for the block's sinks and starts the next block's sources;
    with probability bypass_p a fixed node runs from a pack of the previous block to a pack of
    the next one beside the synchronisation, which then is no cut."""
    src, dst, pack, dur = [], [], [], []

    def node(p=-1, d=0.0):
        pack.append(p)
        dur.append(d)
        return len(pack) - 1

    prev_sync, prev_ids = None, None
    for b in range(nblk):
        ids = [node(32 * b + i) for i in range(32)]
        has_in, has_out = [False] * 32, [False] * 32
        for i in range(1, 32):
            for _ in range(int(rng.integers(0, 3))):
                j = int(rng.integers(0, i))
                src.append(ids[j]); dst.append(ids[i])
                has_in[i] = has_out[j] = True
        if prev_sync is not None:
            for i in range(32):
                if not has_in[i]:
                    src.append(prev_sync); dst.append(ids[i])
            if rng.random() < bypass_p:
                x = node(-1, 0.5)
                src += [prev_ids[int(rng.integers(0, 32))], x]
                dst += [x, ids[int(rng.integers(0, 32))]]
        s = node(-1, float(quantize(rng.uniform(1.0, 5.0))))
        for i in range(32):
            if not has_out[i]:
                src.append(ids[i]); dst.append(s)
        prev_sync, prev_ids = s, ids
    P = 32 * nblk
    t = quantize(rng.uniform(1.0, 9.0, (P, F))).astype(np.float32)
    return Graph(f"blocks-{nblk}", len(pack), np.asarray(src, np.int32), np.asarray(dst, np.int32),
                       np.asarray(pack, np.int32), np.asarray(dur, np.float32), P, F, t,
                       (0.5 * t).astype(np.float32), 0.25)


def config_graph(k: int) -> Graph:
    """The execution graph and tables of benchmark workload `k` (1..5)."""
    spec = CONFIGS[k]
    if k == 1:
        return _launch_graph(spec.seed, spec.name, P=8, S=2, F=4, packs_per_host=2,
                             cross_p=None, n_cross_exact=2, median_us=50.0, sigma=1.0,
                             stream_mod=True)
    if k == 2:
        return _launch_graph(spec.seed, spec.name, P=64, S=1, F=8, packs_per_host=1,
                             cross_p=0.0, n_cross_exact=None, median_us=50.0, sigma=1.0)
    if k == 3:
        return _launch_graph(spec.seed, spec.name, P=512, S=4, F=16, packs_per_host=1,
                             cross_p=0.05, n_cross_exact=None, median_us=50.0, sigma=1.0)
    if k == 4:
        return _packed_graph(spec.seed, spec.name)
    if k == 5:
        return _launch_graph(spec.seed, spec.name, P=65536, S=16, F=16, packs_per_host=1,
                             cross_p=0.0, n_cross_exact=None, median_us=8.0, sigma=1.2)
    raise ValueError(f"unknown config {k}")


def without_cuts(g: Graph) -> Graph:
    """The same graph plus a zero-duration source node into the node of the last pack: no node
    before that pack is a cut node any more (the new node is neither before nor after it)."""
    v = int(np.nonzero(g.node_pack == g.num_packs - 1)[0][0])
    V = g.num_nodes
    return dataclasses.replace(
        g, name=g.name + "-nocut", num_nodes=V + 1,
        edge_src=np.append(g.edge_src, np.int32(V)).astype(np.int32),
        edge_dst=np.append(g.edge_dst, np.int32(v)).astype(np.int32),
        node_pack=np.append(g.node_pack, np.int32(-1)).astype(np.int32),
        node_duration=np.append(g.node_duration, np.float32(0)).astype(np.float32),
        node_stream=None if g.node_stream is None else np.append(g.node_stream, np.int32(-1)).astype(np.int32))


def scaled_times(g: Graph, factor: float) -> Graph:
    """The same graph with every table time multiplied by `factor` (rounded to fp32): 1.1 takes
    the times off any common power-of-two grid, as durations measured in integer nanoseconds
    are."""
    return dataclasses.replace(g, name=f"{g.name}-t{factor:g}",
                               pack_time=(g.pack_time * np.float32(factor)).astype(np.float32))


# ----------------------------------------------------------------------------- policies

def exhaustive_policies(num_packs: int, num_levels: int, start: int, count: int) -> np.ndarray:
    """Rows start..start+count of the full policy space in mixed radix, pack 0 least significant."""
    c = np.arange(start, start + count, dtype=np.int64)
    out = np.empty((count, num_packs), dtype=np.uint8)
    for p in range(num_packs):
        out[:, p] = (c // (num_levels ** p)) % num_levels
    return out


def _chunk(seed: int, chunk: int, rows: int, P: int, F: int, dist: str) -> np.ndarray:
    rng = np.random.default_rng([seed, chunk])
    if F == 1:
        return np.zeros((rows, P), dtype=np.uint8)
    if dist == "uniform":
        return rng.integers(0, F, size=(rows, P), dtype=np.uint8)
    if dist != "mixture":
        raise ValueError(dist)
    # mixture: candidate c lowers each pack independently with probability rho_c ~ U(0,1) to a
    # uniform level in [0, F-2], else keeps it at F-1.  Each (candidate, pack) draws one 32-bit
    # word: its high half against rho_c (16-bit fixed point) decides whether to lower, its low
    # half picks the lowered level.
    thresh = (rng.random(rows) * 65536.0).astype(np.uint32)
    out = np.empty((rows, P), dtype=np.uint8)
    sub = 512
    for s in range(0, rows, sub):
        n = min(sub, rows - s)
        u = np.frombuffer(rng.bytes(n * P * 4), dtype=np.uint32).reshape(n, P)
        low = (((u & np.uint32(0xFFFF)) * np.uint32(F - 1)) >> np.uint32(16)).astype(np.uint8)
        keep = (u >> np.uint32(16)) >= thresh[s:s + n, None]
        np.maximum(low, keep.view(np.uint8) * np.uint8(F - 1), out=out[s:s + n])
    return out


def random_policies(seed: int, num_packs: int, num_levels: int, start: int, count: int,
                    dist: str = "mixture") -> np.ndarray:
    """Rows start..start+count of a seeded policy batch; row 0 is the all-max policy."""
    out = np.empty((count, num_packs), dtype=np.uint8)
    r = start
    while r < start + count:
        ch = r // POLICY_CHUNK
        lo = ch * POLICY_CHUNK
        hi = min(lo + POLICY_CHUNK, start + count)
        blk = _chunk(seed, ch, POLICY_CHUNK, num_packs, num_levels, dist)
        out[r - start:hi - start] = blk[r - lo:hi - lo]
        r = hi
    if start == 0 and count > 0:
        out[0, :] = num_levels - 1
    return out


def _chunk_job(args):
    seed, ch, P, F, dist = args
    return ch, _chunk(seed, ch, POLICY_CHUNK, P, F, dist)


def random_policies_parallel(seed: int, num_packs: int, num_levels: int, count: int,
                             dist: str = "mixture", workers: int = 8) -> np.ndarray:
    """Rows 0..count of random_policies(...) generated by a pool of worker processes (spawned,
    so that a parent that already holds a GPU context is never forked)."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor
    out = np.empty((count, num_packs), dtype=np.uint8)
    nch = (count + POLICY_CHUNK - 1) // POLICY_CHUNK
    if nch <= 2 or workers <= 1:
        return random_policies(seed, num_packs, num_levels, 0, count, dist)
    jobs = [(seed, ch, num_packs, num_levels, dist) for ch in range(nch)]
    with ProcessPoolExecutor(max_workers=min(workers, nch),
                             mp_context=mp.get_context("spawn")) as ex:
        for ch, blk in ex.map(_chunk_job, jobs):
            lo = ch * POLICY_CHUNK
            hi = min(lo + POLICY_CHUNK, count)
            out[lo:hi] = blk[:hi - lo]
    if count > 0:
        out[0, :] = num_levels - 1
    return out


def iter_policy_chunks(k: int, graph: Graph, dist: str = "mixture",
                       rows: int | None = None) -> Iterator[tuple[int, np.ndarray]]:
    """Yield (start_row, block) over the whole candidate batch of workload `k`."""
    spec = CONFIGS[k]
    B = spec.num_candidates if rows is None else rows
    step = POLICY_CHUNK
    for s in range(0, B, step):
        n = min(step, B - s)
        yield s, config_policies(k, graph, s, n, dist)


def config_policies(k: int, graph: Graph, start: int = 0, count: int | None = None,
                    dist: str = "mixture") -> np.ndarray:
    spec = CONFIGS[k]
    if count is None:
        count = spec.num_candidates - start
    if spec.exhaustive:
        return exhaustive_policies(graph.num_packs, graph.num_levels, start, count)
    return random_policies(spec.policy_seed, graph.num_packs, graph.num_levels, start, count, dist)


def bench_policies(k: int, graph: Graph, workers: int = 8) -> np.ndarray:
    """The whole candidate batch of workload `k` as the benchmark step evaluates it, all-max
    policy first: the tiny workload's exhaustive space in reverse mixed-radix order, the others'
    seeded mixture batch."""
    spec = CONFIGS[k]
    if spec.exhaustive:
        return np.ascontiguousarray(config_policies(k, graph)[::-1])
    return random_policies_parallel(spec.policy_seed, graph.num_packs, graph.num_levels,
                                    spec.num_candidates, workers=workers)


def sample_rows(num_candidates: int, n: int, seed: int = 7) -> np.ndarray:
    """A seeded sample of candidate rows that always includes the first and last rows."""
    rng = np.random.default_rng(seed)
    n = min(n, num_candidates)
    rows = set([0, num_candidates - 1])
    if num_candidates > 2:
        rows.update(int(x) for x in rng.choice(num_candidates, size=n, replace=False))
    return np.asarray(sorted(rows), dtype=np.int64)


# ----------------------------------------------------------------------------- small graphs

def random_dag(rng: np.random.Generator, num_nodes: int, edge_prob: float, pack_frac: float,
               num_levels: int, on_grid: bool = True, shuffle_ids: bool = True,
               shuffle_packs: bool = True, name: str = "random") -> Graph:
    """A random DAG with random node numbering and pack numbering.

    Tables are non-increasing in level.  With `on_grid` every time is a multiple of Q.
    """
    V = num_nodes
    order = rng.permutation(V) if shuffle_ids else np.arange(V)
    src, dst = [], []
    for i in range(V):
        for j in range(i + 1, V):
            if rng.random() < edge_prob:
                src.append(int(order[i]))
                dst.append(int(order[j]))
    is_pack = rng.random(V) < pack_frac
    pack_nodes = np.nonzero(is_pack)[0]
    P = int(pack_nodes.size)
    pids = rng.permutation(P) if shuffle_packs else np.arange(P)
    node_pack = np.full(V, -1, dtype=np.int32)
    node_pack[pack_nodes] = pids
    if on_grid:
        dur = quantize(rng.uniform(0.5, 40.0, V))
        raw = rng.uniform(0.5, 60.0, (P, num_levels))
        t = np.sort(quantize(raw), axis=1)[:, ::-1].copy()
    else:
        dur = rng.uniform(0.1, 40.0, V).astype(np.float32)
        t = np.sort(rng.uniform(0.1, 60.0, (P, num_levels)).astype(np.float32), axis=1)[:, ::-1].copy()
    dur[node_pack >= 0] = 0.0
    e = np.sort(rng.uniform(0.0, 5.0, (P, num_levels)).astype(np.float32), axis=1).copy()
    return Graph(name=name, num_nodes=V, edge_src=np.asarray(src, dtype=np.int32),
                 edge_dst=np.asarray(dst, dtype=np.int32), node_pack=node_pack,
                 node_duration=dur.astype(np.float32), num_packs=P, num_levels=num_levels,
                 pack_time=np.ascontiguousarray(t, dtype=np.float32),
                 pack_energy=np.ascontiguousarray(e, dtype=np.float32),
                 static_power=float(np.float32(rng.uniform(0.0, 1.0))))


MODEL_METRICS = 16      # metrics per pack (counter groups, read and write split)
MODEL_BENCHMARKS = 12   # microbenchmarks in the proxy suite


@dataclasses.dataclass
class ModelInputs:
    """Inputs of the microbenchmark pack model: the metric matrix of the suite (metrics x
    benchmarks, each metric row scaled to a maximum of 1), the suite's latency and energy at
    every level, and the metric vector of every pack (a non-negative mix of the suite plus
    noise)."""
    metric_matrix: np.ndarray    # float32 [n, m]
    bench_time: np.ndarray       # float32 [m, F]
    bench_energy: np.ndarray     # float32 [m, F]
    pack_metrics: np.ndarray     # float32 [P, n]
    true_weights: np.ndarray     # float64 [P, m] (the mix before noise)


def model_inputs(seed: int, num_packs: int, num_levels: int, n: int = MODEL_METRICS,
                 m: int = MODEL_BENCHMARKS, noise: float = 0.02) -> ModelInputs:
    rng = np.random.default_rng(seed)
    B = rng.lognormal(0.0, 1.0, (n, m)) * (rng.random((n, m)) < 0.6)
    B[rng.integers(0, n, m), np.arange(m)] += 1.0       # every benchmark touches some metric
    B /= B.max(axis=1, keepdims=True).clip(min=1e-30)
    t, _ = pack_tables(rng, m, num_levels, 200.0, 0.5)
    r = level_ratios(num_levels)
    e = ((STATIC_POWER + C_DYN * r[None, :] ** 3) * t.astype(np.float64)).astype(np.float32)
    w = rng.exponential(1.0, (num_packs, m)) * (rng.random((num_packs, m)) < 0.4)
    w[np.arange(num_packs), rng.integers(0, m, num_packs)] += 0.5
    b = (w @ B.T) * rng.lognormal(0.0, noise, (num_packs, n))
    return ModelInputs(B.astype(np.float32), t, e, b.astype(np.float32), w)
