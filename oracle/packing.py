"""CPU oracle for dependency-aware greedy kernel packing -- TEST INFRASTRUCTURE ONLY.

Follows Sec. IV-D (packing strategies): the critical predecessor of Eq. 5, the three rules
(dependency safety 1 and 2, granularity control) and the greedy pass over the kernels in
topological order; and, for the packed graph, the same section's statement that a pack keeps
only the incoming dependencies of its first kernel and the outgoing ones of its last.

Input: an execution graph in the form the evaluator loads (node_pack, per-pack tables), where
every GPU compute kernel is its own input pack, plus the stream of every node.  Output: the new
pack (group) of every input pack, and the contracted graph whose packs are those groups.

Readings where the section leaves a choice open (they are the library's as well):

* Default frequency = level F-1 (the maximum); a kernel's duration there is its table's last
  column.  Completion times C_k of Eq. 5 are the all-maximum schedule of Eq. 1 in double
  precision (``oracle.slack`` at the all-maximum row).
* Eq. 5's argmax takes the first maximal predecessor in the canonical topological order, as Alg. 1
  does with its strict comparison; the critical successors of u are the nodes whose critical
  predecessor is u.
* Packs are contiguous runs of kernels on one stream: kernels are visited in the canonical
  topological order and each stream has its own open pack.  A kernel v may join the open pack of
  its stream only if the pack's last kernel u is a direct predecessor of v (an edge u -> v), and
  then only if rule 1 (v and its critical predecessor share a stream), rule 2 (every critical
  successor of u is on u's stream) and rule 3 (the pack's default-frequency duration plus v's,
  summed in double in member order, stays strictly below max_pack_duration) all hold.
  Otherwise the open pack is closed and v opens a new one.
* A node's stream is an integer >= 0; -1 (host or other off-GPU nodes) equals no stream.
* Groups are numbered in the order their first kernels appear in the canonical order.
* Contraction: one packed node per non-kernel node and per group, numbered by increasing
  original id of the node that stands for it (a group: its first kernel).  An edge a -> b
  survives as rep(a) -> rep(b) when a is a non-kernel node or the last kernel of its group and b
  is a non-kernel node or the first kernel of its group, and rep(a) != rep(b); duplicates are
  merged and edges listed in increasing (src, dst) order.  A group's latency and energy at level
  f are the sums over its members, in member order, accumulated in double and rounded to fp32.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import slack, topo_order


class PackingError(ValueError):
    pass


@dataclass
class PackedGraph:
    """The contracted graph, in the field layout the evaluator loads."""
    name: str
    num_nodes: int
    edge_src: np.ndarray
    edge_dst: np.ndarray
    node_pack: np.ndarray
    node_duration: np.ndarray
    num_packs: int
    num_levels: int
    pack_time: np.ndarray
    pack_energy: np.ndarray
    static_power: float
    node_stream: np.ndarray
    packed_node: np.ndarray      # [V of the input] packed node standing for each input node

    @property
    def num_edges(self) -> int:
        return int(self.edge_src.shape[0])


def _kernel_of_pack(g):
    pk = np.asarray(g.node_pack)
    P = int(g.num_packs)
    node_of = np.full(P, -1, dtype=np.int64)
    for v in range(int(g.num_nodes)):
        p = int(pk[v])
        if p >= 0:
            if node_of[p] >= 0:
                raise PackingError(f"pack {p} is used by several nodes")
            node_of[p] = v
    if P and (node_of < 0).any():
        raise PackingError("a pack is used by no node")
    return node_of


def critical_links(g):
    """All-maximum completion times, the critical predecessor of every node (Eq. 5; -1 for a
    source) and the canonical position of every node."""
    F = int(g.num_levels)
    r = slack(g, np.full(int(g.num_packs), F - 1, dtype=np.uint8))
    order, _ = topo_order(g.num_nodes, g.edge_src, g.edge_dst)
    pos = np.empty(int(g.num_nodes), dtype=np.int64)
    pos[order] = np.arange(int(g.num_nodes))
    return r.eft, r.critical_pred, order, pos


def pack_kernels(g, node_stream, max_pack_duration: float):
    """Greedy dependency-aware packing: (group of every input pack [P] int32, number of groups)."""
    V = int(g.num_nodes)
    F = int(g.num_levels)
    stream = np.asarray(node_stream, dtype=np.int64)
    pk = np.asarray(g.node_pack)
    _kernel_of_pack(g)
    if any(stream[v] < 0 for v in range(V) if pk[v] >= 0):
        raise PackingError("every kernel needs a stream >= 0")
    limit = float(np.float32(max_pack_duration))
    _, cpred, order, _ = critical_links(g)

    preds = [set() for _ in range(V)]
    succs = [[] for _ in range(V)]
    for a, b in zip(np.asarray(g.edge_src).tolist(), np.asarray(g.edge_dst).tolist()):
        if b not in succs[a]:
            succs[a].append(b)
        preds[b].add(a)

    def default_duration(v):
        return float(g.pack_time[int(pk[v]), F - 1])

    def same_stream(a, b):
        return stream[a] >= 0 and stream[a] == stream[b]

    group = np.full(int(g.num_packs), -1, dtype=np.int32)
    open_pack = {}          # stream -> [group id, last kernel, accumulated duration]
    n_groups = 0
    for v in order.tolist():
        if pk[v] < 0:
            continue
        s = int(stream[v])
        cur = open_pack.get(s)
        t_v = default_duration(v)
        joins = False
        if cur is not None:
            gid, u, acc = cur
            adjacent = u in preds[v]
            r1 = cpred[v] >= 0 and same_stream(v, int(cpred[v]))
            r2 = all(same_stream(k, u) for k in succs[u] if cpred[k] == u)
            r3 = acc + t_v < limit
            joins = adjacent and r1 and r2 and r3
        if joins:
            group[pk[v]] = gid
            open_pack[s] = [gid, v, acc + t_v]
        else:
            group[pk[v]] = n_groups
            open_pack[s] = [n_groups, v, t_v]
            n_groups += 1
    return group, n_groups


def contract(g, group, num_groups: int, node_stream=None) -> PackedGraph:
    """The packed graph of a grouping of the input packs (see the module docstring)."""
    V = int(g.num_nodes)
    F = int(g.num_levels)
    pk = np.asarray(g.node_pack)
    group = np.asarray(group)
    _kernel_of_pack(g)
    _, _, order, pos = critical_links(g)

    members = [[] for _ in range(num_groups)]
    for v in order.tolist():
        if pk[v] >= 0:
            members[int(group[pk[v]])].append(v)
    if any(not m for m in members):
        raise PackingError("a group has no member")
    first = {m[0] for m in members}
    last = {m[-1] for m in members}

    reps = sorted([v for v in range(V) if pk[v] < 0] + [m[0] for m in members])
    new_id = {v: i for i, v in enumerate(reps)}
    packed_node = np.empty(V, dtype=np.int32)
    for v in range(V):
        packed_node[v] = new_id[v] if pk[v] < 0 else new_id[members[int(group[pk[v]])][0]]

    edges = set()
    for a, b in zip(np.asarray(g.edge_src).tolist(), np.asarray(g.edge_dst).tolist()):
        if pk[a] >= 0 and a not in last:
            continue
        if pk[b] >= 0 and b not in first:
            continue
        ra, rb = int(packed_node[a]), int(packed_node[b])
        if ra != rb:
            edges.add((ra, rb))
    edges = sorted(edges)

    n = len(reps)
    node_pack = np.full(n, -1, dtype=np.int32)
    node_duration = np.zeros(n, dtype=np.float32)
    stream_out = np.full(n, -1, dtype=np.int32)
    for v in reps:
        if pk[v] < 0:
            node_duration[new_id[v]] = g.node_duration[v]
        else:
            node_pack[new_id[v]] = group[pk[v]]
        if node_stream is not None:
            stream_out[new_id[v]] = node_stream[v]
    pt = np.zeros((num_groups, F), dtype=np.float32)
    pe = np.zeros((num_groups, F), dtype=np.float32)
    for gid, m in enumerate(members):
        for f in range(F):
            st = 0.0
            se = 0.0
            for v in m:
                st += float(g.pack_time[int(pk[v]), f])
                se += float(g.pack_energy[int(pk[v]), f])
            pt[gid, f] = np.float32(st)
            pe[gid, f] = np.float32(se)
    return PackedGraph(
        name=f"{getattr(g, 'name', 'graph')}-packed", num_nodes=n,
        edge_src=np.asarray([e[0] for e in edges], dtype=np.int32),
        edge_dst=np.asarray([e[1] for e in edges], dtype=np.int32),
        node_pack=node_pack, node_duration=node_duration, num_packs=int(num_groups),
        num_levels=F, pack_time=pt, pack_energy=pe, static_power=float(g.static_power),
        node_stream=stream_out, packed_node=packed_node)


def expand_levels(group, levels):
    """Kernel-level rows of packed-graph rows: every kernel takes its group's level."""
    levels = np.asarray(levels)
    return np.ascontiguousarray(levels[:, np.asarray(group)])
