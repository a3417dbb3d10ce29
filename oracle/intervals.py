"""CPU oracle for time-interval frequency policies -- TEST INFRASTRUCTURE ONLY.

A policy in the paper's general form (Sec. IV-A, the policy P = {<T_i, F_i>} of the optimisation
problem; Alg. 1) is a list of change points with one frequency each.  Here the change points are
shared by all candidates of a batch and each candidate gives the level of every interval:

* interval i is [T_i, T_{i+1}) with T_0 = 0 and T_K = infinity (half-open, as in Alg. 1's
  lookup; the closed interval of the problem statement would give a start that equals a change
  point two intervals);
* a pack runs at the level of the interval that contains its start time (the largest finish
  time among its predecessors, 0 for a source; Eq. 1 and Alg. 1), so a pack's level depends on
  the schedule;
* makespan as in Eq. 1-2; energy = the packs' table energies + the idle term of Alg. 1, read as
  each interval's idle power p_idle[F_i] times the wall time the interval covers inside
  [0, makespan).  With one idle power for every level this is the static_power * makespan term
  of the per-pack evaluation, which is how that reading generalises it;
* a level byte >= F anywhere in a candidate's row makes its makespan and energy NaN.

Plain double precision over the fp32 inputs, one candidate at a time in the oracle's own
topological order (``oracle.topo_order``).  Pure Python: for small batches and sampled rows.
"""
from __future__ import annotations

import bisect

import numpy as np

from . import topo_order


class IntervalError(ValueError):
    pass


def check_policy(num_levels, change_points, idle_power):
    pts = [float(np.float32(x)) for x in change_points]
    if any(not np.isfinite(x) or x <= 0.0 for x in pts):
        raise IntervalError("change points must be finite and positive")
    if any(b <= a for a, b in zip(pts, pts[1:])):
        raise IntervalError("change points must increase strictly")
    idle = [float(np.float32(x)) for x in idle_power]
    if len(idle) != num_levels or any(not np.isfinite(x) or x < 0.0 for x in idle):
        raise IntervalError("idle_power needs one finite value >= 0 per level")
    return pts, idle


def interval_of(pts, t):
    """Index of the interval [T_i, T_{i+1}) holding time t >= 0 (T_0 = 0)."""
    return bisect.bisect_right(pts, t)


def idle_energy(pts, idle, row, T):
    """Sum over intervals of p_idle[F_i] * |[T_i, T_{i+1}) inside [0, T)|."""
    lo = [0.0] + pts
    hi = pts + [float("inf")]
    e = 0.0
    for i in range(len(lo)):
        span = min(T, hi[i]) - lo[i]
        if span > 0.0:
            e += idle[int(row[i])] * span
    return e


def eval_intervals(g, change_points, levels, idle_power):
    """Makespan and energy (float64 [B]) of each row of `levels` ([B, K] uint8, K = number of
    change points + 1)."""
    pts, idle = check_policy(int(g.num_levels), change_points, idle_power)
    K = len(pts) + 1
    lv = np.asarray(levels, dtype=np.uint8).reshape(-1, K)
    V, F = int(g.num_nodes), int(g.num_levels)
    order, _ = topo_order(V, g.edge_src, g.edge_dst)
    preds = [[] for _ in range(V)]
    for s, d in zip(np.asarray(g.edge_src), np.asarray(g.edge_dst)):
        preds[int(d)].append(int(s))
    pack = [int(x) for x in np.asarray(g.node_pack)]
    dur = [float(x) for x in np.asarray(g.node_duration, dtype=np.float32)]
    tt = np.asarray(g.pack_time, dtype=np.float32).astype(np.float64)
    te = np.asarray(g.pack_energy, dtype=np.float32).astype(np.float64)
    B = lv.shape[0]
    T = np.empty(B)
    E = np.empty(B)
    for c in range(B):
        row = lv[c]
        if (row >= F).any():
            T[c] = E[c] = np.nan
            continue
        eft = [0.0] * V
        ea = 0.0
        for v in order:
            start = max((eft[k] for k in preds[v]), default=0.0)
            p = pack[v]
            if p >= 0:
                f = int(row[interval_of(pts, start)])
                d = tt[p, f]
                ea += te[p, f]
            else:
                d = dur[v]
            eft[v] = start + d
        T[c] = max(eft, default=0.0)
        E[c] = ea + idle_energy(pts, idle, row, T[c])
    return T, E
