"""CPU oracle for the policy search of Alg. 2 -- TEST INFRASTRUCTURE ONLY.

The search of Sec. IV-F written as a recurrence over makespan buckets, with one frequency
interval per pack (the per-pack reading of the policy, R1): the change points are the packs
taken in `pack_order`, and the predictor is the oracle's fp64 evaluation of Eq. 1-3
(``oracle.eval_batch``).

The state after i change points is a table over discretised end-to-end times: bucket t holds
the least energy found for a makespan in that bucket and the policy that reaches it.  Sec. IV-F
builds the table of stage i + 1 from that of stage i only:

    X_i      = every stored policy (in increasing bucket order) with interval i set to every
               level f (in increasing order): |dp[i]| x |F| candidates, evaluated by the
               predictor;
    dp[i+1]  = for each bucket t, the candidate of X_i with makespan in t and within the
               latency target of least energy.

dp[0] holds the all-maximum policy P_0.  The answer is the least-energy state of the last table.

Readings where the paper leaves a choice open (they are the library's as well):

* Buckets: floor(t / quantum), computed in double precision.
* Decisions are taken in fp32, the precision of the library's makespans and energies: the
  predictor's fp64 makespan and energy are rounded to fp32 first, then compared with the fp32
  latency target and with each other.
* Ties in the per-bucket minimum: the first candidate of X_i in the order above (a later one
  replaces a stored one only with strictly lower energy).  Ties in the answer: the lowest
  bucket.
* dp[0] holds P_0 whatever its makespan (the initialisation does not test the constraint); the
  later tables hold only policies with t <= T_max.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import eval_batch


@dataclass
class DPResult:
    levels: np.ndarray | None   # uint8 [P], None when no policy meets the target
    energy: float               # fp32 value, NaN when none
    makespan: float             # fp32 value, NaN when none
    num_states: int             # states stored after the last stage (with makespan <= T_max)
    evaluated: int = 0          # candidate policies evaluated (P_0 included)


@dataclass
class _Table:
    """One stage's states, sorted by bucket: bucket [S], energy [S] fp32, makespan [S] fp32,
    policies [S, P] uint8."""
    bucket: np.ndarray
    energy: np.ndarray
    makespan: np.ndarray
    policy: np.ndarray


def _predict(g, policies, quantum):
    """fp32 makespans and energies of the policies, and their buckets."""
    T, E = eval_batch(g, policies)
    T32, E32 = T.astype(np.float32), E.astype(np.float32)
    return T32, E32, np.floor(T32.astype(np.float64) / quantum).astype(np.int64)


def _expand(table: _Table, interval: int, F: int) -> np.ndarray:
    """X_i: each stored policy (bucket order) repeated with `interval` set to 0..F-1."""
    X = np.repeat(table.policy, F, axis=0)
    X[:, interval] = np.tile(np.arange(F, dtype=np.uint8), table.policy.shape[0])
    return X


def _least_per_bucket(X, T32, E32, bucket, t_max) -> _Table:
    """dp[i+1]: per bucket, the feasible candidate of least (energy, position in X)."""
    ok = np.nonzero(T32 <= t_max)[0]
    order = ok[np.lexsort((ok, E32[ok], bucket[ok]))]       # bucket, then energy, then position
    first = np.ones(order.size, dtype=bool)
    first[1:] = bucket[order][1:] != bucket[order][:-1]
    keep = order[first]
    return _Table(bucket[keep], E32[keep], T32[keep], X[keep])


def dp_search(g, latency_target: float, quantum: float, pack_order=None,
              max_stages: int | None = None) -> DPResult:
    """The search over the packs of `g` in `pack_order` (default: pack ids in increasing order).
    max_stages stops after that many stages (for timing a bounded sample)."""
    P, F = int(g.num_packs), int(g.num_levels)
    order = list(range(P)) if pack_order is None else [int(x) for x in pack_order]
    if sorted(order) != list(range(P)):
        raise ValueError("pack_order must be a permutation of the pack ids")
    t_max = np.float32(latency_target)
    q = float(np.float32(quantum))
    if not q > 0.0:
        raise ValueError("quantum must be positive")

    p0 = np.full((1, P), F - 1, dtype=np.uint8)
    T0, E0, b0 = _predict(g, p0, q)
    table = _Table(b0, E0, T0, p0)
    evaluated = 1
    for interval in order[:max_stages]:
        if table.policy.shape[0] == 0:       # nothing stored: every later table is empty too
            break
        X = _expand(table, interval, F)
        T32, E32, bucket = _predict(g, X, q)
        evaluated += X.shape[0]
        table = _least_per_bucket(X, T32, E32, bucket, t_max)

    ok = np.nonzero(table.makespan <= t_max)[0]
    if ok.size == 0:
        return DPResult(None, float("nan"), float("nan"), 0, evaluated)
    best = ok[np.lexsort((table.bucket[ok], table.energy[ok]))[0]]   # energy, then bucket
    return DPResult(table.policy[best].copy(), float(table.energy[best]),
                    float(table.makespan[best]), int(ok.size), evaluated)


def exhaustive_best(g, latency_target: float):
    """Least-energy policy with makespan <= target over the whole policy space F^P (tiny graphs
    only), decided in fp32 like dp_search; ties to the lowest mixed-radix index (pack 0 least
    significant).  Returns (levels or None, energy, makespan)."""
    P, F = int(g.num_packs), int(g.num_levels)
    n = F ** P
    idx = np.arange(n, dtype=np.int64)
    rows = np.empty((n, P), dtype=np.uint8)
    for p in range(P):
        rows[:, p] = (idx // (F ** p)) % F
    T, E = eval_batch(g, rows)
    T32, E32 = T.astype(np.float32), E.astype(np.float32)
    ok = T32 <= np.float32(latency_target)
    if not ok.any():
        return None, float("nan"), float("nan")
    cand = np.nonzero(ok)[0]
    best = cand[np.argmin(E32[cand])]   # argmin returns the first (lowest index) minimum
    return rows[best].copy(), float(E32[best]), float(T32[best])
