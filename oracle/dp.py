"""CPU oracle for the policy search of Alg. 2 -- TEST INFRASTRUCTURE ONLY.

Follows Alg. 2 (Sec. IV-F) step by step, with one frequency interval per pack (the per-pack
reading of the policy, R1): the intervals [p_i, p_{i+1}) are the packs taken in `pack_order`,
and the predictor Pred is the oracle's fp64 evaluation of Alg. 1 (``oracle.eval_batch``).

Readings where the algorithm leaves a choice open (they are the library's as well):

* dp[i] is a map from the discretised makespan to one (energy, policy) pair.  The makespan t is
  discretised as floor(t / quantum), computed in double precision.
* Decisions are taken in fp32, the precision of the library's makespans and energies: the
  predictor's fp64 makespan and energy are rounded to fp32 first, then compared with the fp32
  latency target and with each other.
* "for each (t, (E, P)) in dp[i]" visits the stored states in increasing bucket order, and "for
  each f in F" the levels in increasing order.  The update takes a new pair only when its energy
  is strictly lower, so among equal energies the first candidate in that order stays.
* dp[0] holds the all-maximum policy P_0 whatever its makespan (the initialisation of Alg. 2
  does not test the constraint); the stages keep only policies with t <= T_max.
* The result is the least energy over the final states whose makespan meets T_max; among equal
  energies the lowest bucket wins.
"""
from __future__ import annotations

import math
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


def _f32(x) -> np.float32:
    return np.float32(x)


def dp_search(g, latency_target: float, quantum: float, pack_order=None,
              max_stages: int | None = None) -> DPResult:
    """Alg. 2 over the packs of `g` in `pack_order` (default: pack ids in increasing order).
    max_stages stops after that many stages (for timing a bounded sample)."""
    P, F = int(g.num_packs), int(g.num_levels)
    order = list(range(P)) if pack_order is None else [int(x) for x in pack_order]
    if sorted(order) != list(range(P)):
        raise ValueError("pack_order must be a permutation of the pack ids")
    t_max = _f32(latency_target)
    q = float(_f32(quantum))
    if not q > 0.0:
        raise ValueError("quantum must be positive")

    # P_0: the default (maximum) frequency in every interval; dp[0] = {t_0: (E_0, P_0)}
    p0 = np.full(P, F - 1, dtype=np.uint8)
    T0, E0 = eval_batch(g, p0[None, :])
    states = [(math.floor(float(_f32(T0[0])) / q), _f32(E0[0]), _f32(T0[0]), p0)]
    evaluated = 1

    for p in order[:max_stages]:
        # P' = P with frequency f in interval p, for every stored state and every f
        cands = []
        for (_, _, _, lv) in states:
            for f in range(F):
                lv2 = lv.copy()
                lv2[p] = f
                cands.append(lv2)
        if not cands:          # no state left: every later stage is empty too
            break
        Tc, Ec = eval_batch(g, np.stack(cands))
        evaluated += len(cands)
        nxt = {}
        for c, lv2 in enumerate(cands):
            t, e = _f32(Tc[c]), _f32(Ec[c])
            if not t <= t_max:
                continue
            b = math.floor(float(t) / q)
            if b not in nxt or e < nxt[b][0]:
                nxt[b] = (e, t, lv2)
        states = [(b,) + nxt[b] for b in sorted(nxt)]

    best = None
    for (b, e, t, lv) in states:
        if t <= t_max and (best is None or e < best[1]):
            best = (b, e, t, lv)
    n = sum(1 for s in states if s[2] <= t_max)
    if best is None:
        return DPResult(None, float("nan"), float("nan"), n, evaluated)
    return DPResult(best[3].copy(), float(best[1]), float(best[2]), n, evaluated)


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
    ok = T32 <= _f32(latency_target)
    if not ok.any():
        return None, float("nan"), float("nan")
    cand = np.nonzero(ok)[0]
    best = cand[np.argmin(E32[cand])]   # argmin returns the first (lowest index) minimum
    return rows[best].copy(), float(E32[best]), float(T32[best])
