"""Comparison rules between the HIP path and the oracle.

* Makespan and slack: on the fp32-exact grid (every workload here) they are compared bit for
  bit; otherwise |diff| <= 1e-5 * makespan.
* Energy: |diff| <= 1e-5 * energy.  The library's bound is below 4e-6: fp32 partial sums of at
  most 64 nonnegative terms (relative error <= 63 * 2^-24) added in fp64, one fp32 rounding of
  the total and one of static_power * T.
* Feasibility masks: bit-exact (times are exact, and the same fp32 target is used by both).
* Selection: the index must match exactly unless another feasible candidate's oracle energy is
  within 1e-5 of the best; then any such candidate is accepted.
"""
from __future__ import annotations

import numpy as np

import oracle

REL = 1e-5


def assert_eval(T, E, T_or, E_or, exact=True, what=""):
    T = np.asarray(T, dtype=np.float64)
    E = np.asarray(E, dtype=np.float64)
    nan = np.isnan(T_or)
    assert np.array_equal(np.isnan(T), nan), f"{what}: NaN pattern of makespan differs"
    assert np.array_equal(np.isnan(E), np.isnan(E_or)), f"{what}: NaN pattern of energy differs"
    ok = ~nan
    if exact:
        bad = np.nonzero(T[ok] != T_or[ok])[0]
        assert bad.size == 0, f"{what}: makespan differs at {bad[:5]}: {T[ok][bad[:5]]} vs {T_or[ok][bad[:5]]}"
    else:
        err = np.abs(T[ok] - T_or[ok])
        assert np.all(err <= REL * np.abs(T_or[ok])), f"{what}: makespan rel err {np.max(err / np.maximum(T_or[ok], 1e-30))}"
    e_ok = ~np.isnan(E_or)
    err = np.abs(E[e_ok] - E_or[e_ok])
    lim = REL * np.abs(E_or[e_ok])
    worst = int(np.argmax(err - lim)) if err.size else 0
    assert np.all(err <= lim), f"{what}: energy err {err[worst]} > {lim[worst]}"


def assert_slack(S, S_or, T_or, exact=True, what=""):
    S = np.asarray(S, dtype=np.float64)
    S_or = np.asarray(S_or, dtype=np.float64)
    assert S.shape == S_or.shape
    nan = np.isnan(S_or)
    assert np.array_equal(np.isnan(S), nan), f"{what}: NaN pattern of slack differs"
    ok = ~nan
    if exact:
        bad = np.argwhere(S != S_or)
        bad = [b for b in bad if ok[tuple(b)]]
        assert not bad, f"{what}: slack differs at {bad[:5]}"
    else:
        tol = REL * np.abs(np.asarray(T_or, dtype=np.float64))[:, None]
        err = np.where(ok, np.abs(S - S_or), 0.0)
        assert np.all(err <= tol), f"{what}: slack err {err.max()}"


def assert_selection(sel, mask_bits, T_or, E_or, target, exact_mask=True, what=""):
    idx_or, feas_or, n_or = oracle.select(T_or, E_or, target)
    if exact_mask:
        assert sel.num_feasible == n_or, f"{what}: feasible count {sel.num_feasible} vs {n_or}"
        if mask_bits is not None:
            diff = np.nonzero(mask_bits != feas_or)[0]
            assert diff.size == 0, f"{what}: mask differs at {diff[:5]}"
    if idx_or < 0:
        assert sel.index == -1, f"{what}: expected no selection, got {sel.index}"
        assert np.isnan(sel.energy) and np.isnan(sel.makespan)
        return
    best = E_or[idx_or]
    near = feas_or & (np.abs(E_or - best) <= REL * best)
    if int(near.sum()) == 1:
        assert sel.index == idx_or, f"{what}: selected {sel.index}, oracle {idx_or}"
    else:
        assert 0 <= sel.index < len(T_or) and near[sel.index], \
            f"{what}: selected {sel.index} is not within tolerance of the oracle's best {idx_or}"
    assert abs(sel.energy - E_or[sel.index]) <= REL * E_or[sel.index]
    assert abs(sel.makespan - T_or[sel.index]) <= REL * T_or[sel.index]
