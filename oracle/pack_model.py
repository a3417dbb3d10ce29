"""CPU oracle for the microbenchmark pack model -- TEST INFRASTRUCTURE ONLY.

Sec. IV-E (pack modelling): a pack's metric vector b (measured at the default frequency) is
decomposed into non-negative weights x over the microbenchmark suite by non-negative least
squares against the suite's metric matrix B (Eq. 6), and the pack's latency and energy at every
frequency are the weighted sums of the suite's (Eq. 7).

The NNLS step takes SciPy's solver as a candidate and accepts it only with the optimality
certificate of the problem (the KKT conditions: x >= 0, gradient B^T (b - Bx) <= 0, and 0 where
x > 0).  SciPy 1.15's solver returned uncertified points on rank-deficient suites (fewer metrics
than benchmarks, where it also misreported the residual), so an uncertified candidate is
replaced by the definition itself: the unconstrained least-squares solution on every subset of
the benchmarks, keeping the non-negative one of least residual (an optimal point with linearly
independent support always exists).  The sums of Eq. 7 are plain double loops in benchmark
order, rounded to fp32 at the end.  Inputs are the fp32 arrays the library takes, converted
exactly to double.
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import nnls


def kkt_ok(B, b, x, rel: float = 1e-9) -> bool:
    """The optimality certificate of min ||Bx - b|| subject to x >= 0."""
    B = np.asarray(B, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    w = B.T @ (b - B @ x)
    scale = rel * max(1.0, np.abs(B).sum()) * max(1.0, float(np.abs(b).max(initial=0.0)))
    return bool((x >= 0).all() and (w <= scale).all() and (np.abs(w[x > 0]) <= scale).all())


def enumerate_active_sets(B, b):
    """Least residual over every subset's non-negative least-squares solution."""
    B = np.asarray(B, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    m = B.shape[1]
    best_r, best_x = float(np.linalg.norm(b)), np.zeros(m)
    for mask in range(1, 1 << m):
        S = [i for i in range(m) if mask >> i & 1]
        z = np.linalg.lstsq(B[:, S], b, rcond=None)[0]
        if (z >= 0).all():
            x = np.zeros(m)
            x[S] = z
            r = float(np.linalg.norm(B @ x - b))
            if r < best_r:
                best_r, best_x = r, x
    return best_x, best_r


def fit_pack(metric_matrix, pack_metric_row):
    """Weights x (Eq. 6) and the residual norm ||Bx - b||."""
    B = np.asarray(metric_matrix, dtype=np.float64)
    b = np.asarray(pack_metric_row, dtype=np.float64)
    x, _ = nnls(B, b, maxiter=50 * B.shape[1])
    if not kkt_ok(B, b, x):
        x, _ = enumerate_active_sets(B, b)
    return x, float(np.linalg.norm(B @ x - b))


def predict(weights, bench_time, bench_energy):
    """Eq. 7: T_f = sum_i x_i T_f[B_i], E_f likewise, for every level f (fp32 results)."""
    m, F = np.asarray(bench_time).shape
    t = np.zeros(F, dtype=np.float32)
    e = np.zeros(F, dtype=np.float32)
    for f in range(F):
        st = 0.0
        se = 0.0
        for i in range(m):
            st += float(weights[i]) * float(bench_time[i, f])
            se += float(weights[i]) * float(bench_energy[i, f])
        t[f] = np.float32(st)
        e[f] = np.float32(se)
    return t, e


def pack_tables(metric_matrix, bench_time, bench_energy, pack_metrics):
    """Weights [P, m], latency and energy tables [P, F] and residual norms [P] of every pack."""
    P = int(np.asarray(pack_metrics).shape[0])
    m, F = np.asarray(bench_time).shape
    W = np.zeros((P, m))
    T = np.zeros((P, F), dtype=np.float32)
    E = np.zeros((P, F), dtype=np.float32)
    R = np.zeros(P)
    for p in range(P):
        W[p], R[p] = fit_pack(metric_matrix, pack_metrics[p])
        T[p], E[p] = predict(W[p], bench_time, bench_energy)
    return W, T, E, R
