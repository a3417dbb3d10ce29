"""Pins of the microbenchmark pack-model oracle (Sec. IV-E, Eq. 6-7), on the CPU: exact recovery
of a non-negative mix, the optimality (KKT) certificate of NNLS on full-rank and rank-deficient
suites, brute force over every active set on small suites, the unconstrained least-squares
solution when it is positive, and a pack equal to twice one benchmark."""
import itertools

import numpy as np
import pytest

from oracle import pack_model as pm
from paper_2607_12324_amd import synth


def _problem(seed, n, m):
    rng = np.random.default_rng(seed)
    B = rng.lognormal(0.0, 1.0, (n, m)).astype(np.float32)
    bt = synth.quantize(rng.uniform(10, 400, (m, 5)))
    be = (bt * rng.uniform(0.2, 1.0, (m, 5))).astype(np.float32)
    return rng, B, bt, be


def test_exact_recovery():
    for seed in range(10):
        rng, B, bt, be = _problem(seed, 16, 12)
        x_true = rng.exponential(1.0, 12) * (rng.random(12) < 0.5)
        b = B.astype(np.float64) @ x_true
        x, res = pm.fit_pack(B, b)
        assert np.allclose(x, x_true, atol=1e-9 * max(1.0, x_true.max())) and res < 1e-9 * np.linalg.norm(b)


def test_kkt_certificate():
    """x >= 0, the gradient B^T (b - Bx) is <= 0 everywhere and 0 where x > 0."""
    mi = synth.model_inputs(1, 64, 8)
    B = mi.metric_matrix.astype(np.float64)
    scale = np.abs(B).sum() * np.abs(mi.pack_metrics).max()
    for b in mi.pack_metrics.astype(np.float64):
        x, _ = pm.fit_pack(B, b)
        w = B.T @ (b - B @ x)
        assert (x >= 0).all()
        assert (w <= 1e-10 * scale).all()
        assert np.all(np.abs(w[x > 0]) <= 1e-10 * scale)


def test_kkt_certificate_rank_deficient():
    """Fewer metrics than benchmarks: the oracle's point is certified and no subset does
    better (a point SciPy's solver alone got wrong: pack 16 of this batch)."""
    mi = synth.model_inputs(5, 128, 6, n=8, m=12)
    B = mi.metric_matrix.astype(np.float64)
    for p in (16, 0, 5):
        b = mi.pack_metrics[p].astype(np.float64)
        x, res = pm.fit_pack(B, b)
        assert pm.kkt_ok(B, b, x)
        assert abs(res - np.linalg.norm(B @ x - b)) <= 1e-12
    b16 = mi.pack_metrics[16].astype(np.float64)
    x, res = pm.fit_pack(B, b16)
    _, best = pm.enumerate_active_sets(B, b16)
    assert abs(res - best) <= 1e-9
    raw, _ = pm.nnls(B, b16, maxiter=600)
    print("SciPy's point certified:", pm.kkt_ok(B, b16, raw))


def test_brute_force_active_sets():
    """The least residual over every subset's unconstrained solution that is non-negative."""
    for seed in range(6):
        rng, B, _, _ = _problem(100 + seed, 9, 6)
        b = rng.lognormal(0.0, 1.0, 9)
        Bd = B.astype(np.float64)
        best = (np.linalg.norm(b), np.zeros(6))
        for k in range(1, 7):
            for S in itertools.combinations(range(6), k):
                z = np.linalg.lstsq(Bd[:, S], b, rcond=None)[0]
                if (z >= 0).all():
                    x = np.zeros(6)
                    x[list(S)] = z
                    r = np.linalg.norm(Bd @ x - b)
                    if r < best[0] - 1e-12:
                        best = (r, x)
        x, res = pm.fit_pack(B, b)
        assert abs(res - best[0]) <= 1e-9 * np.linalg.norm(b)
        assert np.allclose(x, best[1], atol=1e-8)


def test_positive_least_squares():
    for seed in range(20):
        rng, B, _, _ = _problem(200 + seed, 16, 4)
        b = B.astype(np.float64) @ rng.uniform(0.5, 2.0, 4) + rng.normal(0, 0.01, 16)
        z = np.linalg.lstsq(B.astype(np.float64), b, rcond=None)[0]
        if (z > 0).all():
            x, _ = pm.fit_pack(B, b)
            assert np.allclose(x, z, rtol=1e-9, atol=1e-12)


def test_one_benchmark_twice():
    _, B, bt, be = _problem(7, 16, 12)
    x, res = pm.fit_pack(B, 2.0 * B[:, 5].astype(np.float64))
    assert np.allclose(x, 2.0 * np.eye(12)[5], atol=1e-9)
    t, e = pm.predict(np.round(x, 6), bt, be)
    assert np.array_equal(t, 2 * bt[5]) and np.array_equal(e, 2 * be[5])
