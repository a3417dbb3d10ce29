"""The library's pack model (emo_pack_model, host code) against the pack-model oracle on the
CPU (Sec. IV-E, Eq. 6-7): weights and tables on the seeded workload, rank-deficient suites (equal
residual and the optimality certificate), thread counts, edge cases and argument errors."""
import numpy as np
import pytest

from oracle import pack_model as pm
from paper_2607_12324_amd import synth


@pytest.fixture(scope="module")
def emo():
    from paper_2607_12324_amd import emo as mod
    return mod


def test_library_matches_oracle(emo):
    mi = synth.model_inputs(3, 2048, 16)
    W, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, mi.pack_metrics)
    Wo, To, Eo, _ = pm.pack_tables(mi.metric_matrix, mi.bench_time, mi.bench_energy,
                                   mi.pack_metrics)
    assert np.all(np.abs(W - Wo) <= 1e-6 * np.maximum(1.0, Wo.max(axis=1, keepdims=True)))
    assert np.all(np.abs(T - To) <= 1e-6 * To) and np.all(np.abs(E - Eo) <= 1e-6 * Eo)
    W1, T1, E1 = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy,
                                mi.pack_metrics, num_threads=1)
    assert np.array_equal(T1.view(np.uint32), T.view(np.uint32))
    assert np.array_equal(W1.view(np.uint32), W.view(np.uint32))


def test_library_rank_deficient(emo):
    """Fewer metrics than benchmarks: weights need not be unique, the residual is; the library's
    weights must reach the oracle's residual and satisfy the optimality certificate."""
    mi = synth.model_inputs(5, 128, 6, n=8, m=12)
    B = mi.metric_matrix.astype(np.float64)
    W, _, _ = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, mi.pack_metrics)
    for p, b in enumerate(mi.pack_metrics.astype(np.float64)):
        _, res = pm.fit_pack(B, b)
        x = W[p].astype(np.float64)
        assert (x >= 0).all()
        assert np.linalg.norm(B @ x - b) <= res + 1e-5 * np.linalg.norm(b)
        w = B.T @ (b - B @ x)
        assert (w <= 1e-4 * np.abs(B).sum() * np.abs(b).max()).all()


def test_library_edge_cases_and_errors(emo):
    mi = synth.model_inputs(2, 4, 1, m=1)
    W, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, mi.pack_metrics)
    Wo, To, Eo, _ = pm.pack_tables(mi.metric_matrix, mi.bench_time, mi.bench_energy,
                                   mi.pack_metrics)
    assert np.allclose(T, To, rtol=1e-6) and np.allclose(E, Eo, rtol=1e-6)
    W, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy,
                             np.zeros((0, mi.metric_matrix.shape[0]), np.float32))
    assert T.shape == (0, 1)
    W, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy,
                             np.zeros((2, mi.metric_matrix.shape[0]), np.float32))
    assert (W == 0).all() and (T == 0).all()
    bad = mi.pack_metrics.copy()
    bad[0, 0] = np.nan
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, bad)
    neg = mi.bench_time.copy()
    neg[0, 0] = -1
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.pack_model(mi.metric_matrix, neg, mi.bench_energy, mi.pack_metrics)
    big = synth.model_inputs(2, 2, 2, m=65)
    with pytest.raises(emo.EmoError, match="INVALID_ARGUMENT"):
        emo.pack_model(big.metric_matrix, big.bench_time, big.bench_energy, big.pack_metrics)


def test_library_step_to_boundary_regression(emo):
    """Packs of the 65,536-pack suite where a weight left at a rounding residue instead of zero
    after the step to the boundary once stopped the iteration at a non-optimal point."""
    mi = synth.model_inputs(5, 65536, 16)
    W, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, mi.pack_metrics)
    B = mi.metric_matrix.astype(np.float64)
    for p in (4868, 15139):
        b = mi.pack_metrics[p].astype(np.float64)
        x, res = pm.fit_pack(B, b)
        to, eo = pm.predict(x, mi.bench_time, mi.bench_energy)
        assert np.allclose(T[p], to, rtol=1e-6) and np.allclose(E[p], eo, rtol=1e-6)
        assert np.linalg.norm(B @ W[p].astype(np.float64) - b) <= res * (1 + 1e-6) + 1e-9
