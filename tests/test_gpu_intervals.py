"""Time-interval policies (emo_eval_intervals) on the GPU through the C ABI, against the interval
oracle (needs an MI355X).  Times lie on the 2^-4 us grid, so start times are exact on both sides
and every interval lookup is taken on identical numbers; makespans are then bit-exact and
energies within 1e-5 relative."""
import numpy as np
import pytest

import oracle
import parity
import pins
from oracle import intervals
from paper_2607_12324_amd import synth

pytestmark = pytest.mark.gpu
REL = 1e-5


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


@pytest.fixture(scope="module")
def emo(torch):
    from paper_2607_12324_amd import emo as mod
    return mod


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def check(T, E, To, Eo, what):
    bad = np.isnan(To)
    assert np.array_equal(np.isnan(T), bad), what
    assert np.array_equal(T[~bad], To[~bad].astype(np.float32)), what
    err = np.abs(E[~bad] - Eo[~bad])
    assert (err <= REL * np.abs(Eo[~bad]) + 1e-30).all(), (what, float(err.max()))


def test_intervals_handworked(torch, emo):
    d = pins.load_golden("handworked_intervals.json")
    g = pins.graph_from_golden(pins.load_golden())
    gh = emo.EmoGraph(g, device=0)
    for case in d["cases"]:
        print(f"[case] intervals hand-worked {case['change_points']} {case['levels']}", flush=True)
        lv = dev(torch, np.asarray([case["levels"]], np.uint8))
        T, E, _, _ = gh.eval_intervals(lv, case["change_points"], d["idle_power"])
        assert gh.info()["last_kernels"] == 7     # the kernel specialised to the graph
        T, E = host(T), host(E)
        if case["makespan"] is None:
            assert np.isnan(T[0]) and np.isnan(E[0]), case
        else:
            assert T[0] == case["makespan"] and E[0] == case["energy"], (case, T, E)


def random_policy(rng, g, K, T_hi):
    pts = np.sort(rng.choice(np.arange(1, max(K + 1, int(T_hi * 16))), size=K - 1, replace=False)) / 16.0
    idle = np.round(rng.uniform(0, 1, g.num_levels) * 64) / 64
    return [float(x) for x in pts], [float(x) for x in idle]


@pytest.mark.parametrize("seed", range(4))
def test_intervals_match_oracle_on_random_dags(torch, emo, seed):
    rng = np.random.default_rng(1300 + seed)
    for i, K in enumerate((1, 3, 16, 17, 64, 256)):
        g = synth.random_dag(rng, int(rng.integers(2, 120)), float(rng.uniform(0.01, 0.08)), 0.7,
                             int(rng.integers(2, 17)), shuffle_packs=bool(i % 2))
        T0 = float(oracle.eval_batch(g, np.zeros((1, g.num_packs), np.uint8))[0][0])
        pts, idle = random_policy(rng, g, K, T0)
        B = int(rng.choice([1, 255, 257, 3001]))
        rows = rng.integers(0, g.num_levels, size=(B, K)).astype(np.uint8)
        if B > 10:
            rows[5, int(rng.integers(0, K))] = g.num_levels      # an invalid level: NaN
        print(f"[case] intervals seed={seed} V={g.num_nodes} P={g.num_packs} F={g.num_levels} K={K} B={B}",
              flush=True)
        To, Eo = intervals.eval_intervals(g, pts, rows, idle)
        gh = emo.EmoGraph(g, device=0)
        lv = dev(torch, rows)
        T, E, _, _ = gh.eval_intervals(lv, pts, idle)
        kind = gh.info()["last_kernels"]
        assert kind in (0, 7)
        check(host(T), host(E), To, Eo, f"seed={seed} K={K} kernels={kind}")
        # the interpreting kernel gives the same bits
        gi = emo.EmoGraph(g, device=0, kernel_mode=1)
        Ti, Ei, _, _ = gi.eval_intervals(lv, pts, idle)
        assert gi.info()["last_kernels"] == 0
        assert np.array_equal(host(T).view(np.uint32), host(Ti).view(np.uint32))
        assert np.array_equal(host(E).view(np.uint32), host(Ei).view(np.uint32))
        gi.close()
        finite = To[~np.isnan(To)]
        tgt = float(np.float32(np.quantile(finite, 0.4))) if finite.size else 1.0
        m = torch.empty(max(1, (B + 31) // 32), dtype=torch.int32, device="cuda")
        r = torch.empty(3, dtype=torch.int64, device="cuda")
        gh.eval_intervals(lv, pts, idle, latency_target=tgt, mask=m, result=r)
        parity.assert_selection(emo.parse_selection(r), emo.unpack_mask(m, B), To, Eo, tgt, True,
                                f"select seed={seed} K={K}")
        gh.close()


def test_intervals_one_interval_is_per_pack_evaluation(torch, emo):
    """One interval with idle power = static_power: the same results as emo_eval_policies with
    the row's level on every pack."""
    rng = np.random.default_rng(77)
    g = synth.config_graph(2)
    gh = emo.EmoGraph(g, device=0)
    rows1 = rng.integers(0, g.num_levels, size=(5000, 1)).astype(np.uint8)
    T, E, _, _ = gh.eval_intervals(dev(torch, rows1), [], [g.static_power] * g.num_levels)
    T2, E2 = gh.eval_policies(dev(torch, np.repeat(rows1, g.num_packs, axis=1)))
    assert np.array_equal(host(T), host(T2))
    assert np.allclose(host(E), host(E2), rtol=REL, atol=0)


def test_intervals_full_workload_sampled(torch, emo):
    """The 64-pack inference graph, 1M candidates, 16 intervals over [0, 1.05 T0): sampled rows
    against the oracle; the selection against what the returned makespans and energies imply."""
    g = synth.config_graph(2)
    B, K = 1 << 20, 16
    T0 = float(oracle.eval_batch(g, np.full((1, g.num_packs), g.num_levels - 1, np.uint8))[0][0])
    pts = [float(synth.quantize(T0 * 1.05 * (i + 1) / K)) for i in range(K - 1)]
    idle = [float(x) for x in synth.quantize(0.3 * np.ones(g.num_levels))]
    rows = synth.random_policies(11, K, g.num_levels, 0, B, "uniform")
    gh = emo.EmoGraph(g, device=0)
    lv = dev(torch, rows)
    tgt = float(np.float32(1.02 * T0))
    m = torch.empty((B + 31) // 32, dtype=torch.int32, device="cuda")
    r = torch.empty(3, dtype=torch.int64, device="cuda")
    print(f"[case] intervals full workload B={B} K={K}", flush=True)
    T, E, _, _ = gh.eval_intervals(lv, pts, idle, latency_target=tgt, mask=m, result=r)
    T, E = host(T), host(E)
    pick = synth.sample_rows(B, 64)
    To, Eo = intervals.eval_intervals(g, pts, rows[pick], idle)
    check(T[pick], E[pick], To, Eo, "sampled rows")
    sel = emo.parse_selection(r)
    feas = T <= np.float32(tgt)
    assert sel.num_feasible == int(feas.sum())
    assert np.array_equal(emo.unpack_mask(m, B), feas)
    if feas.any():
        best = np.flatnonzero(feas & (E == E[feas].min()))[0]
        assert sel.index == best and sel.energy == E[best] and sel.makespan == T[best]
        To1, Eo1 = intervals.eval_intervals(g, pts, rows[[best]], idle)
        check(T[[best]], E[[best]], To1, Eo1, "selected row")


def test_intervals_argument_errors(torch, emo):
    g = pins.graph_from_golden(pins.load_golden())
    gh = emo.EmoGraph(g, device=0)
    lv1 = dev(torch, np.zeros((4, 2), np.uint8))
    for pts, idle in (([12.0, 12.0], [0.1, 0.1]), ([0.0], [0.1, 0.1]), ([float("nan")], [0.1, 0.1]),
                      ([12.0], [0.1, -1.0]), ([12.0], [0.1, float("inf")])):
        lv = dev(torch, np.zeros((4, len(pts) + 1), np.uint8))
        with pytest.raises(emo.EmoError) as ei:
            gh.eval_intervals(lv, pts, idle)
        assert ei.value.status == 1, (pts, idle)
    with pytest.raises(emo.EmoError):
        gh.eval_intervals(dev(torch, np.zeros((4, 258), np.uint8)), list(np.arange(1.0, 258.0)), [0.1, 0.1])
    r = torch.empty(3, dtype=torch.int64, device="cuda")
    with pytest.raises(emo.EmoError):
        gh.eval_intervals(lv1, [12.0], [0.1, 0.1], latency_target=float("nan"), result=r)
    T, E, _, _ = gh.eval_intervals(lv1[:0], [12.0], [0.1, 0.1], result=r)
    assert emo.parse_selection(r).index == -1


@pytest.mark.parametrize("K", [1, 16, 17, 256])
def test_intervals_workload_kernels(torch, emo, K):
    """The 64-pack graph's specialised time-interval kernel (rows and the bucket table of the
    change points in LDS) on 200,003 candidates with K intervals evenly over [0, 1.05 T0): every
    row bit for bit against the interpreting kernel, sampled rows against the oracle, invalid
    levels and a ragged batch included."""
    g = synth.config_graph(2)
    B = 200_003
    T0 = float(oracle.eval_batch(g, np.full((1, g.num_packs), g.num_levels - 1, np.uint8))[0][0])
    pts = [float(synth.quantize(T0 * 1.05 * (i + 1) / K)) for i in range(K - 1)]
    idle = [float(x) for x in synth.quantize(0.3 * (0.5 + 0.5 * synth.level_ratios(g.num_levels)))]
    rows = synth.random_policies(12 + K, K, g.num_levels, 0, B, "uniform")
    rows[7, K // 2] = 200
    rows[B - 1, 0] = g.num_levels
    print(f"[case] interval kernels on the 64-pack graph K={K} B={B}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    lv = dev(torch, rows)
    tgt = float(np.float32(1.02 * T0))
    m = torch.empty((B + 31) // 32, dtype=torch.int32, device="cuda")
    r = torch.empty(3, dtype=torch.int64, device="cuda")
    T, E, _, _ = gh.eval_intervals(lv, pts, idle, latency_target=tgt, mask=m, result=r)
    assert gh.info()["last_kernels"] == 7
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    mi = torch.empty_like(m)
    ri = torch.empty_like(r)
    Ti, Ei, _, _ = gi.eval_intervals(lv, pts, idle, latency_target=tgt, mask=mi, result=ri)
    assert np.array_equal(host(T).view(np.uint32), host(Ti).view(np.uint32))
    assert np.array_equal(host(E).view(np.uint32), host(Ei).view(np.uint32))
    assert torch.equal(m, mi) and torch.equal(r, ri)
    assert np.isnan(host(T)[7]) and np.isnan(host(T)[B - 1])
    pick = np.concatenate([synth.sample_rows(B, 200), [7]])
    To, Eo = intervals.eval_intervals(g, pts, rows[pick], idle)
    check(host(T)[pick], host(E)[pick], To, Eo, f"K={K} sampled rows")
