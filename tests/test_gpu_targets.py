"""Several latency targets in one evaluation (emo_evaluate_targets) against one emo_evaluate call
per target, bit for bit, on every evaluating path, and each target's selection against the
oracle's Eq. 4 (needs an MI355X)."""
import dataclasses

import numpy as np
import pytest

import oracle
import parity
import pins
from paper_2607_12324_amd import synth

pytestmark = pytest.mark.gpu


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


def without_cuts(g):
    """A zero-duration source node into the last pack's node: no cut remains before that pack."""
    v = int(np.nonzero(g.node_pack == g.num_packs - 1)[0][0])
    V = g.num_nodes
    return dataclasses.replace(
        g, name=g.name + "-nocut", num_nodes=V + 1,
        edge_src=np.append(g.edge_src, np.int32(V)).astype(np.int32),
        edge_dst=np.append(g.edge_dst, np.int32(v)).astype(np.int32),
        node_pack=np.append(g.node_pack, np.int32(-1)).astype(np.int32),
        node_duration=np.append(g.node_duration, np.float32(0)).astype(np.float32),
        node_stream=None if g.node_stream is None else np.append(g.node_stream, np.int32(-1)).astype(np.int32))


def graph_of(case):
    if case in ("interpreted", "one-kernel"):
        return synth.config_graph(2)
    if case == "segmented":
        # more than 2048 steps: the forward pass is segmented too
        return without_cuts(synth.packed_graph(2416, 2400, 8, 16, sync_every=128, cross_p=0.05))
    if case == "cut":
        # the 4096-pack graph: too long for one kernel, synchronised every 256 packs
        return synth.config_graph(4)
    if case == "chain-lanes":
        # more than 16 chains: no windowed layout, one lane per chain
        return synth.stream_graph(9020, 9000, 20, 16)
    if case == "chain-windows":
        return synth.stream_graph(8224, 8208, 16, 16)
    raise KeyError(case)


# path kind (graph info last_kernels) of an evaluation without and with slack
KINDS = {"interpreted": (0, 0), "one-kernel": (1, 1), "segmented": (2, 2), "cut": (5, 5),
         "chain-lanes": (3, 3), "chain-windows": (4, None)}


def targets_for(T_or):
    """Eight targets: below every makespan (nothing feasible), quantiles, a repeated one, one
    exactly equal to a candidate's makespan, and +inf (every valid candidate feasible)."""
    ok = T_or[~np.isnan(T_or)]
    q = np.quantile(ok, [0.05, 0.3, 0.5, 0.8]).astype(np.float32)
    exact = np.float32(ok[len(ok) // 3])
    return [float(np.float32(ok.min()) * np.float32(0.5)), float(q[0]), float(q[1]), float(q[2]),
            float(q[2]), float(exact), float(q[3]), float("inf")]


@pytest.mark.parametrize("slack", [False, True], ids=["eval", "slack"])
@pytest.mark.parametrize("case", list(KINDS))
def test_targets_match_single_target_calls(torch, emo, case, slack):
    g = graph_of(case)
    mode = 1 if case == "interpreted" else 0
    gh = emo.EmoGraph(g, device=0, kernel_mode=mode)
    rng = np.random.default_rng(len(case) * 7 + slack)
    B = 2000 - 37                                     # a batch that ends inside a workgroup
    rows = pins.random_rows(rng, g, B)
    rows[11, g.num_packs // 2] = g.num_levels         # invalid levels: NaN, never feasible
    rows[1500, -1] = 255
    print(f"[case] targets {case} slack={slack}: V={g.num_nodes} P={g.num_packs} B={B}", flush=True)
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    tg = targets_for(T_or)
    n = len(tg)
    P = g.num_packs
    T = torch.empty(B, dtype=torch.float32, device="cuda")
    E = torch.empty_like(T)
    S = torch.empty((B, P), dtype=torch.float32, device="cuda") if slack else None
    W = (B + 31) // 32
    masks = [torch.full((W,), -1, dtype=torch.int32, device="cuda") for _ in range(n)]
    masks[3] = None                                   # a target with a result and no mask
    res = torch.full((n, 3), -7, dtype=torch.int64, device="cuda")
    gh.evaluate_targets(lv, tg, makespan=T, energy=E, slack=S, masks=masks, results=res)
    torch.cuda.synchronize()
    kind = KINDS[case][1 if slack else 0]
    got = gh.info()["last_kernels"]
    assert got == kind if kind is not None else got in (6, 8), (case, slack, got)
    parity.assert_eval(host(T), host(E), T_or, E_or, True, case)
    for k, t in enumerate(tg):
        T1 = torch.empty_like(T)
        E1 = torch.empty_like(T)
        S1 = torch.empty_like(S) if slack else None
        m1 = torch.full((W,), -1, dtype=torch.int32, device="cuda")
        r1 = torch.full((3,), -7, dtype=torch.int64, device="cuda")
        gh.evaluate(lv, makespan=T1, energy=E1, slack=S1, latency_target=t, mask=m1, result=r1)
        torch.cuda.synchronize()
        what = f"{case} target {k} ({t})"
        assert np.array_equal(host(T).view(np.uint32), host(T1).view(np.uint32)), what
        assert np.array_equal(host(E).view(np.uint32), host(E1).view(np.uint32)), what
        if slack:
            assert np.array_equal(host(S).view(np.uint32), host(S1).view(np.uint32)), what
        assert np.array_equal(host(res[k]), host(r1)), (what, host(res[k]), host(r1))
        if masks[k] is not None:
            assert np.array_equal(host(masks[k]), host(m1)), what
        parity.assert_selection(emo.parse_selection(res[k]), emo.unpack_mask(m1, B), T_or, E_or, t,
                                True, what)
    sel0 = emo.parse_selection(res[0])
    assert sel0.index == -1 and sel0.num_feasible == 0
    assert emo.parse_selection(res[7]).num_feasible == int((~np.isnan(T_or)).sum())


def test_targets_without_outputs_and_edge_cases(torch, emo):
    """Masks only (no results), one target, the most targets, an empty batch, and the argument
    errors: more than eight targets, a NaN target."""
    g = synth.config_graph(1)
    gh = emo.EmoGraph(g, device=0)
    rng = np.random.default_rng(5)
    B = 777
    rows = pins.random_rows(rng, g, B)
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    tg = targets_for(T_or)
    W = (B + 31) // 32
    masks = [torch.zeros(W, dtype=torch.int32, device="cuda") for _ in tg]
    gh.evaluate_targets(lv, tg, masks=masks)
    for k, t in enumerate(tg):
        _, feas, _ = oracle.select(T_or, E_or, t)
        assert np.array_equal(emo.unpack_mask(masks[k], B), feas), k
    r = torch.empty((1, 3), dtype=torch.int64, device="cuda")
    gh.evaluate_targets(lv, tg[2:3], results=r)
    parity.assert_selection(emo.parse_selection(r[0]), None, T_or, E_or, tg[2], True, "one target")
    # an empty batch: every result says no selection
    r8 = torch.full((8, 3), 5, dtype=torch.int64, device="cuda")
    gh.evaluate_targets(lv[:0], tg, results=r8)
    for k in range(8):
        s = emo.parse_selection(r8[k])
        assert s.index == -1 and s.num_feasible == 0
    with pytest.raises(emo.EmoError) as ei:
        gh.evaluate_targets(lv, tg + [1.0], results=torch.empty((9, 3), dtype=torch.int64, device="cuda"))
    assert ei.value.status == 1
    with pytest.raises(emo.EmoError) as ei:
        gh.evaluate_targets(lv, [1.0, float("nan")], results=torch.empty((2, 3), dtype=torch.int64, device="cuda"))
    assert ei.value.status == 1
