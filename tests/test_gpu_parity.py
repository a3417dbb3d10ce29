"""HIP path against the oracle, through the C ABI (needs an MI355X)."""
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


MODES = {"auto": 0, "interpreted": 1}


def run_all(torch, emo, g, rows, targets, exact=True, per_node=True, what="", mode=0):
    """eval, slack (per pack and per node), fused select and select-from-results vs oracle."""
    print(f"[case] {what} mode={mode}: V={g.num_nodes} P={g.num_packs} F={g.num_levels} B={len(rows)}",
          flush=True)
    gh = emo.EmoGraph(g, device=0, kernel_mode=mode)
    lv = dev(torch, rows)
    B = len(rows)
    T, E = gh.eval_policies(lv)
    torch.cuda.synchronize()
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    parity.assert_eval(host(T), host(E), T_or, E_or, exact, what)
    # slack of every pack (+ makespan/energy from the same pass)
    T2 = torch.empty_like(T)
    E2 = torch.empty_like(E)
    S = gh.slack(lv, makespan=T2, energy=E2)
    parity.assert_eval(host(T2), host(E2), T_or, E_or, exact, what + " (slack pass)")
    pick = synth.sample_rows(B, 48) if B else np.zeros(0, np.int64)
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in pick]) if len(pick) else np.zeros((0, g.num_packs))
    parity.assert_slack(host(S)[pick], S_or, T_or[pick], exact, what + " pack slack")
    if per_node:
        SN = gh.slack(lv, per_node=True)
        SN_or = np.stack([oracle.slack(g, rows[c]).slack for c in pick]) if len(pick) else np.zeros((0, g.num_nodes))
        parity.assert_slack(host(SN)[pick], SN_or, T_or[pick], exact, what + " node slack")
    # the fused entry point: every output of the hot path from one launch
    for pn in ((False, True) if per_node else (False,)):
        cols = g.num_nodes if pn else g.num_packs
        T3 = torch.empty_like(T)
        E3 = torch.empty_like(E)
        S3 = torch.empty((B, cols), dtype=torch.float32, device="cuda")
        m3 = torch.empty(max(1, (B + 31) // 32), dtype=torch.int32, device="cuda")
        r3 = torch.empty(3, dtype=torch.int64, device="cuda")
        tgt = float(np.float32(targets[0]))
        gh.evaluate(lv, makespan=T3, energy=E3, slack=S3, per_node=pn, latency_target=tgt,
                    mask=m3, result=r3)
        parity.assert_eval(host(T3), host(E3), T_or, E_or, exact, what + f" evaluate pn={pn}")
        ref = S_or if not pn else np.stack([oracle.slack(g, rows[c]).slack for c in pick])
        parity.assert_slack(host(S3)[pick], ref, T_or[pick], exact, what + f" evaluate slack pn={pn}")
        parity.assert_selection(emo.parse_selection(r3), emo.unpack_mask(m3, B), T_or, E_or, tgt,
                                exact, what + f" evaluate select pn={pn}")
    for tgt in targets:
        tgt = float(np.float32(tgt))
        res, mask = gh.select_policy(lv, tgt)
        sel = emo.parse_selection(res)
        bits = emo.unpack_mask(mask, B)
        parity.assert_selection(sel, bits, T_or, E_or, tgt, exact, what + f" select@{tgt}")
        res2, mask2 = emo.select_from_results(T, E, tgt)
        sel2 = emo.parse_selection(res2)
        parity.assert_selection(sel2, emo.unpack_mask(mask2, B), T_or, E_or, tgt, exact,
                                what + f" select_from_results@{tgt}")
    gh.close()


def test_handworked_example(torch, emo):
    d = pins.load_golden()
    g = pins.graph_from_golden(d)
    rows = synth.exhaustive_policies(g.num_packs, g.num_levels, 0, 8)
    gh = emo.EmoGraph(g, device=0)
    T, E = gh.eval_policies(dev(torch, rows))
    assert host(T).tolist() == d["makespan"]
    assert np.allclose(host(E), d["energy"], rtol=1e-6, atol=0)
    SN = host(gh.slack(dev(torch, rows), per_node=True))
    for c, expect in d["node_slack"].items():
        assert SN[int(c)].tolist() == expect
    for s in d["selection"]:
        res, mask = gh.select_policy(dev(torch, rows), s["target"])
        sel = emo.parse_selection(res)
        assert sel.index == s["index"] and sel.num_feasible == s["num_feasible"], (s, sel)
    for mode in MODES.values():
        run_all(torch, emo, g, rows, [16.8, 18.0, 20.0, 22.0, 15.9], what="handworked", mode=mode)


@pytest.mark.parametrize("seed", range(8))
def test_random_dags_on_grid(torch, emo, seed):
    rng = np.random.default_rng(1000 + seed)
    for i in range(4):
        V = int(rng.integers(1, 300))
        F = int(rng.integers(1, 20))
        g = synth.random_dag(rng, V, float(rng.uniform(1.0, 6.0)) / max(V, 1),
                             float(rng.uniform(0.2, 1.0)), F, shuffle_packs=bool(i % 2))
        B = int(rng.integers(1, 1500))
        rows = pins.random_rows(rng, g, B)
        T_or, _ = oracle.eval_batch(g, rows)
        targets = [float(np.quantile(T_or, q)) for q in (0.0, 0.3, 0.9)] + [float(T_or.min()) - 1.0]
        for mode in MODES.values():
            run_all(torch, emo, g, rows, targets, exact=True, what=f"random seed={seed} i={i}", mode=mode)


@pytest.mark.parametrize("seed", range(3))
def test_random_dags_off_grid(torch, emo, seed):
    rng = np.random.default_rng(2000 + seed)
    for i in range(3):
        V = int(rng.integers(2, 200))
        F = int(rng.integers(2, 9))
        g = synth.random_dag(rng, V, 3.0 / V, 0.6, F, on_grid=False)
        B = int(rng.integers(100, 3000))
        rows = pins.random_rows(rng, g, B)
        T_or, _ = oracle.eval_batch(g, rows)
        for mode in MODES.values():
            run_all(torch, emo, g, rows, [float(np.quantile(T_or, 0.5))], exact=False,
                    what=f"offgrid seed={seed} i={i}", mode=mode)


@pytest.mark.parametrize("F,P", [(16, 700), (200, 64), (5, 1800), (256, 40)])
def test_interpreter_table_windows(torch, emo, F, P):
    """Tables too large for LDS with packs in increasing topological order: the interpreting
    kernels stage windows of table rows (and stream the rest when windows cannot apply)."""
    rng = np.random.default_rng(F * 1000 + P)
    V = int(P * 1.5)
    g = synth.random_dag(rng, V, 2.5 / V, P / V, F, shuffle_ids=False, shuffle_packs=False)
    assert g.num_packs * F * 8 > 60 * 1024 or F == 256
    rows = pins.random_rows(rng, g, 700)
    gh = emo.EmoGraph(g, device=0, kernel_mode=1)
    assert gh.info()["pack_order_monotone"] == 1
    T_or, _ = oracle.eval_batch(g, rows)
    run_all(torch, emo, g, rows, [float(np.median(T_or))], what=f"windows F={F} P={P}", mode=1)


def without_cuts(g):
    """The same graph without cut nodes (a zero-duration source into the last pack's node), so
    that the cut-segment kernels do not apply."""
    return synth.without_cuts(g)


def with_host_source(g, dur=7.5):
    """The same graph plus a fixed-duration node before every source (a candidate-independent
    start-time floor for the first packs)."""
    V = g.num_nodes
    srcs = np.setdiff1d(np.arange(V), g.edge_dst).astype(np.int32)
    return dataclasses.replace(
        g, name=g.name + "-host", num_nodes=V + 1,
        edge_src=np.concatenate([g.edge_src, np.full(len(srcs), V, np.int32)]),
        edge_dst=np.concatenate([g.edge_dst, srcs]),
        node_pack=np.append(g.node_pack, np.int32(-1)).astype(np.int32),
        node_duration=np.append(g.node_duration, np.float32(dur)).astype(np.float32),
        node_stream=None if g.node_stream is None else np.append(g.node_stream, np.int32(-1)).astype(np.int32))


SEGMENTED_CASES = {
    # name: (packs, streams, levels, shuffled pack ids)
    "staged-F16": (1024, 8, 16, False),      # slack written through LDS, table windows in LDS
    "ragged-F16": (1000, 6, 16, False),      # pack count not a multiple of 16: direct stores
    "shuffled-F8": (700, 4, 8, True),        # packs out of order: byte loads, direct stores
    "monotone-F5": (896, 8, 5, False),       # level count not a power of two
    "wide-F16": (2400, 8, 16, False),        # past one kernel's limit even without slack
}


@pytest.mark.parametrize("case", list(SEGMENTED_CASES))
def test_segmented_kernels(torch, emo, case):
    """Graphs too large to keep every finish time in registers (slack) and, without slack, too
    large for one kernel or for its table in LDS (the wide case): the chained segment kernels, with finish times recomputed per
    sub-segment in the backward kernels, against the oracle on every row, including rows with an
    invalid level byte and a batch that ends inside a workgroup."""
    P, S_, F, shuffled = SEGMENTED_CASES[case]
    g = without_cuts(synth.packed_graph(P + F, P, S_, F, sync_every=128, cross_p=0.05,
                                        shuffle_pack_ids=shuffled))
    rng = np.random.default_rng(P * F)
    rows = pins.random_rows(rng, g, 1000 - 23)
    rows[7, g.num_packs // 2] = F              # invalid levels: NaN results, never feasible
    rows[300, -1] = 255
    print(f"[case] segmented {case}: V={g.num_nodes} P={g.num_packs} B={len(rows)}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    assert gh.info()["cut_segments"] == 0
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    T, E = gh.eval_policies(lv)
    S = gh.slack(lv)
    torch.cuda.synchronize()
    info = gh.info()
    assert info["specialized"] & 8 and info["last_kernels"] == 2, info   # segmented kernels ran
    ok = ~np.isnan(T_or)
    assert np.isnan(host(T)[7]) and np.isnan(host(T)[300]) and not ok[7] and not ok[300]
    parity.assert_eval(host(T), host(E), T_or, E_or, True, case)
    Sh = host(S)
    assert np.all(np.isnan(Sh[~ok]))
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in np.nonzero(ok)[0]])
    parity.assert_slack(Sh[ok], S_or, T_or[ok], True, case + " pack slack")
    # the same through the fused entry point, and the interpreted kernels bit for bit
    tgt = float(np.float32(np.median(T_or[ok])))
    run_all(torch, emo, g, rows, [tgt], per_node=False, what="segmented " + case)
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    Ti, Ei = gi.eval_policies(lv)
    Si = gi.slack(lv)
    for a, b in ((T, Ti), (E, Ei), (S, Si)):
        assert np.array_equal(host(a).view(np.uint32), host(b).view(np.uint32)), case


@pytest.mark.parametrize("B", [3 * 256 + 64, 3 * 256 + 1, 5 * 256 + 192])
def test_segmented_kernels_ragged_last_workgroup(torch, emo, B):
    """Batches that end one wave (or one lane) into a 256-thread workgroup of the segmented
    forward kernels: the workgroup's remaining waves hold only lanes past the batch, which
    repeat candidate B - 1.  Its running makespan and energy, read back and added to by the next
    kernel, must be stored once; every row, B - 1 included, against the oracle."""
    g = without_cuts(synth.packed_graph(2400 + 16, 2400, 8, 16, sync_every=128, cross_p=0.05))
    rng = np.random.default_rng(B)
    rows = pins.random_rows(rng, g, B)
    print(f"[case] segmented ragged B={B}: V={g.num_nodes} P={g.num_packs}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    for rep in range(3):
        T, E = gh.eval_policies(lv)
        torch.cuda.synchronize()
        assert gh.info()["last_kernels"] == 2, gh.info()
        parity.assert_eval(host(T), host(E), T_or, E_or, True, f"segmented ragged B={B} rep={rep}")
    tgt = float(np.float32(np.median(T_or)))
    res, mask = gh.select_policy(lv, tgt)
    parity.assert_selection(emo.parse_selection(res), emo.unpack_mask(mask, B), T_or, E_or, tgt,
                            True, f"segmented ragged B={B} select")


CUT_CASES = {
    # name: (packs, streams, levels, packs between synchronisations, segments)
    "sync-256-F16": (1024, 8, 16, 256, 4),   # 256-pack segments, as in the 4096-pack workload
    "sync-128-F8": (2048, 4, 8, 128, 8),     # pieces of 128 packs, two per segment
    "open-end-F16": (1056, 8, 16, 256, 5),   # 32 packs after the last synchronisation
    "sync-96-F5": (960, 6, 5, 96, 5),        # level count not a power of two; 192-pack segments
    "sync-128-F32": (1024, 4, 32, 128, 8),   # 32 levels: 128 packs fill the table window
    "host-source": (1024, 8, 16, 256, 4),    # a fixed node before every source
}


@pytest.mark.parametrize("case", list(CUT_CASES))
def test_cut_segment_kernels(torch, emo, case):
    """Graphs with all-stream synchronisations: the segments between them evaluated on their own
    (finish times from the segment's start, exact on the time grid), against the oracle on every
    row, with rows holding invalid level bytes (two in one wave: the last kernel rewrites their
    slack rows with NaN), a batch that ends inside a workgroup, and the interpreted kernels bit
    for bit."""
    P, S_, F, se, m = CUT_CASES[case]
    g = synth.packed_graph(P + F + se, P, S_, F, sync_every=se, cross_p=0.05)
    if case == "host-source":
        g = with_host_source(g)
    rng = np.random.default_rng(P + se)
    rows = pins.random_rows(rng, g, 1000 - 23)
    rows[7, P // 2] = F
    rows[300, -1] = 255
    rows[301, 0] = F
    print(f"[case] cut segments {case}: V={g.num_nodes} P={P} B={len(rows)}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    assert gh.info()["cut_segments"] == m
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    T, E = gh.eval_policies(lv)
    torch.cuda.synchronize()
    # without slack: one kernel while its (time, energy) table (plus 256 pad entries when F is not
    # a power of two) fits its 64 KB of LDS, else the cut kernels
    tb = (P * F + (0 if F & (F - 1) == 0 else 256)) * 8
    assert gh.info()["last_kernels"] == (1 if tb <= 65536 else 5), (tb, gh.info())
    S = gh.slack(lv)
    torch.cuda.synchronize()
    info = gh.info()
    assert info["specialized"] & 16 and info["last_kernels"] == 5, info
    ok = ~np.isnan(T_or)
    assert not ok[[7, 300, 301]].any()
    parity.assert_eval(host(T), host(E), T_or, E_or, True, case)
    Sh = host(S)
    assert np.all(np.isnan(Sh[~ok]))
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in np.nonzero(ok)[0]])
    parity.assert_slack(Sh[ok], S_or, T_or[ok], True, case + " pack slack")
    tgt = float(np.float32(np.median(T_or[ok])))
    run_all(torch, emo, g, rows, [tgt], per_node=False, what="cut " + case)
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    Ti, Ei = gi.eval_policies(lv)
    Si = gi.slack(lv)
    for a, b in ((T, Ti), (E, Ei), (S, Si)):
        assert np.array_equal(host(a).view(np.uint32), host(b).view(np.uint32)), case


@pytest.mark.parametrize("case", ["sync-256-F16", "sync-96-F5", "host-source"])
def test_cut_segments_off_grid(torch, emo, case):
    """Times off the exact-sum grid (every table time scaled by 1.1): the cut-segment kernels still
    apply, timing each segment from its start, so they round differently from the program
    order.  Makespan, energy and every slack element against the oracle within 1e-5 of the
    makespan, every mask bit whose candidate's makespan is not within that bound of the target,
    the selection, and the interpreted kernels to the same bound."""
    P, S_, F, se, m = CUT_CASES[case]
    g = synth.packed_graph(P + F + se, P, S_, F, sync_every=se, cross_p=0.05)
    if case == "host-source":
        g = with_host_source(g)
    g = synth.scaled_times(g, 1.1)
    rng = np.random.default_rng(P + se + 1)
    rows = pins.random_rows(rng, g, 1000 - 23)
    rows[7, P // 2] = F
    rows[300, -1] = 255
    print(f"[case] cut segments off the grid {case}: V={g.num_nodes} P={P} B={len(rows)}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    info = gh.info()
    assert info["cut_segments"] == m and info["exact_time_sums"] == 0, info
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    ok = ~np.isnan(T_or)
    tgt = float(np.float32(np.median(T_or[ok])))
    B = len(rows)
    T = torch.empty(B, dtype=torch.float32, device="cuda")
    E = torch.empty_like(T)
    S = torch.empty((B, P), dtype=torch.float32, device="cuda")
    mk = torch.empty((B + 31) // 32, dtype=torch.int32, device="cuda")
    r = torch.empty(3, dtype=torch.int64, device="cuda")
    gh.evaluate(lv, makespan=T, energy=E, slack=S, latency_target=tgt, mask=mk, result=r)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == 5
    parity.assert_eval(host(T), host(E), T_or, E_or, False, case)
    Sh = host(S)
    assert np.all(np.isnan(Sh[~ok]))
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in np.nonzero(ok)[0]])
    parity.assert_slack(Sh[ok], S_or, T_or[ok], False, case + " pack slack")
    bits = emo.unpack_mask(mk, B)
    _, feas_or, _ = oracle.select(T_or, E_or, tgt)
    clear = ~ok | (np.abs(T_or - tgt) > parity.REL * np.abs(T_or))
    assert np.array_equal(bits[clear], feas_or[clear]), case + " mask"
    parity.assert_selection(emo.parse_selection(r), bits, T_or, E_or, tgt, False, case + " select")
    run_all(torch, emo, g, rows, [tgt], exact=False, per_node=False, what="cut off the grid " + case)
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    Ti, Ei = gi.eval_policies(lv)
    Si = gi.slack(lv)
    torch.cuda.synchronize()
    parity.assert_eval(host(T), host(E), host(Ti).astype(np.float64), host(Ei).astype(np.float64), False,
                       case + " vs interpreted")
    parity.assert_slack(Sh[ok], host(Si)[ok], T_or[ok], False, case + " slack vs interpreted")


def test_cut_segments_small_batches(torch, emo):
    """Cut-segment kernels with batches smaller than a workgroup and one past it (lanes past the
    batch repeat the last row and store nothing), repeated calls bit for bit."""
    g = synth.packed_graph(5, 1024, 8, 16, sync_every=256, cross_p=0.05)
    rng = np.random.default_rng(5)
    gh = emo.EmoGraph(g, device=0)
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    for B in (1, 3, 512, 513):
        rows = pins.random_rows(rng, g, B)
        print(f"[case] cut segments B={B}", flush=True)
        lv = dev(torch, rows)
        T, E = gh.eval_policies(lv)
        S = gh.slack(lv)
        torch.cuda.synchronize()
        assert gh.info()["last_kernels"] == 5
        T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
        parity.assert_eval(host(T), host(E), T_or, E_or, True, f"cut B={B}")
        S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in range(B)])
        parity.assert_slack(host(S), S_or, T_or, True, f"cut B={B} pack slack")
        T2, E2 = gh.eval_policies(lv)
        S2 = gh.slack(lv)
        Ti, Ei = gi.eval_policies(lv)
        Si = gi.slack(lv)
        for a, b in ((T, T2), (E, E2), (S, S2), (T, Ti), (E, Ei), (S, Si)):
            assert np.array_equal(host(a).view(np.uint32), host(b).view(np.uint32)), B


@pytest.mark.parametrize("seed", range(3))
def test_cut_segments_on_block_graphs(torch, emo, seed):
    """Random block graphs: synchronisations (some bypassed by a fixed node), packs that are cuts
    themselves, 16, 32 or 64 levels (segments of at most 256, 128 or 64 packs).  Slack runs on the
    cut-segment kernels wherever the graph has cut segments; every call matches the oracle and
    the interpreted kernels bit for bit."""
    grng = np.random.default_rng(950 + seed)
    rrng = np.random.default_rng(960 + seed)
    ran = 0
    for i in range(4):
        F = int(grng.choice([16, 32, 64]))
        g = synth.block_graph(grng, int(grng.integers(6, 20)), float(grng.uniform(0.0, 0.4)), F)
        rows = pins.random_rows(rrng, g, 300)
        gh = emo.EmoGraph(g, device=0)
        m = gh.info()["cut_segments"]
        print(f"[case] block graph seed={seed} #{i}: P={g.num_packs} F={F} segments={m}", flush=True)
        lv = dev(torch, rows)
        T, E = gh.eval_policies(lv)
        S = gh.slack(lv)
        torch.cuda.synchronize()
        if m:
            assert gh.info()["last_kernels"] == 5
            ran += 1
        T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
        parity.assert_eval(host(T), host(E), T_or, E_or, True, f"block graph {seed}/{i}")
        S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in range(len(rows))])
        parity.assert_slack(host(S), S_or, T_or, True, f"block graph {seed}/{i} pack slack")
        gi = emo.EmoGraph(g, device=0, kernel_mode=1)
        Ti, Ei = gi.eval_policies(lv)
        Si = gi.slack(lv)
        for a, b in ((T, Ti), (E, Ei), (S, Si)):
            assert np.array_equal(host(a).view(np.uint32), host(b).view(np.uint32)), (seed, i)
    assert ran >= 3


def test_cut_segments_unaligned_buffers(torch, emo):
    """A graph with cut segments and level rows or a slack buffer that are not 16-byte aligned:
    the call takes other kernels (the cut-segment kernels load levels and store slack in 16-byte
    pieces) and the results stay those of the oracle and of the aligned call, bit for bit."""
    g = synth.packed_graph(6, 1024, 8, 16, sync_every=256, cross_p=0.05)
    rng = np.random.default_rng(6)
    rows = pins.random_rows(rng, g, 700)
    print("[case] cut segments, unaligned buffers", flush=True)
    gh = emo.EmoGraph(g, device=0)
    lv = dev(torch, rows)
    T, E = gh.eval_policies(lv)
    S = gh.slack(lv)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == 5
    lm = misaligned(torch, rows)
    Tm, Em = gh.eval_policies(lm)
    Sm = gh.slack(lm)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] != 5
    sbuf = torch.empty(rows.shape[0] * g.num_packs + 4, dtype=torch.float32, device="cuda")
    Su = sbuf[1:1 + rows.shape[0] * g.num_packs].view(rows.shape[0], g.num_packs)
    gh.slack(lv, out=Su)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] != 5
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    parity.assert_eval(host(T), host(E), T_or, E_or, True, "cut aligned")
    for a, b in ((T, Tm), (E, Em), (S, Sm), (S, Su)):
        assert np.array_equal(host(a).view(np.uint32), host(b).view(np.uint32))


CHAIN_CASES = {"1-stream": (10000, 1, 16), "5-streams": (9000, 5, 16), "33-streams": (8500, 33, 8),
               "64-streams": (8300, 64, 5),
               # a block's table rows exceed the LDS stage: every lane reads the table itself
               "64-streams-F16": (8300, 64, 16),
               # pack count not a multiple of 4: the lane-per-chain kernel (unaligned buffers) stores
               # slack directly in pack order
               "odd-packs": (8301, 7, 8),
               # windowed kernel: 16 chains (one workgroup of 64 candidates), 3 chains (5 groups
               # of 64 candidates), 9 chains with 32 levels (narrower windows); more than 8192
               # steps, so that the segmented kernels do not apply
               "16-streams": (8208, 16, 16), "3-streams-F8": (8224, 3, 8), "9-streams-F32": (8208, 9, 32)}
# packs per window of the windowed kernel (0: lane-per-chain kernels only)
# (9000 and 8301 packs: rows that are not 16-byte aligned, copied from the dwords around each
# piece, with windows narrow enough for one piece per thread; 8301: slack rows stored a float at
# a time)
CHAIN_WINDOW = {"1-stream": 16, "5-streams": 64, "odd-packs": 64, "16-streams": 256, "3-streams-F8": 64,
                "9-streams-F32": 64}


def off_grid(g):
    """The same graph plus one isolated node of 2^-30 us.  The common power of two of all times
    drops to 2^-30, so the loader can no longer show that every time sum is exact
    (exact_time_sums 0); every value the chains compute is still on the 2^-4 us grid, so results
    stay exact and the kernels must still match the oracle bit for bit."""
    V = g.num_nodes
    return dataclasses.replace(
        g, name=g.name + "-offgrid", num_nodes=V + 1,
        node_pack=np.append(g.node_pack, np.int32(-1)).astype(np.int32),
        node_duration=np.append(g.node_duration, np.float32(2.0 ** -30)).astype(np.float32),
        node_stream=None if g.node_stream is None else np.append(g.node_stream, np.int32(-1)).astype(np.int32))


def check_windowed_off_grid(torch, emo, g, rows, win, what):
    """The windowed kernels on the off-grid copy of `g` (the chain scan for slack, whose time
    sums the loader cannot show exact): makespan, energy and slack against the oracle, makespan
    and slack bit for bit against the interpreter."""
    g2 = off_grid(g)
    gh = emo.EmoGraph(g2, device=0)
    info = gh.info()
    assert info["exact_time_sums"] == 0 and info["chain_window"] == win and info["chain_scan_window"] == win
    lv = dev(torch, rows)
    T, E = gh.eval_policies(lv)
    assert gh.info()["last_kernels"] == 4, gh.info()
    S = gh.slack(lv)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == (8 if info["chain_scan_full"] else 6), gh.info()
    T_or, E_or = oracle.eval_batch(g2, rows, nthreads=8)
    parity.assert_eval(host(T), host(E), T_or, E_or, True, what + " off grid")
    ok = ~np.isnan(T_or)
    _, _, S_or = oracle.slack_batch(g2, rows[ok], nthreads=8)
    parity.assert_slack(host(S)[ok], S_or, T_or[ok], True, what + " off grid slack")
    gi = emo.EmoGraph(g2, device=0, kernel_mode=1)
    Ti, _ = gi.eval_policies(lv)
    Si = gi.slack(lv)
    assert np.array_equal(host(T).view(np.uint32), host(Ti).view(np.uint32)), what
    assert np.array_equal(host(S).view(np.uint32), host(Si).view(np.uint32)), what


def misaligned(torch, rows):
    """The rows in device memory at an address that is not 16-byte aligned."""
    buf = torch.empty(rows.size + 16, dtype=torch.uint8, device="cuda")
    v = buf[1:1 + rows.size].view(rows.shape)
    v.copy_(torch.from_numpy(np.ascontiguousarray(rows)).to("cuda"))
    return v


@pytest.mark.parametrize("case", list(CHAIN_CASES))
def test_chain_lanes(torch, emo, case):
    """Graphs whose candidate-dependent kernels form disjoint stream chains, too long for the
    specialised kernels: one lane per chain and candidate, against the oracle on every row and
    against the interpreting kernels (makespan and slack bit for bit), with invalid levels and a
    batch that ends inside a workgroup."""
    P, S_, F = CHAIN_CASES[case]
    g = synth.stream_graph(P + S_, P, S_, F)
    rng = np.random.default_rng(P + S_ + F)
    rows = pins.random_rows(rng, g, 777)
    rows[5, g.num_packs // 3] = F
    rows[600, 0] = 255
    rows[7, g.num_packs - 1] = 128
    print(f"[case] chain lanes {case}: V={g.num_nodes} P={g.num_packs} B={len(rows)}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    lanes = 1
    while lanes < S_:
        lanes *= 2
    win = CHAIN_WINDOW.get(case, 0)
    assert gh.info()["chain_lanes"] == lanes
    assert gh.info()["chain_window"] == win
    # on the time grid the two-pass scan kernel takes the windowed layout's place
    assert gh.info()["chain_scan_window"] == win
    # without slack the windowed kernel; with it the two-pass scan (per-thread copy plans when
    # every window is full and there are enough chains)
    kind = 4 if win else 3
    skind = (8 if gh.info()["chain_scan_full"] else 6) if win else 3
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    T, E = gh.eval_policies(lv)
    assert gh.info()["last_kernels"] == kind
    S = gh.slack(lv)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == skind
    ok = ~np.isnan(T_or)
    assert not ok[5] and not ok[600] and not ok[7]
    parity.assert_eval(host(T), host(E), T_or, E_or, True, case)
    Sh = host(S)
    assert np.all(np.isnan(Sh[~ok]))
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in np.nonzero(ok)[0]])
    parity.assert_slack(Sh[ok], S_or, T_or[ok], True, case + " pack slack")
    tgt = float(np.float32(np.median(T_or[ok])))
    run_all(torch, emo, g, rows, [tgt], per_node=False, what="chain lanes " + case)
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    Ti, _ = gi.eval_policies(lv)
    Si = gi.slack(lv)
    assert np.array_equal(host(T).view(np.uint32), host(Ti).view(np.uint32)), case
    assert np.array_equal(Sh.view(np.uint32), host(Si).view(np.uint32)), case
    if win:
        # the same candidates through the lane-per-chain kernel (unaligned levels): makespans
        # and slack bit for bit, energies (summed in another order) to the bound
        lm = misaligned(torch, rows)
        Tm, Em = gh.eval_policies(lm)
        Sm = gh.slack(lm)
        torch.cuda.synchronize()
        assert gh.info()["last_kernels"] == 3
        assert np.array_equal(host(T).view(np.uint32), host(Tm).view(np.uint32)), case
        assert np.array_equal(Sh.view(np.uint32), host(Sm).view(np.uint32)), case
        parity.assert_eval(host(Tm), host(Em), T_or, E_or, True, case + " lane-per-chain")
        check_windowed_off_grid(torch, emo, g, rows, win, "chain lanes " + case)


def test_one_kernel_ragged_batches(torch, emo):
    """512-pack graph in one kernel: batches that leave the last workgroup partly or wholly past
    the batch, with an invalid level among the rows, against the oracle, and the selection."""
    g = synth.config_graph(3)
    gh = emo.EmoGraph(g, device=0)
    for B in (1, 65, 777, 1025, 3000):
        rows = synth.config_policies(3, g, 5000 + B, B)
        if B > 2:
            rows[B // 2, 7] = 200   # an invalid level
        print(f"[case] one kernel B={B}", flush=True)
        T, E = gh.eval_policies(dev(torch, rows))
        torch.cuda.synchronize()
        assert gh.info()["last_kernels"] == 1
        T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
        assert np.isnan(host(T)[B // 2]) == (B > 2)
        parity.assert_eval(host(T), host(E), T_or, E_or, True, f"one kernel B={B}")
        tgt = float(np.float32(1.05 * float(np.nanmin(T_or))))
        run_all(torch, emo, g, rows, [tgt], per_node=False, what=f"one kernel B={B}")


@pytest.mark.parametrize("grid", ["on", "off", "unaligned"])
def test_chain_windows_small_batches(torch, emo, grid):
    """Two-pass scan kernel (slack) and windowed kernel (eval), on the time grid, on a graph
    whose sums the loader cannot show exact, and with 8211 packs (rows that are not 4-byte
    aligned: a batch of one row reads its last piece's dwords up to the batch's end only), with
    batches smaller than a workgroup's 64 candidates and one past it (lanes past the batch
    repeat the last row and store nothing), repeated calls bit for bit."""
    g = synth.stream_graph(77, 8211 if grid == "unaligned" else 8208, 16, 16)
    if grid == "off":
        g = off_grid(g)
    rng = np.random.default_rng(77)
    gh = emo.EmoGraph(g, device=0)
    assert gh.info()["chain_window"] == 256
    assert gh.info()["chain_scan_window"] == 256
    assert gh.info()["exact_time_sums"] == (0 if grid == "off" else 1)
    assert gh.info()["chain_scan_full"] == 0     # 8208 and 8211 packs: the last window is partial
    for B in (1, 3, 64, 65):
        rows = pins.random_rows(rng, g, B)
        print(f"[case] windowed chains grid={grid} B={B}", flush=True)
        lv = dev(torch, rows)
        T, E = gh.eval_policies(lv)
        S = gh.slack(lv)
        torch.cuda.synchronize()
        assert gh.info()["last_kernels"] == 6     # (the slack call)
        T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
        parity.assert_eval(host(T), host(E), T_or, E_or, True, f"windowed B={B}")
        S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in range(B)])
        parity.assert_slack(host(S), S_or, T_or, True, f"windowed B={B} pack slack")
        T2, E2 = gh.eval_policies(lv)
        S2 = gh.slack(lv)
        assert np.array_equal(host(T).view(np.uint32), host(T2).view(np.uint32))
        assert np.array_equal(host(E).view(np.uint32), host(E2).view(np.uint32))
        assert np.array_equal(host(S).view(np.uint32), host(S2).view(np.uint32))


@pytest.mark.parametrize("case", ["8208", "8448", "fixed"])
def test_chain_scan_off_grid(torch, emo, case):
    """Chain graphs with every table time scaled by 1.1 (off any common power-of-two grid): the
    two-pass scan takes slack from prefix sums along each chain, so it rounds differently from
    the backward recurrence.  Makespan, energy and every slack element against the oracle within
    1e-5 of the makespan, and against the interpreter to the same bound (makespans bit for bit:
    the forward walk is the recurrence's).  8208 packs on 16 streams run the general scan
    kernel, 8448 the one with per-thread copy plans (both more than 8192 steps, past the
    segmented kernels); "fixed" is 16 chains of packs and fixed-duration nodes (the copy-plan
    kernel with fixed durations)."""
    rng = np.random.default_rng(len(case) + 78)
    if case == "fixed":
        g = fixed_chains_graph(rng, [768] * 16)
    else:
        g = synth.stream_graph(78, int(case), 16, 16)
    g = synth.scaled_times(g, 1.1)
    P = g.num_packs
    rows = pins.random_rows(rng, g, 300)
    rows[9, P // 2] = g.num_levels
    print(f"[case] chain scan off the grid {case}: V={g.num_nodes} P={P}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    info = gh.info()
    full = P % 256 == 0
    assert info["exact_time_sums"] == 0 and info["chain_scan_window"] == 256
    assert info["chain_scan_full"] == (1 if full else 0)
    lv = dev(torch, rows)
    T = torch.empty(len(rows), dtype=torch.float32, device="cuda")
    E = torch.empty_like(T)
    S = gh.slack(lv, makespan=T, energy=E)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == (8 if full else 6), gh.info()
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    ok = ~np.isnan(T_or)
    assert not ok[9]
    parity.assert_eval(host(T), host(E), T_or, E_or, False, f"scan off grid {case}")
    Sh = host(S)
    assert np.all(np.isnan(Sh[~ok]))
    _, _, S_or = oracle.slack_batch(g, rows[ok], nthreads=8)
    parity.assert_slack(Sh[ok], S_or, T_or[ok], False, f"scan off grid {case} slack")
    gi = emo.EmoGraph(g, device=0, kernel_mode=1)
    Ti, _ = gi.eval_policies(lv)
    Si = gi.slack(lv)
    assert np.array_equal(host(T).view(np.uint32), host(Ti).view(np.uint32))
    parity.assert_slack(Sh[ok], host(Si)[ok], T_or[ok], False, f"scan off grid {case} vs interpreted")


# stream-chain graphs short enough for the segmented kernels: (packs, streams, levels) and the
# kernels their slack call takes (2 segmented, 6 chain scan, 8 chain scan with copy plans)
SCAN_FIRST_CASES = {"512": (512, 16, 16, 2), "768": (768, 16, 16, 8), "2000-5s": (2000, 5, 16, 6),
                    "4100-unaligned": (4100, 16, 16, 6), "3000-7s-F8": (3000, 7, 8, 6)}


@pytest.mark.parametrize("case", list(SCAN_FIRST_CASES))
def test_chain_scan_before_segmented(torch, emo, case):
    """Slack on disjoint stream chains of 768 to 8192 steps takes the windowed chain scan rather
    than the segmented kernels (512 steps still the segmented ones); calls without slack keep the
    one-kernel (table in LDS) or segmented kernels, and a slack buffer that is not 16-byte
    aligned leaves the scan.  Every row against the oracle; makespan and slack bit for bit
    between the kernel kinds (the graphs are on the exact-sum grid)."""
    P, S_, F, skind = SCAN_FIRST_CASES[case]
    g = synth.stream_graph(P + S_, P, S_, F)
    rng = np.random.default_rng(P + 31 * S_)
    rows = pins.random_rows(rng, g, 300)
    rows[11, P // 2] = F
    print(f"[case] chain scan before segmented {case}: V={g.num_nodes} P={P}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    assert gh.info()["exact_time_sums"] == 1 and gh.info()["chain_scan_window"] > 0
    lv = dev(torch, rows)
    T = torch.empty(len(rows), dtype=torch.float32, device="cuda")
    E = torch.empty_like(T)
    S = gh.slack(lv, makespan=T, energy=E)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == skind, gh.info()
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    ok = ~np.isnan(T_or)
    assert not ok[11]
    parity.assert_eval(host(T), host(E), T_or, E_or, True, f"scan first {case}")
    Sh = host(S)
    assert np.all(np.isnan(Sh[~ok]))
    _, _, S_or = oracle.slack_batch(g, rows[ok], nthreads=8)
    parity.assert_slack(Sh[ok], S_or, T_or[ok], True, f"scan first {case} slack")
    T1, E1 = gh.eval_policies(lv)
    torch.cuda.synchronize()
    # one kernel while its (time, energy) table fits its 64 KB of LDS, else the segmented kernels
    assert gh.info()["last_kernels"] == (1 if P <= 2048 and P * F * 8 <= 65536 else 2), gh.info()
    assert np.array_equal(host(T).view(np.uint32), host(T1).view(np.uint32))
    # (energy blocks are grouped per chain window here, in program order there)
    parity.assert_eval(host(T1), host(E1), T_or, E_or, True, f"scan first {case} eval")
    buf = torch.empty(len(rows) * P + 1, dtype=torch.float32, device="cuda")
    S2 = buf[1:].view(len(rows), P)
    gh.slack(lv, out=S2)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] not in (6, 8), gh.info()
    assert np.array_equal(Sh.view(np.uint32), host(S2).view(np.uint32)), case


def fixed_chains_graph(rng, lengths):
    """Chains that mix packs with fixed-duration nodes (a fixed node every third step), constant
    floors from one host node every 50 steps, and chains of the given lengths."""
    src, dst, pack, dur = [], [], [], []
    h0 = 0   # a host node: candidate-independent floor for some chain nodes
    pack.append(-1)
    dur.append(5.0)
    P = 0
    for L in lengths:
        prev = None
        for k in range(L):
            v = len(pack)
            if k % 3 == 2:
                pack.append(-1)
                dur.append(float(synth.quantize(rng.uniform(0.5, 6.0))))
            else:
                pack.append(P)
                P += 1
                dur.append(0.0)
            if prev is not None:
                src.append(prev)
                dst.append(v)
            if k % 50 == 0:
                src.append(h0)
                dst.append(v)
            prev = v
    V = len(pack)
    F = 8
    t = np.sort(synth.quantize(rng.uniform(1.0, 30.0, (P, F))), axis=1)[:, ::-1].copy()
    e = (0.7 * t * rng.uniform(0.2, 1.0, (P, F))).astype(np.float32)
    g = synth.Graph("chains-with-fixed", V, np.asarray(src, np.int32), np.asarray(dst, np.int32),
                    np.asarray(pack, np.int32), np.asarray(dur, np.float32), P, F, t, e, 0.3)
    return g


@pytest.mark.parametrize("lengths", [[3100, 2900, 3400], [3100, 2900, 3406], [768] * 16],
                         ids=["unaligned-rows", "windowed", "scan-full"])
def test_chain_lanes_with_fixed_nodes(torch, emo, lengths):
    """Chains that mix packs with fixed-duration nodes (which depend on the candidate through the
    pack before them), constant floors from a host node, and chains of different lengths (6268
    packs: windowed kernels on rows that are not 16-byte aligned; 6272 packs: windowed kernels;
    16 chains of 512 packs: the two-pass scan with per-thread copy plans, every 256-pack window
    full), and the lane-per-chain kernel (unaligned level buffer) bit for bit."""
    rng = np.random.default_rng(42)
    g = fixed_chains_graph(rng, lengths)
    V, P = g.num_nodes, g.num_packs
    rows = pins.random_rows(rng, g, 300)
    print(f"[case] chain lanes with fixed nodes: V={V} P={P}", flush=True)
    gh = emo.EmoGraph(g, device=0)
    full = len(lengths) == 16
    assert gh.info()["chain_lanes"] == (16 if full else 4)
    # (rows that are not 16-byte aligned: windows narrow enough for one level piece per thread)
    win = 256 if full else (64 if P % 16 == 0 else 32)
    assert gh.info()["chain_window"] == win
    assert gh.info()["chain_scan_window"] == win
    lv = dev(torch, rows)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    T, E = gh.eval_policies(lv)
    S = gh.slack(lv)
    # (3 chains are too few for the per-thread plans of 64-pack windows)
    assert gh.info()["chain_scan_full"] == (1 if full else 0)
    assert gh.info()["last_kernels"] == (8 if full else 6)
    parity.assert_eval(host(T), host(E), T_or, E_or, True, "chains with fixed nodes")
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in range(len(rows))])
    parity.assert_slack(host(S), S_or, T_or, True, "chains with fixed nodes: pack slack")
    # the lane-per-chain kernel on the same rows (an unaligned level buffer): bit for bit
    lm = misaligned(torch, rows)
    Tm, _ = gh.eval_policies(lm)
    Sm = gh.slack(lm)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == 3
    assert np.array_equal(host(T).view(np.uint32), host(Tm).view(np.uint32))
    assert np.array_equal(host(S).view(np.uint32), host(Sm).view(np.uint32))
    check_windowed_off_grid(torch, emo, g, rows, win, "chains with fixed nodes")


def skewed_chains(seed, P, S, F, share):
    """P kernels on S streams, stream 0 taking `share` of them, each launched by a node of one
    host launch chain: in a window of the scan kernel one chain holds far more than 64 steps."""
    rng = np.random.default_rng(seed)
    stream = np.where(rng.random(P) < share, 0, rng.integers(1, S, P))
    src, dst, pack, dur = [], [], [], []
    last = {}
    prev_h = None
    for p in range(P):
        h = len(pack)
        pack.append(-1)
        dur.append(float(synth.quantize(rng.uniform(0.5, 3.0))))
        if prev_h is not None:
            src.append(prev_h)
            dst.append(h)
        prev_h = h
        k = len(pack)
        pack.append(p)
        dur.append(0.0)
        src.append(h)
        dst.append(k)
        if stream[p] in last:
            src.append(last[stream[p]])
            dst.append(k)
        last[stream[p]] = k
    t = np.sort(synth.quantize(rng.uniform(1.0, 30.0, (P, F))), axis=1)[:, ::-1].copy()
    e = (0.7 * t * rng.uniform(0.2, 1.0, (P, F))).astype(np.float32)
    return synth.Graph(f"skewed-{P}k-{S}s", len(pack), np.asarray(src, np.int32), np.asarray(dst, np.int32),
                       np.asarray(pack, np.int32), np.asarray(dur, np.float32), P, F, t, e, 0.3)


def test_chain_scan_long_window_lists(torch, emo):
    """Two-pass scan kernel where one chain holds about 230 steps of a 256-pack window (records
    loaded 64 at a time), with an invalid level and a ragged batch, against the oracle."""
    g = skewed_chains(5, 8448, 16, 16, 0.9)
    gh = emo.EmoGraph(g, device=0)
    assert gh.info()["chain_scan_window"] == 256, gh.info()
    assert gh.info()["chain_scan_full"] == 1, gh.info()
    rng = np.random.default_rng(6)
    rows = pins.random_rows(rng, g, 130)
    rows[77, 4000] = 16
    print(f"[case] chain scan, long window lists: V={g.num_nodes} P={g.num_packs}", flush=True)
    lv = dev(torch, rows)
    T, E = gh.eval_policies(lv)
    S = gh.slack(lv)
    torch.cuda.synchronize()
    assert gh.info()["last_kernels"] == 8
    T_or, E_or, S_or = oracle.slack_batch(g, rows, nthreads=8)
    assert np.isnan(T_or[77])
    parity.assert_eval(host(T), host(E), T_or, E_or, True, "skewed chains")
    parity.assert_slack(host(S), S_or, T_or, True, "skewed chains slack")


@pytest.mark.parametrize("mode", [0, 1], ids=["auto", "interpreted"])
def test_scratch_reuse_across_streams(torch, emo, mode):
    """One handle used from two streams with batches that grow and shrink: the calls share the
    handle's scratch and must still give exactly the single-stream results."""
    g = synth.packed_graph(9, 1024, 8, 16, sync_every=128, cross_p=0.05)
    rng = np.random.default_rng(11)
    sizes = [300, 2000, 64, 4096, 1000, 4096]
    rows = [pins.random_rows(rng, g, n) for n in sizes]
    print(f"[case] scratch reuse mode={mode}: sizes={sizes}", flush=True)
    gh = emo.EmoGraph(g, device=0, kernel_mode=mode)
    lvs = [dev(torch, r) for r in rows]
    ref = []
    for lv in lvs:   # reference: one stream, synchronised after each call
        S = gh.slack(lv)
        T, E = gh.eval_policies(lv)
        torch.cuda.synchronize()
        ref.append((host(S).copy(), host(T).copy(), host(E).copy()))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = []
    for i, lv in enumerate(lvs):   # alternate streams without host synchronisation
        st = streams[i % 2]
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            S = torch.empty((lv.shape[0], g.num_packs), dtype=torch.float32, device="cuda")
            gh.slack(lv, out=S, stream=st)
            T, E = gh.eval_policies(lv, stream=st)
        outs.append((S, T, E))
    torch.cuda.synchronize()
    for (S, T, E), (Sr, Tr, Er) in zip(outs, ref):
        assert np.array_equal(host(S).view(np.uint32), Sr.view(np.uint32))
        assert np.array_equal(host(T).view(np.uint32), Tr.view(np.uint32))
        assert np.array_equal(host(E).view(np.uint32), Er.view(np.uint32))
    T_or, E_or = oracle.eval_batch(g, rows[3], nthreads=8)
    parity.assert_eval(ref[3][1], ref[3][2], T_or, E_or, True, "scratch reuse")


def test_scratch_with_many_streams(torch, emo):
    """Calls from twelve streams without host synchronisation: the first eight streams get a
    scratch buffer each, the others share one ordered by an event; growing batches make every
    kind of buffer grow while earlier calls may still be running.  Every result equals the
    single-stream one bit for bit."""
    g = synth.packed_graph(9, 1024, 8, 16, sync_every=128, cross_p=0.05)
    rng = np.random.default_rng(12)
    sizes = [64, 300, 1000, 2000, 4096, 128, 3000, 700, 4096, 50, 2500, 4096] * 2
    rows = [pins.random_rows(rng, g, n) for n in sizes[:12]]
    print(f"[case] scratch with 12 streams", flush=True)
    gh = emo.EmoGraph(g, device=0)
    lvs = [dev(torch, r) for r in rows]
    ref = []
    for lv in lvs:
        S = gh.slack(lv)
        T, E = gh.eval_policies(lv)
        torch.cuda.synchronize()
        ref.append((host(S).copy(), host(T).copy(), host(E).copy()))
    gh2 = emo.EmoGraph(g, device=0)
    streams = [torch.cuda.Stream() for _ in range(12)]
    outs = []
    for i, n in enumerate(sizes):
        st = streams[i % 12]
        lv = lvs[i % 12]
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            S = torch.empty((lv.shape[0], g.num_packs), dtype=torch.float32, device="cuda")
            gh2.slack(lv, out=S, stream=st)
            T, E = gh2.eval_policies(lv, stream=st)
            res, _ = emo.select_from_results(T, E, 1e9, stream=st)
        outs.append((i % 12, S, T, E, res))
    torch.cuda.synchronize()
    for j, S, T, E, res in outs:
        Sr, Tr, Er = ref[j]
        assert np.array_equal(host(S).view(np.uint32), Sr.view(np.uint32)), j
        assert np.array_equal(host(T).view(np.uint32), Tr.view(np.uint32)), j
        assert np.array_equal(host(E).view(np.uint32), Er.view(np.uint32)), j
        sel = emo.parse_selection(res)
        assert sel.num_feasible == len(Tr) and sel.index == int(np.argmin(Er)), j


def test_large_slot_count_uses_device_scratch(torch, emo):
    """A wide antichain of packs feeding one sink keeps many finish times live at once."""
    rng = np.random.default_rng(5)
    W = 3000
    V = W + 2
    src = [0] * W + list(range(1, W + 1))
    dst = list(range(1, W + 1)) + [W + 1] * W
    pack = np.full(V, -1, np.int32)
    pack[1:W + 1] = np.arange(W)
    F = 4
    t = np.sort(synth.quantize(rng.uniform(1, 50, (W, F))), axis=1)[:, ::-1].copy()
    e = rng.uniform(0, 3, (W, F)).astype(np.float32)
    g = synth.Graph("antichain", V, np.asarray(src, np.int32), np.asarray(dst, np.int32), pack,
                    synth.quantize(rng.uniform(1, 9, V)), W, F, t, e, 0.25)
    rows = pins.random_rows(rng, g, 777)
    gh = emo.EmoGraph(g, device=0)
    assert gh.info()["eval_slots"] >= W
    T_or, _ = oracle.eval_batch(g, rows)
    run_all(torch, emo, g, rows, [float(np.median(T_or))], what="antichain")


@pytest.mark.parametrize("mode", [0, 1], ids=["auto", "interpreted"])
def test_edge_cases(torch, emo, mode):
    g = pins.graph_from_golden(pins.load_golden())
    gh = emo.EmoGraph(g, device=0, kernel_mode=mode)
    # B = 0
    empty = torch.zeros((0, g.num_packs), dtype=torch.uint8, device="cuda")
    T, E = gh.eval_policies(empty)
    res, _ = gh.select_policy(empty, 100.0)
    sel = emo.parse_selection(res)
    assert sel.index == -1 and sel.num_feasible == 0 and np.isnan(sel.energy)
    S = gh.slack(empty)
    assert S.shape == (0, g.num_packs)
    # invalid level bytes: NaN results, never feasible
    rows = np.asarray([[1, 1, 1], [2, 0, 0], [1, 1, 255], [0, 0, 0]], np.uint8)
    T, E = gh.eval_policies(dev(torch, rows))
    Th, Eh = host(T), host(E)
    assert np.isnan(Th[1]) and np.isnan(Th[2]) and np.isnan(Eh[1]) and np.isnan(Eh[2])
    assert Th[0] == 16.0 and Th[3] == 22.0
    S = host(gh.slack(dev(torch, rows)))
    assert np.all(np.isnan(S[1])) and np.all(np.isnan(S[2])) and not np.any(np.isnan(S[0]))
    res, mask = gh.select_policy(dev(torch, rows), 1e9)
    sel = emo.parse_selection(res)
    assert sel.num_feasible == 2 and emo.unpack_mask(mask, 4).tolist() == [True, False, False, True]
    assert sel.index == 3 and sel.makespan == 22.0
    # all rows identical: ties go to the lowest index
    rows = np.tile(np.asarray([[0, 1, 0]], np.uint8), (1000, 1))
    res, _ = gh.select_policy(dev(torch, rows), 1e9)
    assert emo.parse_selection(res).index == 0
    rows[:500] = 1   # all packs at the higher level: more energy, so the cheapest rows start at 500
    res, _ = gh.select_policy(dev(torch, rows), 1e9)
    T_or, E_or = oracle.eval_batch(g, rows)
    assert emo.parse_selection(res).index == oracle.select(T_or, E_or, 1e9)[0]
    # target below every makespan
    res, mask = gh.select_policy(dev(torch, rows), 1.0)
    sel = emo.parse_selection(res)
    assert sel.index == -1 and sel.num_feasible == 0 and not emo.unpack_mask(mask, 1000).any()
    # empty graph and a graph without packs
    z = np.zeros(0, np.int32)
    zf = np.zeros((0, 1), np.float32)
    ge = synth.Graph("empty", 0, z, z, z, np.zeros(0, np.float32), 0, 1, zf, zf, 0.5)
    gh0 = emo.EmoGraph(ge, device=0, kernel_mode=mode)
    T, E = gh0.eval_policies(torch.zeros((5, 0), dtype=torch.uint8, device="cuda"))
    assert host(T).tolist() == [0.0] * 5 and host(E).tolist() == [0.0] * 5
    gn = synth.Graph("nopacks", 3, np.asarray([0, 1], np.int32), np.asarray([1, 2], np.int32),
                     np.full(3, -1, np.int32), np.asarray([1.0, 2.0, 4.0], np.float32), 0, 1,
                     zf, zf, 0.5)
    ghn = emo.EmoGraph(gn, device=0, kernel_mode=mode)
    T, E = ghn.eval_policies(torch.zeros((3, 0), dtype=torch.uint8, device="cuda"))
    assert host(T).tolist() == [7.0] * 3 and host(E).tolist() == [3.5] * 3
    SN = host(ghn.slack(torch.zeros((3, 0), dtype=torch.uint8, device="cuda"), per_node=True))
    assert SN.tolist() == [[0.0, 0.0, 0.0]] * 3


@pytest.mark.parametrize("mode", [0, 1], ids=["auto", "interpreted"])
def test_determinism(torch, emo, mode):
    g = synth.config_graph(3)
    rows = synth.config_policies(3, g, 0, 20000)
    gh = emo.EmoGraph(g, device=0, kernel_mode=mode)
    lv = dev(torch, rows)
    a = [host(x).copy() for x in gh.eval_policies(lv)]
    b = [host(x).copy() for x in gh.eval_policies(lv)]
    assert all(np.array_equal(x.view(np.uint32), y.view(np.uint32)) for x, y in zip(a, b))
    s1 = host(gh.slack(lv[:2000])).copy()
    s2 = host(gh.slack(lv[:2000])).copy()
    assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32))


@pytest.mark.parametrize("mode", [0, 1], ids=["auto", "interpreted"])
def test_selection_across_calls(torch, emo, mode):
    """Calls that select, calls that do not (which reuse the same scratch buffer for other data)
    and selections from stored results, with batches that shrink and grow, on one stream: every
    selection matches the oracle's."""
    rng = np.random.default_rng(4242 + mode)
    g = synth.random_dag(rng, 180, 3.0 / 180, 0.6, 9)
    rows = pins.random_rows(rng, g, 70001)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=8)
    gh = emo.EmoGraph(g, device=0, kernel_mode=mode)
    lv = dev(torch, rows)
    tq = [float(np.float32(np.quantile(T_or, q))) for q in (0.05, 0.5, 1.0)]
    for n, tgt in ((70001, tq[0]), (513, tq[1]), (70001, tq[2]), (1, tq[2]), (40000, tq[0]), (256, tq[1])):
        print(f"[case] across calls mode={mode} B={n} target={tgt}", flush=True)
        res, mask = gh.select_policy(lv[:n], tgt)
        parity.assert_selection(emo.parse_selection(res), emo.unpack_mask(mask, n), T_or[:n], E_or[:n],
                                tgt, True, f"select B={n}")
        T, E = gh.eval_policies(lv[:n])                        # no selection: scratch reused
        S = gh.slack(lv[:min(n, 3000)])
        del S
        res2, mask2 = emo.select_from_results(T, E, tgt)
        parity.assert_selection(emo.parse_selection(res2), emo.unpack_mask(mask2, n), T_or[:n], E_or[:n],
                                tgt, True, f"select_from_results B={n}")
    gh.close()


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_workload_full_batch(torch, emo, k):
    """Every candidate of workload k: makespan/energy of all rows, masks and selection for each
    target, slack on sampled rows (slack of all rows is computed, as the benchmark does)."""
    spec = synth.CONFIGS[k]
    g = synth.config_graph(k)
    B = spec.num_candidates
    print(f"[case] workload {k} {spec.name} B={B}", flush=True)
    if spec.exhaustive:
        rows = synth.config_policies(k, g)
    else:
        rows = synth.random_policies_parallel(spec.policy_seed, g.num_packs, g.num_levels, B, workers=8)
    T_or, E_or = oracle.eval_batch(g, rows, nthreads=16)
    T0 = float(np.min(T_or)) if spec.exhaustive else float(T_or[0])
    assert np.all(rows[0 if not spec.exhaustive else -1] == g.num_levels - 1)
    gh = emo.EmoGraph(g, device=0)
    lv = dev(torch, rows)
    T, E = gh.eval_policies(lv)
    parity.assert_eval(host(T), host(E), T_or, E_or, True, spec.name)
    # one specialised kernel up to 2048 steps, cut-segment kernels for the 4096-pack graph (16
    # synchronisations), chain lanes for the 65536-kernel graph (16 stream chains)
    inf = gh.info()
    assert inf["last_kernels"] == {1: 1, 2: 1, 3: 1, 4: 5, 5: 4}[k], inf
    if k <= 4:
        # the interpreting kernels on the same batch: bit-identical
        gi = emo.EmoGraph(g, device=0, kernel_mode=1)
        Ti, Ei = gi.eval_policies(lv)
        assert torch.equal(Ti.view(torch.int32), T.view(torch.int32))
        assert torch.equal(Ei.view(torch.int32), E.view(torch.int32))
        tgt = float(np.float32(spec.targets[0] * (float(np.min(T_or)) if spec.exhaustive else float(T_or[0]))))
        res_i, mask_i = gi.select_policy(lv, tgt)
        parity.assert_selection(emo.parse_selection(res_i), emo.unpack_mask(mask_i, B), T_or, E_or,
                                tgt, True, f"{spec.name} interpreted select")
        gi.close()
    for r in spec.targets:
        tgt = float(np.float32(r * T0))
        res, mask = gh.select_policy(lv, tgt)
        parity.assert_selection(emo.parse_selection(res), emo.unpack_mask(mask, B), T_or, E_or,
                                tgt, True, f"{spec.name} select@{r}")
        res2, mask2 = emo.select_from_results(T, E, tgt)
        parity.assert_selection(emo.parse_selection(res2), emo.unpack_mask(mask2, B), T_or, E_or,
                                tgt, True, f"{spec.name} select_from_results@{r}")
    pick = synth.sample_rows(B, 24)
    S = gh.slack(lv)
    # slack: one kernel while every finish time fits in registers, then segmented kernels
    # (cut segments for the 4096-pack graph)
    assert gh.info()["last_kernels"] == {1: 1, 2: 1, 3: 2, 4: 5, 5: 8}[k], gh.info()
    S_or = np.stack([oracle.pack_slack(g, rows[c]) for c in pick])
    idx = torch.from_numpy(pick).cuda()
    parity.assert_slack(host(S.index_select(0, idx)), S_or, T_or[pick], True, spec.name + " slack")
    if k in (3, 4, 5):
        # segmented / chain-lane slack against the interpreting kernels on a leading slice
        gi = emo.EmoGraph(g, device=0, kernel_mode=1)
        nb = min(B, 8192)
        Si = gi.slack(lv[:nb])
        assert torch.equal(Si.view(torch.int32), S[:nb].view(torch.int32)), spec.name
        gi.close()
    del S
    # per-node slack over a leading slice
    nb = min(B, 512)
    SN = gh.slack(lv[:nb], per_node=True)
    pick2 = synth.sample_rows(nb, 6)
    SN_or = np.stack([oracle.slack(g, rows[c]).slack for c in pick2])
    parity.assert_slack(host(SN)[pick2], SN_or, T_or[pick2], True, spec.name + " node slack")
    gh.close()
