"""The benchmark's step at each workload's full size, against the oracle (needs an MI355X).

The step is the call bench.py times: one evaluation of the whole batch (makespan, energy, slack
of every pack when the workload has the backward pass, and a mask and a selection for every
latency target), through emo_evaluate with one target and emo_evaluate_targets with several.
Makespans, energies, masks and selections are compared on every candidate; emo_select_from_results
on the stored makespans and energies is checked against the same selections.  Slack is compared element by element on every row
of the two smaller workloads, and on a leading slice plus every row of the last workgroups of
the three larger ones (65,536 rows of the 512- and 4096-pack graphs, 4,096 of the 65,536-kernel
graph), the oracle computing them on all host cores.  The 4096-pack and 65,536-kernel graphs
with every table time scaled by 1.1 (off the exact-sum grid, as the benchmark's variants) are
checked the same way within the off-grid tolerance: 1e-5 of the makespan, and every mask bit
whose candidate's makespan is not within that bound of the target.
"""
import os

import numpy as np
import pytest

import oracle
import parity
from paper_2607_12324_amd import synth

pytestmark = pytest.mark.gpu

NT = min(16, os.cpu_count() or 1)
SLICE = {1: None, 2: None, 3: 65536, 4: 65536, 5: 4096}   # None: every row
TAIL = 1024                                                 # rows at the batch's end
CHUNK_ELEMS = 1 << 26                                       # oracle slack compared in pieces


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


@pytest.fixture(scope="module")
def emo(torch):
    from paper_2607_12324_amd import emo as mod
    return mod


def host(t):
    return t.detach().cpu().numpy()


def slack_rows(B, k):
    """Rows whose slack is compared: all, or a leading slice and the batch's last rows."""
    n = SLICE[k]
    if n is None or n + TAIL >= B:
        return np.arange(B, dtype=np.int64)
    return np.concatenate([np.arange(n), np.arange(B - TAIL, B)]).astype(np.int64)


def compare_slack(torch, g, rows, S_dev, pick, T_or, what, exact=True):
    """Oracle slack of rows[pick] against the device slack rows, in pieces of bounded size."""
    step = max(1, CHUNK_ELEMS // max(1, g.num_packs))
    for a in range(0, len(pick), step):
        idx = pick[a:a + step]
        _, _, S_or = oracle.slack_batch(g, rows[idx], nthreads=NT)
        sel = torch.from_numpy(idx).to(S_dev.device)
        S = host(S_dev.index_select(0, sel))
        parity.assert_slack(S, S_or, T_or[idx], exact, f"{what} rows {idx[0]}..{idx[-1]}")
        print(f"  slack rows {idx[0]}..{idx[-1]} ok", flush=True)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_bench_step_full_size(torch, emo, k):
    run_step(torch, emo, k, synth.config_graph(k), True)


@pytest.mark.parametrize("k", [4, 5])
def test_bench_step_off_grid(torch, emo, k):
    run_step(torch, emo, k, synth.scaled_times(synth.config_graph(k), 1.1), False)


def run_step(torch, emo, k, g, exact):
    """The benchmark's step of workload k on graph g (its own or a variant with the same packs
    and levels) against the oracle; exact: bit for bit where the comparison rules allow."""
    spec = synth.CONFIGS[k]
    B, P = spec.num_candidates, g.num_packs
    print(f"[case] bench step, workload {k} {g.name}: B={B} P={P}", flush=True)
    rows = synth.bench_policies(k, g)
    assert np.all(rows[0] == g.num_levels - 1)
    if spec.slack and SLICE[k] is None:
        T_or, E_or, S_or_all = oracle.slack_batch(g, rows, nthreads=NT)
    else:
        T_or, E_or = oracle.eval_batch(g, rows, nthreads=NT)
        S_or_all = None
    print("  oracle done", flush=True)
    T0 = float(T_or[0])
    targets = [float(np.float32(r * T0)) for r in spec.targets]

    dev = torch.device("cuda", 0)
    gh = emo.EmoGraph(g, device=0)
    lv = torch.from_numpy(rows).to(dev)
    T = torch.empty(B, dtype=torch.float32, device=dev)
    E = torch.empty(B, dtype=torch.float32, device=dev)
    S = torch.empty((B, P), dtype=torch.float32, device=dev) if spec.slack else None
    masks = [torch.empty((B + 31) // 32, dtype=torch.int32, device=dev) for _ in targets]
    res_all = torch.empty((len(targets), 3), dtype=torch.int64, device=dev)
    results = [res_all[j] for j in range(len(targets))]
    # the benchmark's call
    if len(targets) == 1:
        gh.evaluate(lv, makespan=T, energy=E, slack=S, latency_target=targets[0], mask=masks[0],
                    result=results[0])
    else:
        gh.evaluate_targets(lv, targets, makespan=T, energy=E, slack=S, masks=masks, results=res_all)
    torch.cuda.synchronize()
    print(f"  device step done (kernels {gh.info()['last_kernels']})", flush=True)

    parity.assert_eval(host(T), host(E), T_or, E_or, exact, g.name)
    for tgt, m, r in zip(targets, masks, results):
        bits = emo.unpack_mask(m, B)
        parity.assert_selection(emo.parse_selection(r), bits, T_or, E_or, tgt, exact,
                                f"{g.name} select@{tgt}")
        if not exact:
            _, feas_or, _ = oracle.select(T_or, E_or, tgt)
            clear = np.isnan(T_or) | (np.abs(T_or - tgt) > parity.REL * np.abs(T_or))
            assert np.array_equal(bits[clear], feas_or[clear]), f"{g.name} mask@{tgt}"
    for tgt, m, r in zip(targets, masks, results):
        r2, m2 = emo.select_from_results(T, E, tgt)
        assert np.array_equal(host(r2), host(r)) and np.array_equal(host(m2), host(m)), tgt
    print("  makespan, energy, masks and selections ok", flush=True)

    if S_or_all is not None:
        parity.assert_slack(host(S), S_or_all, T_or, exact, g.name + " slack, every row")
        print("  slack of every row ok", flush=True)
    else:
        if S is None:
            # the step has no backward pass: the slack entry point on the compared rows
            n = SLICE[k]
            S = gh.slack(lv[:n])
            pick = np.arange(n, dtype=np.int64)
        else:
            pick = slack_rows(B, k)
        compare_slack(torch, g, rows, S, pick, T_or, g.name + " slack", exact)
    gh.close()
