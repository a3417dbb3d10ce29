"""How far the policy search of Alg. 2 (one frequency interval per pack) lands from the exhaustive
optimum, on graphs small enough to enumerate every policy.  Runs on the CPU with the oracle only:

    python tests/dp_gap_report.py

On a DAG the discretised makespan is not a sufficient state (two policies with the same makespan
bucket can differ in the slack they leave on other paths), so the search keeps one policy per
bucket and can miss the optimum; on a chain with one-grid-step buckets it is exact.  The report
gives, per setting, the share of searches that find the optimum and the mean and largest relative
energy excess over it.
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

from oracle import dp, eval_batch  # noqa: E402
from paper_2607_12324_amd import synth  # noqa: E402


def gap(g, target, quantum):
    r = dp.dp_search(g, target, quantum)
    lv, e_opt, _ = dp.exhaustive_best(g, target)
    if lv is None:
        assert r.levels is None
        return None
    assert r.levels is not None and r.energy >= e_opt
    return (r.energy - e_opt) / e_opt


def summarize(name, gaps):
    g = np.asarray([x for x in gaps if x is not None])
    if g.size == 0:
        print(f"| {name} | 0 | - | - | - |")
        return
    print(f"| {name} | {g.size} | {np.mean(g == 0.0):.2f} | {g.mean():.2e} | {g.max():.2e} |")


def main():
    print("| setting | searches | optimum found | mean excess | max excess |")
    print("|---|---|---|---|---|")
    g = synth.config_graph(1)                      # 8 packs x 4 levels: 65,536 policies
    T0 = float(eval_batch(g, np.full((1, g.num_packs), g.num_levels - 1, np.uint8))[0][0])
    for div in (16, 64, 256):
        q = T0 / div
        gaps = [gap(g, float(np.float32(T0 * r)), q) for r in (1.0, 1.02, 1.05, 1.1, 1.2, 1.4)]
        summarize(f"tiny 8-pack workload, quantum T0/{div}, targets 1.0-1.4 T0", gaps)
    gaps = [gap(g, float(np.float32(T0 * r)), synth.Q) for r in (1.0, 1.02, 1.05, 1.1, 1.2, 1.4)]
    summarize("tiny 8-pack workload, quantum = time grid (2^-4 us)", gaps)
    for q_exp in (-4, 0, 2):
        rng = np.random.default_rng(900 + q_exp)
        gaps = []
        while len(gaps) < 150:
            gr = synth.random_dag(rng, int(rng.integers(3, 10)), float(rng.uniform(0.2, 0.6)), 0.7,
                                  int(rng.integers(2, 4)))
            if gr.num_packs == 0 or gr.num_levels ** gr.num_packs > 4096:
                continue
            T0 = float(eval_batch(gr, np.full((1, gr.num_packs), gr.num_levels - 1, np.uint8))[0][0])
            gaps.append(gap(gr, float(np.float32(T0 * rng.uniform(1.0, 1.3))), 2.0 ** q_exp))
        summarize(f"random DAGs (<= 4096 policies), quantum 2^{q_exp} us", gaps)


if __name__ == "__main__":
    main()
