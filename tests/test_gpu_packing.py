"""Packed graphs on the GPU (needs an MI355X): the library packs a per-kernel graph on the host
(emo_pack_kernels, emo_contract_packs), the evaluator runs both graphs through the C ABI, and
the results are checked against the oracle and against each other: the same makespan at the
default frequency (the rules keep every critical dependency, Sec. IV-D), never a larger one at
any level vector uniform within each pack, and the packed graph's makespan and energy equal to
the oracle's on sampled rows."""
import numpy as np
import pytest

import oracle
import packing_cases as pc
from oracle import packing
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


def fast_host(g):
    host = g.node_pack < 0
    g.node_duration[host] = synth.quantize(np.full(int(host.sum()), 0.25))
    return g


def graphs():
    return [
        ("unpacked-65536k-16s-F16", lambda: synth.config_graph(5), 5000.0, 1024),
        ("streams-8192k-16s-F16-fast-host",
         lambda: fast_host(synth._launch_graph(4, "fast-host", P=8192, S=16, F=16,
                                               packs_per_host=1, cross_p=0.0, n_cross_exact=None,
                                               median_us=8.0, sigma=1.2)), 5000.0, 4096),
        ("training-512p-4s-F16", lambda: synth.config_graph(3), 5000.0, 8192),
        ("packed-4096p-8s-F16", lambda: synth.config_graph(4), 200.0, 4096),
        ("streamdag-3", lambda: pc.stream_dag(3, 41, 4, F=6), 15.0, 8192),
    ]


@pytest.mark.parametrize("case", graphs(), ids=lambda c: c[0])
def test_packed_graph(torch, emo, case):
    name, make, lim, B = case
    print(f"[case] packed graph {name} bound {lim} B {B}", flush=True)
    g = make()
    grp, n = emo.pack_kernels(g, g.node_stream, lim)
    pg = emo.contract_packs(g, grp, n)
    F = g.num_levels
    rng = np.random.default_rng(17)
    rows = rng.integers(0, F, (B, n)).astype(np.uint8)
    mix = rng.random(B) < 0.5
    rows[mix, :] = np.where(                # half of the rows: mostly at the maximum
        rng.random((int(mix.sum()), n)) < 0.1,
                            rng.integers(0, F, (int(mix.sum()), n)), F - 1)
    rows[0] = F - 1
    kernel_rows = packing.expand_levels(grp, rows)
    hp = emo.EmoGraph(pg, device=0)
    hu = emo.EmoGraph(g, device=0)
    Tp, Ep = hp.eval_policies(torch.from_numpy(rows).cuda())
    Tu, Eu = hu.eval_policies(torch.from_numpy(kernel_rows).cuda())
    Tp, Ep, Tu, Eu = (x.cpu().numpy() for x in (Tp, Ep, Tu, Eu))
    assert Tp[0] == Tu[0], "all-maximum makespans differ"
    assert (Tp <= Tu).all()
    sample = np.unique(np.concatenate([[0, B - 1], rng.integers(0, B, 24)]))
    To, Eo = oracle.eval_batch(pg, rows[sample])
    assert np.all(np.abs(Tp[sample] - To) <= 1e-5 * To)
    assert np.all(np.abs(Ep[sample] - Eo) <= 1e-5 * Eo)
    print(f"[result] {name}: {g.num_packs} kernels -> {n} packs, "
          f"mean makespan gap {float(np.mean((Tu - Tp) / Tu)):.2e}", flush=True)
    hp.close()
    hu.close()


def test_model_tables_feed_the_evaluator(torch, emo):
    """Tables from the pack model (emo_pack_model, Eq. 6-7) on the 512-pack training graph,
    evaluated through the C ABI against the oracle on the same tables."""
    print("[case] pack-model tables on training-512p-4s-F16", flush=True)
    import dataclasses
    g = synth.config_graph(3)
    mi = synth.model_inputs(2, g.num_packs, g.num_levels)
    _, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, mi.pack_metrics)
    gm = dataclasses.replace(g, pack_time=T, pack_energy=E)
    rng = np.random.default_rng(3)
    rows = rng.integers(0, g.num_levels, (4096, g.num_packs)).astype(np.uint8)
    rows[0] = g.num_levels - 1
    h = emo.EmoGraph(gm, device=0)
    Tg, Eg = (x.cpu().numpy() for x in h.eval_policies(torch.from_numpy(rows).cuda()))
    sample = np.arange(0, 4096, 97)
    To, Eo = oracle.eval_batch(gm, rows[sample])
    assert np.all(np.abs(Tg[sample] - To) <= 1e-5 * To)
    assert np.all(np.abs(Eg[sample] - Eo) <= 1e-5 * Eo)
    h.close()
