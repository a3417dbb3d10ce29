"""emo_select_from_results_noalloc (static scratch, no allocation) through the C ABI against
emo_select_from_results and the oracle's selection, on two calls in a row with the second on a
smaller batch (the array keeps the first call's records), plus its size limit (needs an
MI355X)."""
import ctypes

import numpy as np
import pytest

import oracle
import parity

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


def results(rng, B):
    """Makespans on a coarse grid (many exact ties with the target) with a few NaNs, energies
    with repeated values (ties broken by index)."""
    T = (rng.integers(900, 1100, B) / 4.0).astype(np.float32)
    T[rng.choice(B, size=max(1, B // 1000), replace=False)] = np.nan
    E = (rng.integers(1, 5000, B) / 8.0).astype(np.float32)
    return T, E


@pytest.mark.parametrize("sizes", [(3_000_001, 70_001), (1 << 20, 1000)])
def test_noalloc_selection_matches(torch, emo, sizes):
    rng = np.random.default_rng(sum(sizes))
    dev = torch.device("cuda", 0)
    for B in sizes:
        print(f"[case] select_from_results_noalloc B={B}", flush=True)
        T, E = results(rng, B)
        Td, Ed = torch.from_numpy(T).to(dev), torch.from_numpy(E).to(dev)
        target = float(np.float32(250.0))
        m_ref = torch.empty((B + 31) // 32, dtype=torch.int32, device=dev)
        r_ref = torch.empty(3, dtype=torch.int64, device=dev)
        emo.select_from_results(Td, Ed, target, mask=m_ref, result=r_ref)
        m = torch.full(((B + 31) // 32,), -1, dtype=torch.int32, device=dev)
        r = torch.full((3,), -7, dtype=torch.int64, device=dev)
        emo.select_from_results_noalloc(Td, Ed, target, mask=m, result=r)
        torch.cuda.synchronize()
        assert torch.equal(m, m_ref), "mask words differ from emo_select_from_results"
        assert torch.equal(r, r_ref), (emo.parse_selection(r), emo.parse_selection(r_ref))
        parity.assert_selection(emo.parse_selection(r), emo.unpack_mask(m, B), T.astype(np.float64),
                                E.astype(np.float64), target, True, f"noalloc B={B}")
        # without a mask, and with a target nothing meets
        r2 = torch.empty(3, dtype=torch.int64, device=dev)
        emo.select_from_results_noalloc(Td, Ed, target, mask=None, result=r2)
        r3 = torch.empty(3, dtype=torch.int64, device=dev)
        emo.select_from_results_noalloc(Td, Ed, 1.0, mask=None, result=r3)
        torch.cuda.synchronize()
        assert torch.equal(r2, r_ref)
        s3 = emo.parse_selection(r3)
        assert s3.index == -1 and s3.num_feasible == 0 and np.isnan(s3.energy)
        idx, _, n = oracle.select(T.astype(np.float64), E.astype(np.float64), target)
        assert emo.parse_selection(r).index == idx and emo.parse_selection(r).num_feasible == n


def test_noalloc_limits(torch, emo):
    """B = 0 writes the empty selection; a batch beyond the static scratch is rejected on the
    host before anything is launched (the small buffers passed are never touched)."""
    dev = torch.device("cuda", 0)
    T = torch.zeros(4, dtype=torch.float32, device=dev)
    E = torch.zeros(4, dtype=torch.float32, device=dev)
    r = torch.zeros(3, dtype=torch.int64, device=dev)
    emo.select_from_results_noalloc(T[:0], E[:0], 1.0, mask=None, result=r)
    s = emo.parse_selection(r)
    assert s.index == -1 and s.num_feasible == 0
    too_many = (1 << 28) + 1
    st = emo.lib.emo_select_from_results_noalloc(ctypes.c_void_p(T.data_ptr()), ctypes.c_void_p(E.data_ptr()),
                                                 too_many, ctypes.c_float(1.0), None,
                                                 ctypes.c_void_p(r.data_ptr()), None)
    assert st == 1 and b"static scratch" in emo.lib.emo_last_error()
    torch.cuda.synchronize()
    assert emo.parse_selection(r).index == -1          # untouched by the rejected call
