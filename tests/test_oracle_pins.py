"""The oracle against its pins (CPU only)."""
import numpy as np
import pytest

import oracle
import pins
from paper_2607_12324_amd import synth


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(oracle_lib, pin):
    pin()


def test_bruteforce_off_grid(oracle_lib):
    pins.pin_bruteforce_paths(seed=77, count=40, on_grid=False)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_workload_paths_stay_on_exact_grid(oracle_lib, k):
    """Every path sum stays below 2**20 us, so sums of grid values are exact in fp32: checked on
    the slowest policy (all packs at level 0), whose makespan bounds every other policy's."""
    g = synth.config_graph(k)
    low = np.zeros((1, g.num_packs), dtype=np.uint8)
    T, _ = oracle.eval_batch(g, low)
    assert T[0] < 2.0 ** 20
    assert np.all(np.diff(g.pack_time.astype(np.float64), axis=1) <= 0)
    q = np.float64(synth.Q)
    assert np.all(np.mod(g.pack_time.astype(np.float64), q) == 0)
    assert np.all(np.mod(g.node_duration.astype(np.float64), q) == 0)


@pytest.mark.parametrize("k", [2, 3])
def test_invariants_on_workloads(oracle_lib, k):
    g = synth.config_graph(k)
    rows = synth.config_policies(k, g, 0, 3)
    pins.pin_invariants(g, rows, check_whatif=(k == 2))
