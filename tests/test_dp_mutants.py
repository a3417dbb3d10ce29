"""Plant plausible mistakes in copies of the policy-search oracle (on the CPU) and check that
its pins catch every one: a wrong tie rule, a strict latency test, the wrong interval changed, a
state table not kept per bucket."""
import importlib.util
import os
import sys

import numpy as np
import pytest

import test_dp_oracle as pins_dp
from oracle import dp

SRC = os.path.abspath(dp.__file__)

MUTANTS = {
    "strict_latency": ("ok = np.nonzero(T32 <= t_max)[0]", "ok = np.nonzero(T32 < t_max)[0]"),
    "bucket_tie_takes_last": ("np.lexsort((ok, E32[ok], bucket[ok]))",
                              "np.lexsort((-ok, E32[ok], bucket[ok]))"),
    "answer_tie_highest_bucket": ("np.lexsort((table.bucket[ok], table.energy[ok]))",
                                  "np.lexsort((-table.bucket[ok], table.energy[ok]))"),
    "answer_least_makespan": ("np.lexsort((table.bucket[ok], table.energy[ok]))",
                              "np.lexsort((table.energy[ok], table.bucket[ok]))"),
    "wrong_interval": ("X[:, interval] = np.tile", "X[:, (interval + 1) % X.shape[1]] = np.tile"),
    "one_state_per_stage": ("first[1:] = bucket[order][1:] != bucket[order][:-1]",
                            "first[1:] = False"),
    "bucket_by_rounding": ("np.floor(T32.astype(np.float64) / quantum)",
                           "np.round(T32.astype(np.float64) / quantum)"),
    "highest_level_skipped": ("np.tile(np.arange(F, dtype=np.uint8)",
                              "np.tile(np.arange(F, dtype=np.uint8) * 0 + np.minimum(np.arange(F), F - 2).astype(np.uint8)"),
}


def _load_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found"
    pkg = tmp_path / "oracle_mut"
    pkg.mkdir()
    # the mutant imports the real predictor: `from . import eval_batch` becomes absolute
    (pkg / "dp.py").write_text(src.replace(old, new).replace("from . import eval_batch",
                                                             "from oracle import eval_batch"))
    spec = importlib.util.spec_from_file_location(f"dp_mut_{name}", str(pkg / "dp.py"))
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod
    spec.loader.exec_module(mod)
    return mod


PINS = [pins_dp.test_dp_handworked, lambda: [pins_dp.test_dp_is_exact_on_chains(s) for s in range(4)],
        lambda: [pins_dp.test_dp_invariants_on_dags(s) for s in range(4)]]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_dp_pins_catch_planted_mistake(oracle_lib, tmp_path, name, monkeypatch):
    old, new = MUTANTS[name]
    mod = _load_mutant(tmp_path, name, old, new)
    monkeypatch.setattr(pins_dp, "dp", mod)
    caught = 0
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except (AssertionError, ValueError, IndexError, TypeError):
            caught += 1
    assert caught, f"no pin caught mutant {name}"
