"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that the pins catch
every one: a dropped term, a wrong sign, a wrong comparison, a transposed index, an off-by-one."""
import os
import subprocess

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(os.path.abspath(oracle.__file__)), "emo_oracle.c")

MUTANTS = {
    "static_energy_dropped": ("*E_out = Ea + g->static_power * T;", "*E_out = Ea;"),
    "backward_sign": ("double lst_u = lft[u] - dur[u];", "double lst_u = lft[u] + dur[u];"),
    "backward_takes_max": ("if (j == g->succ_off[v] || lst_u < l) l = lst_u;",
                           "if (j == g->succ_off[v] || lst_u > l) l = lst_u;"),
    "critical_pred_min": ("C[k] > C[best]", "C[k] < C[best]"),
    "critical_pred_tie_last": ("g->pos[k] < g->pos[best]", "g->pos[k] > g->pos[best]"),
    "table_transposed": ("(size_t)p * g->F + l", "(size_t)l * g->P + p"),
    "sink_lft_is_own_eft": ("double l = T;", "double l = C[v];"),
    "feasibility_strict": ("int ok = T[c] <= target;", "int ok = T[c] < target;"),
    "tie_takes_last": ("En[c] < En[best]", "En[c] <= En[best]"),
    "depth_not_incremented": ("int dk = g->depth[g->pred[i]] + 1;", "int dk = g->depth[g->pred[i]];"),
    "makespan_last_node": ("if (C[v] > T) T = C[v];", "T = C[v];"),
    "energy_overwritten": ("Ea += en[v];", "Ea = en[v];"),
    "duration_not_added": ("C[v] = s + dur[v];", "C[v] = s;"),
    "start_from_last_pred": ("if (C[k] > s) s = C[k];", "s = C[k];"),
    "slack_uses_lft_only": ("slack[v] = l - C[v];", "slack[v] = l;"),
    "level_off_by_one": ("int l = lv[p];", "int l = lv[p] > 0 ? lv[p] - 1 : 0;"),
    "bad_level_ignored": ("if (l >= g->F) { bad = 1;", "if (l >= g->F) { bad = 0;"),
    "batch_slack_row_shifted": ("else if (g.pack[v] >= 0) row[g.pack[v]] = s;",
                                "else if (g.pack[v] >= 0) row[(g.pack[v] + 1) % P] = s;"),
}


def _build_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o",
                           str(so), str(path), "-lm"])
    return str(so)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(oracle_lib, tmp_path, name):
    old, new = MUTANTS[name]
    so = _build_mutant(tmp_path, name, old, new)
    prev = oracle.use_library(so)
    caught = []
    try:
        for pin in pins.ALL_PINS:
            try:
                pin()
            except (AssertionError, oracle.OracleError, IndexError, ValueError):
                caught.append(pin.__name__)
    finally:
        oracle.use_library(prev)
    assert caught, f"no pin caught mutant {name}"
