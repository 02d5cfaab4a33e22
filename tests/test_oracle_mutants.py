"""Planted mistakes in the oracle must be caught by its pins.

Each case copies the oracle's C source, applies one plausible mistake (a
dropped term, a flipped comparison, a wrong tie-break ...), compiles it to a
temporary library on the CPU, and runs the pin checks of test_oracle_pins
against it: at least one of them has to fail. Nothing here touches a GPU.
"""
import os
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
import workloads as W
from tests import test_oracle_pins as pins

MUTANTS = {
    "tl_drops_pred_comp": ("tl[u] + comp[u] + comm_cost", "tl[u] + comm_cost"),
    "bl_drops_own_comp": ("bl[v] = comp[v] + best;", "bl[v] = best;"),
    "comm_inverted": ("label[src[e]] == label[dst[e]] ? 0 : edge_cost[e]",
                      "label[src[e]] != label[dst[e]] ? 0 : edge_cost[e]"),
    "comm_ignores_label": ("label[src[e]] == label[dst[e]] ? 0 : edge_cost[e]", "edge_cost[e]"),
    "bl_uses_wrong_endpoint": ("int64_t cand = comm_cost(label, src, dst, edge_cost, e) + bl[s];",
                               "int64_t cand = comm_cost(label, src, dst, edge_cost, e) + bl[v];"),
    "makespan_from_tl_only": ("if (tl[v] + bl[v] > m)\n                m = tl[v] + bl[v];",
                              "if (tl[v] > m)\n                m = tl[v];"),
    "path_tiebreak_max_id": ("(next < 0 || s < next)", "(next < 0 || s > next)"),
    "path_start_any_source": ("if (indeg[v] == 0 && is_critical[v]) {",
                              "if (is_critical[v]) {"),
    "path_not_tight": ("if (through == makespan && (next < 0 || s < next))",
                       "if (through <= makespan && (next < 0 || s < next))"),
    "level_no_increment": ("if (level[u] + 1 > level[s])\n                    level[s] = level[u] + 1;",
                           "if (level[u] > level[s])\n                    level[s] = level[u];"),
    "level_min_not_max": ("if (level[u] + 1 > level[s])", "if (level[s] == 0)"),
    "order_unstable": ("order[cursor[level[v]]++] = v;",
                       "order[cursor[level[v]]++] = n_nodes - 1 - v;"),
    "label_sum_off_by_one": ("label_mem[label[v]] += mem[v];",
                             "label_mem[label[v] % (n_labels > 1 ? n_labels - 1 : 1)] += mem[v];"),
    "overflow_sign": ("label_mem[k] > cap ? label_mem[k] - cap : 0",
                      "label_mem[k] > cap ? cap - label_mem[k] : 0"),
    "overflow_guard_missing_cost": ("if (edge_cost[e] > INT64_MAX - total)\n            return ORC_E_OVERFLOW;",
                                    "if (0)\n            return ORC_E_OVERFLOW;"),
}


def _run_pins():
    """The pin checks, in an order that fails fast; raises on the first failure."""
    for path in pins.GOLDEN:
        pins.test_golden(path, oracle)
    for seed in range(40):
        pins.test_bruteforce_random(seed, oracle)
    pins.test_chain_closed_form(7, oracle)
    pins.test_fork_join_closed_form(oracle)
    for seed in range(5):
        pins.test_networkx_small_random(seed, oracle)
    pins.test_label_memory(0, oracle)
    pins.test_errors(oracle)
    pins.test_config_invariants(0, oracle)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    before, after = MUTANTS[name]
    src = open(oracle.SRC_PATH).read()
    assert src.count(before) == 1, f"mutation site for {name} not unique"
    mutated = src.replace(before, after)
    cfile = tmp_path / "mut.c"
    cfile.write_text(mutated)
    so = tmp_path / f"liboracle_{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-fPIC", "-shared",
                           "-I", os.path.dirname(oracle.SRC_PATH), "-o", str(so), str(cfile)])
    saved = oracle._lib
    oracle._lib = oracle.bind(str(so))
    try:
        with pytest.raises((AssertionError, oracle.OracleError)):
            _run_pins()
    finally:
        oracle._lib = saved


def test_unmutated_passes():
    oracle.build(force=False)
    _run_pins()
