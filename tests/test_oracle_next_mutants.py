"""Planted mistakes in the oracles of the rows after the core path must be
caught by their pins.

Each case takes one of oracle/memory_balance.py, clusters.py, span_work.py,
slicing.py, applies one plausible mistake to a copy of its source (a flipped
comparison, a dropped term, a wrong tie-break, a wrong reading of the paper),
loads the copy as a module of the oracle package, and runs the pins of
test_oracle_next against it: at least one of them has to fail. CPU only.
"""
import os
import types

import pytest

import oracle  # noqa: F401  (the package the mutated copies import from)
from tests import test_oracle_next as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    # Memory Heuristic II (Sec. 3.2.2, Eq. 6)
    "eq6_strict": ("memory_balance", "(share_res + share_nor) >= 1)",
                   "(share_res + share_nor) > 1)"),
    "reference_counted_as_normal": ("memory_balance",
                                    "is_res, is_nor = node_type == RESIDUAL, node_type == NORMAL",
                                    "is_res, is_nor = node_type == RESIDUAL, node_type != RESIDUAL"),
    "misplaced_inverted": ("memory_balance", "(label[refs] != label[ref_target[refs]])",
                           "(label[refs] == label[ref_target[refs]])"),
    "missing_kind_zero_share": ("memory_balance", "if RES > 0 else Fraction(1, K)",
                                "if RES > 0 else Fraction(0)"),
    # cluster criticality (Sec. 3.1.2)
    "criticality_counts_last_twice": ("clusters", "+ int(bl[last]) - int(comp[last]))",
                                      "+ int(bl[last]))"),
    "criticality_no_path_check": ("clusters",
                                  "if any((nodes[i], nodes[i + 1]) not in edges for i in range(len(nodes) - 1)):",
                                  "if False:"),
    "criticality_order_ascending": ("clusters", "key=lambda c: (-crit[c], c)",
                                    "key=lambda c: (crit[c], c)"),
    "criticality_members_by_id": ("clusters",
                                  "nodes = sorted(members[c], key=lambda v: (int(level[v]), v))",
                                  "nodes = sorted(members[c])"),
    # Eq. 2 span-work terms
    "span_lo_without_comp": ("span_work", "int(tl[p] + comp[p])", "int(tl[p])"),
    "span_hi_default_zero": ("span_work", "default=makespan)", "default=0)"),
    "span_exclusive_low": ("span_work", "(tl >= lo[r]) & (tl <= hi[r])",
                           "(tl > lo[r]) & (tl <= hi[r])"),
    "comm_counts_inside_edges": ("span_work",
                                 "out_e = in_c[src] & ~in_c[dst] & (label[dst] >= 0)",
                                 "out_e = in_c[src] & (label[dst] >= 0)"),
    "choice_tie_small_comm": ("span_work", "(cost[k], -int(comm[r, k]), k)",
                              "(cost[k], int(comm[r, k]), k)"),
    # graph slicing (Alg. 1)
    "primary_not_removed": ("slicing", "        alive[p] = False\n", "        alive[p] = alive[p]\n"),
    "walk_takes_smallest_priority": ("slicing", "(w[t], -t) > (w[best], -best)",
                                     "(w[t], -t) < (w[best], -best)"),
    "walk_tie_larger_id": ("slicing", "(w[t], -t) > (w[best], -best)",
                           "(w[t], t) > (w[best], best)"),
    "walk_start_smallest_priority": ("slicing",
                                     "sources = [(-w[v], v) for v in range(R) if indeg[v] == 0]",
                                     "sources = [(w[v], v) for v in range(R) if indeg[v] == 0]"),
    "walk_edges_stay": ("slicing", "                indeg[t] -= 1\n", "                indeg[t] -= 0\n"),
}

# the pins of each oracle, cheapest first; each raises on a wrong result
PINS = {
    "memory_balance": (
        [("memory_balance", "memory_balance")],
        lambda: ([pins.test_heuristic2_paper_example(), pins.test_heuristic2_invariants(),
                  pins.test_heuristic2_one_kind_missing()]
                 + [pins.test_heuristic2_sums_against_a_node_loop(s) for s in range(6)])),
    "clusters": (
        [("cluster_criticality", "cluster_criticality")],
        lambda: ([pins.test_cluster_criticality_hand_example(),
                  pins.test_cluster_criticality_special_cases()]
                 + [pins.test_cluster_criticality_against_path_enumeration(s) for s in range(40)])),
    "span_work": (
        [("span_work", "span_work")],
        lambda: ([pins.test_eq2_hand_example(), pins.test_eq2_invariants()]
                 + [pins.test_eq2_work_matches_fenwick_trees_through_a_mapping_loop(s)
                    for s in range(6)]
                 + [pins.test_eq2_comm_ignores_the_clusters_own_partitions()])),
    "slicing": (
        [("slice_primaries", "slice_primaries"), ("slice_all", "slice_all")],
        lambda: ([pins.test_slicing_chain_and_exhaustion(), pins.test_slicing_invariants(),
                  pins.test_secondary_clusters_invariants()]
                 + [pins.test_slicing_against_path_enumeration(s) for s in range(12)]
                 + [pins.test_secondary_clusters_against_path_enumeration(s)
                    for s in range(100)])),
}


def load_mutant(modname, before, after):
    path = os.path.join(ROOT, "oracle", modname + ".py")
    src = open(path).read()
    assert src.count(before) == 1, f"mutation site not unique in {modname}: {before!r}"
    m = types.ModuleType(f"oracle._mutant_{modname}")
    m.__package__ = "oracle"
    m.__file__ = path
    exec(compile(src.replace(before, after), path, "exec"), m.__dict__)
    return m


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_next_row_mutant_is_caught(name, monkeypatch):
    modname, before, after = MUTANTS[name]
    mutant = load_mutant(modname, before, after)
    names, run = PINS[modname]
    for pin_name, fn in names:
        monkeypatch.setattr(pins, pin_name, getattr(mutant, fn))
    with pytest.raises(Exception):
        run()


@pytest.mark.parametrize("modname", sorted(PINS))
def test_unmutated_copies_pass(modname, monkeypatch):
    """The same loading path without a mutation passes every pin, so a caught
    mutant is caught by its mistake, not by the loading."""
    mutant = load_mutant(modname, "from __future__ import annotations",
                         "from __future__ import annotations")
    names, run = PINS[modname]
    for pin_name, fn in names:
        monkeypatch.setattr(pins, pin_name, getattr(mutant, fn))
    run()
