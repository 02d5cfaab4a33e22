"""Pins for the CPU oracle, against things other than the oracle itself.

* hand-derived golden examples (tests/golden/*.json, each with its derivation);
* exhaustive path enumeration on tiny random DAGs (tests/bruteforce.py);
* closed forms (chain, fork/join);
* library routines for special cases (networkx topological generations and
  DAG longest path on the node-split graph);
* invariants on the synthetic configs (slack, tightness, duality,
  monotonicity in the placement, renumbering invariance).
"""
import functools
import glob
import json
import os

import networkx as nx
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import workloads as W
from tests.bruteforce import brute_force, hop_levels

GOLDEN = sorted(glob.glob(os.path.join(os.path.dirname(__file__), "golden", "*.json")))


@functools.lru_cache(maxsize=None)
def cfg(i):
    return W.make_config(i)


def comm_vec(g, label):
    return np.where(label[g.src] == label[g.dst], 0, g.edge_cost)


# ---------------------------------------------------------------- golden --

@pytest.mark.parametrize("path", GOLDEN, ids=[os.path.basename(p) for p in GOLDEN])
def test_golden(path, oracle_lib):
    d = json.load(open(path))
    x = d["expect"]
    n = d["n_nodes"]
    level, order, lptr, nl = oracle.levelize(n, d["src"], d["dst"])
    assert level.tolist() == x["level"]
    assert order.tolist() == x["order"]
    assert lptr.tolist() == x["level_ptr"]
    tl, bl, m = oracle.tb_levels(n, d["src"], d["dst"], d["comp"], d["edge_cost"], d["label"])
    assert tl.tolist() == x["tl"] and bl.tolist() == x["bl"] and m == x["makespan"]
    crit, path = oracle.critical_path(n, d["src"], d["dst"], d["comp"], d["edge_cost"],
                                      d["label"], tl, bl, m)
    assert crit.tolist() == x["is_critical"] and path.tolist() == x["path"]
    sums, over = oracle.label_memory(n, d["mem"], d["label"], d["n_labels"], d["capacity"])
    assert sums.tolist() == x["label_mem"] and over.tolist() == x["overflow"]


def test_walk_through_noncritical_node(oracle_lib):
    """The path rule steps along tight edges from whatever node it reached,
    critical or not (Table 2, CP; the walk of Sec. 3.1.1). Hand-derived:
    edges 0->1, 1->2, 1->3, every comp 1, no cost. Consistent levels are
    tl = [0, 1, 2, 2], bl = [3, 2, 1, 1], M = 3; raising tl(1) by one and
    lowering bl(3) by one leaves node 1 off the critical set (w = 4) but keeps
    0->1 (0 + 1 + 2 = 3) and 1->3 (2 + 1 + 0 = 3) tight, while 1->2 gives 4."""
    src, dst = [0, 1, 1], [1, 2, 3]
    comp, cost, lab = [1, 1, 1, 1], [0, 0, 0], [0, 0, 0, 0]
    tl, bl, m = oracle.tb_levels(4, src, dst, comp, cost, lab)
    assert tl.tolist() == [0, 1, 2, 2] and bl.tolist() == [3, 2, 1, 1] and m == 3
    tl[1] += 1
    bl[3] -= 1
    crit, path = oracle.critical_path(4, src, dst, comp, cost, lab, tl, bl, m)
    assert crit.tolist() == [1, 0, 1, 0]
    assert path.tolist() == [0, 1, 3]


# ----------------------------------------------------------- brute force --

def _check_against_brute_force(g):
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    crit, path = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost,
                                      g.placement, tl, bl, m)
    btl, bbl, bm, bcrit, bpath = brute_force(g.n_nodes, g.src, g.dst, g.comp,
                                             g.edge_cost, g.placement)
    assert tl.tolist() == btl
    assert bl.tolist() == bbl
    assert m == bm
    assert crit.tolist() == bcrit
    assert path.tolist() == bpath
    level, order, lptr, nl = oracle.levelize(g.n_nodes, g.src, g.dst)
    assert level.tolist() == hop_levels(g.n_nodes, g.src, g.dst)
    # order: ids sorted by (level, id); level_ptr: level boundaries
    assert order.tolist() == sorted(range(g.n_nodes), key=lambda v: (level[v], v))
    assert lptr.tolist() == [0] + np.cumsum(np.bincount(level, minlength=nl)).tolist()


@pytest.mark.parametrize("seed", range(60))
def test_bruteforce_random(seed, oracle_lib):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 11))
    g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.1, 0.6)),
                     max_weight=int(rng.integers(0, 4)), n_labels=int(rng.integers(1, 4)))
    _check_against_brute_force(g)


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(n=st.integers(0, 9), seed=st.integers(0, 2**31), p=st.floats(0.0, 0.8),
       w=st.integers(0, 3), k=st.integers(1, 4))
def test_bruteforce_hypothesis(n, seed, p, w, k):
    oracle.build(force=False)
    g = W.random_dag(np.random.default_rng(seed), n, p_edge=p, max_weight=w, n_labels=k)
    _check_against_brute_force(g)


# ----------------------------------------------------------- closed forms --

@pytest.mark.parametrize("n", [1, 2, 7, 300])
def test_chain_closed_form(n, oracle_lib):
    g = W.chain_graph(np.random.default_rng(n), n)
    c = comm_vec(g, g.placement)
    tl, bl, m = oracle.tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    # tl_i = sum_{j<i} (comp_j + c_j); bl_i = sum_{j>=i} comp_j + sum_{j>=i} c_j
    exp_tl = np.concatenate([[0], np.cumsum(g.comp[:-1] + c)]) if n else np.zeros(0)
    exp_bl = np.cumsum((g.comp + np.concatenate([c, [0]]))[::-1])[::-1]
    assert tl.tolist() == exp_tl.tolist()
    assert bl.tolist() == exp_bl.tolist()
    assert m == int(g.comp.sum() + c.sum())
    crit, path = oracle.critical_path(n, g.src, g.dst, g.comp, g.edge_cost, g.placement, tl, bl, m)
    assert crit.all() and path.tolist() == list(range(n))
    level, order, lptr, nl = oracle.levelize(n, g.src, g.dst)
    assert level.tolist() == list(range(n)) and nl == n


def test_fork_join_closed_form(oracle_lib):
    # source 0 -> k middle nodes -> sink k+1; the heaviest middle branch wins
    rng = np.random.default_rng(7)
    k = 50
    n = k + 2
    src = np.r_[np.zeros(k, np.int32), np.arange(1, k + 1, dtype=np.int32)]
    dst = np.r_[np.arange(1, k + 1, dtype=np.int32), np.full(k, k + 1, np.int32)]
    comp = rng.integers(0, 100, n)
    cost = rng.integers(0, 100, 2 * k)
    label = rng.integers(0, 3, n).astype(np.int32)
    c = np.where(label[src] == label[dst], 0, cost)
    branch = comp[1:k + 1] + c[:k] + c[k:]
    tl, bl, m = oracle.tb_levels(n, src, dst, comp, cost, label)
    assert m == comp[0] + branch.max() + comp[k + 1]
    assert tl[k + 1] == comp[0] + branch.max()
    crit, path = oracle.critical_path(n, src, dst, comp, cost, label, tl, bl, m)
    winners = np.nonzero(branch == branch.max())[0] + 1
    assert path.tolist() == [0, int(winners.min()), k + 1]
    assert sorted(np.nonzero(crit)[0].tolist()) == [0] + winners.tolist() + [k + 1]


# ------------------------------------------------------ library routines --

def _node_split_longest(g, label):
    """Longest path length via networkx on the node-split graph: node v becomes
    v_in -> v_out with weight comp(v); edge (u, v) becomes u_out -> v_in with
    its communication cost (the heaviest of parallel edges)."""
    G = nx.DiGraph()
    for v in range(g.n_nodes):
        G.add_edge(("i", v), ("o", v), weight=int(g.comp[v]))
    c = comm_vec(g, label)
    for e in range(g.n_edges):
        a, b = ("o", int(g.src[e])), ("i", int(g.dst[e]))
        w = int(c[e])
        if G.has_edge(a, b):
            w = max(w, G[a][b]["weight"])
        G.add_edge(a, b, weight=w)
    return nx.dag_longest_path_length(G, weight="weight") if g.n_nodes else 0


@pytest.mark.parametrize("i", [0, 1])
def test_networkx_levels(i, oracle_lib):
    g = cfg(i)
    G = nx.DiGraph()
    G.add_nodes_from(range(g.n_nodes))
    G.add_edges_from(zip(g.src.tolist(), g.dst.tolist()))
    level, order, lptr, nl = oracle.levelize(g.n_nodes, g.src, g.dst)
    gens = list(nx.topological_generations(G))
    assert nl == len(gens)
    for k, gen in enumerate(gens):
        assert sorted(gen) == order[lptr[k]:lptr[k + 1]].tolist()


@pytest.mark.parametrize("i", [0, 1])
@pytest.mark.parametrize("mode", ["same", "distinct"])
def test_networkx_longest_path(i, mode, oracle_lib):
    g = cfg(i)
    label = (np.zeros(g.n_nodes, np.int32) if mode == "same"
             else np.arange(g.n_nodes, dtype=np.int32))
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, label)
    assert m == _node_split_longest(g, label)


@pytest.mark.parametrize("seed", range(20))
def test_networkx_small_random(seed, oracle_lib):
    rng = np.random.default_rng(seed)
    g = W.random_dag(rng, int(rng.integers(1, 40)), p_edge=0.15, max_weight=50, n_labels=3)
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    assert m == _node_split_longest(g, g.placement)


def test_unit_weights_give_levels(oracle_lib):
    # comp = 1, cost = 0  =>  tl(v) is the hop level of v
    g = cfg(1)
    level, *_ = oracle.levelize(g.n_nodes, g.src, g.dst)
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, np.ones(g.n_nodes, np.int64),
                                 np.zeros(g.n_edges, np.int64), g.placement)
    assert (tl == level).all()


# -------------------------------------------------------------- invariants --

@pytest.mark.parametrize("i", [0, 1, 2, 3])
def test_config_invariants(i, oracle_lib):
    g = cfg(i)
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    crit, path = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost,
                                      g.placement, tl, bl, m)
    c = comm_vec(g, g.placement)
    w = tl + bl
    assert (w <= m).all()
    assert ((w == m) == crit.astype(bool)).all()
    # slack >= 0 on every edge, both directions
    through = tl[g.src] + g.comp[g.src] + c
    assert (through <= tl[g.dst]).all()
    assert (g.comp[g.src] + c + bl[g.dst] <= bl[g.src]).all()
    # every non-source has a tight in-edge; every non-sink a tight out-edge
    indeg = np.bincount(g.dst, minlength=g.n_nodes)
    outdeg = np.bincount(g.src, minlength=g.n_nodes)
    best_in = np.zeros(g.n_nodes, np.int64)
    np.maximum.at(best_in, g.dst, through)
    assert (best_in[indeg > 0] == tl[indeg > 0]).all() and (tl[indeg == 0] == 0).all()
    best_out = np.zeros(g.n_nodes, np.int64)
    np.maximum.at(best_out, g.src, c + bl[g.dst])
    assert (g.comp + best_out == bl).all() and (bl[outdeg == 0] == g.comp[outdeg == 0]).all()
    # M is reached at a source
    assert m == bl[indeg == 0].max()
    # the path is a chain of tight edges from a source to a sink of length M
    assert indeg[path[0]] == 0 and outdeg[path[-1]] == 0 and crit[path].all()
    edge_map = {}
    for e in range(g.n_edges):
        edge_map.setdefault((int(g.src[e]), int(g.dst[e])), []).append(int(c[e]))
    length = int(g.comp[path].sum()) + sum(max(edge_map[(int(a), int(b))])
                                           for a, b in zip(path[:-1], path[1:]))
    assert length == m


@pytest.mark.parametrize("i", [0, 1, 2])
def test_reverse_duality(i, oracle_lib):
    # bl in G equals tl in the reversed graph plus comp
    g = cfg(i)
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    rtl, rbl, rm = oracle.tb_levels(g.n_nodes, g.dst, g.src, g.comp, g.edge_cost, g.placement)
    assert (bl == rtl + g.comp).all() and (tl == rbl - g.comp).all() and m == rm


@pytest.mark.parametrize("i", [0, 1, 2])
def test_placement_monotone(i, oracle_lib):
    g = cfg(i)
    same = np.zeros(g.n_nodes, np.int32)
    dist = np.arange(g.n_nodes, dtype=np.int32)
    ms = [oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab)[2]
          for lab in (same, g.placement, dist)]
    assert ms[0] <= ms[1] <= ms[2]


@pytest.mark.parametrize("i", [0, 1])
def test_renumber_and_shuffle_invariance(i, oracle_lib):
    g = cfg(i)
    rng = np.random.default_rng(99)
    perm = rng.permutation(g.n_nodes)
    ep = rng.permutation(g.n_edges)
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    comp2 = np.empty_like(g.comp); comp2[perm] = g.comp
    lab2 = np.empty_like(g.placement); lab2[perm] = g.placement
    tl2, bl2, m2 = oracle.tb_levels(g.n_nodes, perm[g.src][ep], perm[g.dst][ep], comp2,
                                    g.edge_cost[ep], lab2)
    assert m2 == m and (tl2[perm] == tl).all() and (bl2[perm] == bl).all()
    level, *_ = oracle.levelize(g.n_nodes, g.src, g.dst)
    level2, *_ = oracle.levelize(g.n_nodes, perm[g.src][ep], perm[g.dst][ep])
    assert (level2[perm] == level).all()


# ------------------------------------------------------------ label memory --

@pytest.mark.parametrize("i", [0, 2])
def test_label_memory(i, oracle_lib):
    g = cfg(i)
    sums, over = oracle.label_memory(g.n_nodes, g.mem, g.placement, g.n_labels, g.capacity)
    exp = np.zeros(g.n_labels, np.int64)
    np.add.at(exp, g.placement, g.mem)
    assert (sums == exp).all() and int(sums.sum()) == int(g.mem.sum())
    assert (over == np.maximum(0, exp - g.capacity)).all()
    one, _ = oracle.label_memory(g.n_nodes, g.mem, np.zeros(g.n_nodes, np.int32), 1)
    assert one.tolist() == [int(g.mem.sum())]


# ------------------------------------------------------------- error paths --

def test_errors(oracle_lib):
    with pytest.raises(oracle.OracleError) as e:
        oracle.levelize(3, [0, 1, 2], [1, 2, 0])
    assert e.value.status == oracle.E_CYCLE
    with pytest.raises(oracle.OracleError) as e:
        oracle.tb_levels(2, [1], [1], [1, 1], [1], [0, 0])
    assert e.value.status == oracle.E_CYCLE
    with pytest.raises(oracle.OracleError) as e:
        oracle.levelize(2, [0], [2])
    assert e.value.status == oracle.E_INVAL
    with pytest.raises(oracle.OracleError) as e:
        oracle.label_memory(2, [1, 1], [0, 2], 2)
    assert e.value.status == oracle.E_INVAL
    assert oracle.validate(2, [0], [1], [1, -1], [0], [0, 0]) == oracle.E_INVAL
    assert oracle.validate(2, [0], [1], [1, 1], [-5], [0, 0]) == oracle.E_INVAL
    big = np.iinfo(np.int64).max
    assert oracle.validate(2, [0], [1], [big, 1], [0], [0, 0]) == oracle.E_OVERFLOW
    assert oracle.validate(2, [0], [1], [big - 1, 0], [1], [0, 0]) == oracle.OK
    assert oracle.validate(2, [0], [1], [big - 5, 0], [10], [0, 0]) == oracle.E_OVERFLOW
    assert oracle.validate(2, [0], [1], [0, 0], [0], [big, 1]) == oracle.E_OVERFLOW
    assert oracle.validate(0, [], [], [], [], []) == oracle.OK


def test_empty_graph(oracle_lib):
    level, order, lptr, nl = oracle.levelize(0, [], [])
    assert nl == 0 and lptr.tolist() == [0]
    tl, bl, m = oracle.tb_levels(0, [], [], [], [], [])
    assert m == 0
    crit, path = oracle.critical_path(0, [], [], [], [], [], tl, bl, m)
    assert path.size == 0
