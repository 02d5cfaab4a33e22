"""Pins of the oracle functions for the rows after the core path: Memory
Heuristic II evaluation (Sec. 3.2.2). CPU only.

The paper's own worked example of Heuristic II (a fixture under tests/golden/)
pins the Eq. 6 predicate and the memory kinds; a per-node loop written here
pins the vectorised sums; invariants pin the rest.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.memory_balance import memory_balance
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "next")


def test_heuristic2_paper_example():
    d = json.load(open(os.path.join(GOLDEN, "heuristic2_paper_example.json")))
    for name, lab in d["placements"].items():
        r = memory_balance(d["n_nodes"], d["mem"], d["node_type"], d["ref_target"], lab,
                           d["n_labels"])
        exp = d["expect"][name]
        assert r["res_mem"].tolist() == exp["res_mem"], name
        assert r["nor_mem"].tolist() == exp["nor_mem"], name
        assert r["balanced"].tolist() == exp["balanced"], name
        assert r["ref_misplaced"] == exp["ref_misplaced"], name


def _per_node(n, mem, kind, target, label, K):
    res, nor = [0] * K, [0] * K
    mis = 0
    for v in range(n):
        if kind[v] == 1:
            res[label[v]] += int(mem[v])
        elif kind[v] == 0:
            nor[label[v]] += int(mem[v])
        elif target[v] >= 0 and label[target[v]] != label[v]:
            mis += 1
    return res, nor, mis


@pytest.mark.parametrize("seed", range(6))
def test_heuristic2_sums_against_a_node_loop(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 300))
    K = int(rng.integers(1, 9))
    mem = rng.integers(0, 1000, n)
    kind = rng.integers(0, 3, n)
    res_nodes = np.nonzero(kind == 1)[0]
    target = np.full(n, -1)
    for v in np.nonzero(kind == 2)[0]:
        if res_nodes.size and rng.random() < 0.9:
            target[v] = res_nodes[rng.integers(res_nodes.size)]
    label = rng.integers(0, K, n)
    r = memory_balance(n, mem, kind, target, label, K)
    res, nor, mis = _per_node(n, mem, kind, target, label, K)
    assert r["res_mem"].tolist() == res and r["nor_mem"].tolist() == nor
    assert r["ref_misplaced"] == mis
    # the K shares of each kind sum to one, so their mean is 1 / K and some
    # partition is at or above it: Eq. 6 holds somewhere
    assert r["balanced"].any()


def test_heuristic2_invariants():
    rng = np.random.default_rng(7)
    n, K = 500, 5
    mem = rng.integers(1, 10 ** 6, n)
    kind = rng.integers(0, 2, n)
    label = rng.integers(0, K, n)
    tgt = np.full(n, -1)
    r = memory_balance(n, mem, kind, tgt, label, K)
    assert r["res_mem"].sum() == mem[kind == 1].sum()
    assert r["nor_mem"].sum() == mem[kind == 0].sum()
    # relabelling the partitions permutes the outputs
    perm = rng.permutation(K)
    r2 = memory_balance(n, mem, kind, tgt, perm[label], K)
    assert (r2["res_mem"][perm] == r["res_mem"]).all()
    assert (r2["balanced"][perm] == r["balanced"]).all()
    # one partition holds everything: balanced
    assert memory_balance(n, mem, kind, tgt, np.zeros(n, int), 1)["balanced"].tolist() == [1]
    # identical per-label content (node i on label i mod K, kind (i div K)
    # mod 2, equal memory): every partition exactly at its share
    i = np.arange(n)
    r3 = memory_balance(n, np.full(n, 7), (i // K) % 2, tgt, i % K, K)
    assert r3["balanced"].all()


def test_heuristic2_one_kind_missing():
    # no residual memory: the residual share counts as 1/K on every partition,
    # so Eq. 6 reads K/2 (1/K + share) >= 1, i.e. share >= 1/K
    n, K = 6, 3
    mem = [30, 30, 20, 10, 5, 5]
    kind = [0] * 6
    label = [0, 0, 1, 1, 2, 2]
    r = memory_balance(n, mem, kind, [-1] * 6, label, K)
    shares = [Fraction(60, 100), Fraction(30, 100), Fraction(10, 100)]
    assert r["balanced"].tolist() == [int(s >= Fraction(1, K)) for s in shares] == [1, 0, 0]
    # no memory at all: balanced everywhere
    r0 = memory_balance(n, [0] * 6, kind, [-1] * 6, label, K)
    assert r0["balanced"].tolist() == [1, 1, 1]


def test_heuristic2_rejects_bad_input():
    with pytest.raises(ValueError):
        memory_balance(2, [1, 1], [0, 0], [-1, -1], [0, 2], 2)
    with pytest.raises(ValueError):
        memory_balance(2, [1, 1], [0, 3], [-1, -1], [0, 1], 2)
    with pytest.raises(ValueError):
        memory_balance(2, [1, 1], [0, 2], [-1, 5], [0, 1], 2)


def test_transformer_kinds_are_variables_and_their_updates():
    g = W.make_config(2)
    kind, tgt = W.node_kinds(g)
    refs = np.nonzero(kind == 2)[0]
    assert refs.size > 0 and (kind[tgt[refs]] == 1).all()
    # an optimiser op is a direct successor of the variable it updates
    pairs = set(zip(g.src.tolist(), g.dst.tolist()))
    assert all((int(tgt[v]), int(v)) in pairs for v in refs[:500])


# ---------------------------------------------------------------------------
# Graph slicing primaries (Alg. 1)
# ---------------------------------------------------------------------------
from oracle.slicing import slice_primaries  # noqa: E402


def _brute_rounds(n, src, dst, comp, cost, K):
    """Every round by enumerating all source-to-sink paths of the remaining
    graph: the longest (all edges pay), ties to the smallest node sequence."""
    alive = set(range(n))
    out = []
    for _ in range(K):
        succ = {v: [] for v in alive}
        indeg = {v: 0 for v in alive}
        for e, (a, b) in enumerate(zip(src, dst)):
            if a in alive and b in alive:
                succ[a].append((b, cost[e]))
                indeg[b] += 1
        best = None

        def walk(v, seq, length):
            nonlocal best
            length += comp[v]
            seq = seq + [v]
            if not succ[v]:
                key = (-length, seq)
                if best is None or key < best:
                    best = key
                return
            for b, c in succ[v]:
                walk(b, seq, length + c)

        for v in sorted(alive):
            if indeg[v] == 0:
                walk(v, [], 0)
        if best is None:
            out.append(([], 0))
            continue
        out.append((best[1], -best[0]))
        alive -= set(best[1])
    return out


@pytest.mark.parametrize("seed", range(12))
def test_slicing_against_path_enumeration(seed):
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(1, 11))
    g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.1, 0.6)),
                     max_weight=int(rng.integers(0, 4)), n_labels=1)
    K = int(rng.integers(1, n + 2))
    primary, paths, ms = slice_primaries(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    brute = _brute_rounds(g.n_nodes, g.src.tolist(), g.dst.tolist(), g.comp.tolist(),
                          g.edge_cost.tolist(), K)
    for j, (seq, length) in enumerate(brute):
        assert paths[j].tolist() == seq, (j, paths[j], seq)
        assert ms[j] == length
        assert all(primary[v] == j for v in seq)


def test_slicing_invariants():
    g = W.make_config(0)
    K = 8
    primary, paths, ms = slice_primaries(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    edges = set(zip(g.src.tolist(), g.dst.tolist()))
    seen = set()
    for j, p in enumerate(paths):
        assert len(p) > 0 and not (set(p.tolist()) & seen)   # disjoint clusters
        seen |= set(p.tolist())
        assert all((int(a), int(b)) in edges for a, b in zip(p[:-1], p[1:]))
        # the path's own length (all edges pay; of parallel edges the
        # costliest) is the round's makespan
        cost = {}
        for x, y, c in zip(g.src.tolist(), g.dst.tolist(), g.edge_cost.tolist()):
            cost[(x, y)] = max(cost.get((x, y), 0), c)
        length = int(g.comp[p].sum()) + sum(cost[(int(a), int(b))] for a, b in zip(p[:-1], p[1:]))
        assert length == ms[j]
    assert (np.diff(ms) <= 0).all()   # removing nodes never lengthens the longest path
    assert (primary >= 0).sum() == len(seen)


from oracle.slicing import slice_all  # noqa: E402


def _brute_secondaries(n, src, dst, comp, cost, alive):
    """The secondary clusters of the remaining graph `alive` by enumeration:
    w(v) is the longest source-to-sink path through v (all edges pay); then,
    repeatedly, of all maximal paths (from a node without a remaining
    predecessor to one without a remaining successor) the one whose sequence
    of keys (w(v), -v) is lexicographically largest leaves the graph."""
    alive = set(alive)

    def adjacency(nodes):
        succ = {v: [] for v in nodes}
        indeg = {v: 0 for v in nodes}
        for e, (a, b) in enumerate(zip(src, dst)):
            if a in nodes and b in nodes:
                succ[a].append((b, cost[e]))
                indeg[b] += 1
        return succ, indeg

    succ, indeg = adjacency(alive)
    w = {v: -1 for v in alive}

    def through(v, seq, length):
        length += comp[v]
        seq = seq + [v]
        if not succ[v]:
            for x in seq:
                w[x] = max(w[x], length)
            return
        for b, c in succ[v]:
            through(b, seq, length + c)

    for v in alive:
        if indeg[v] == 0:
            through(v, [], 0)
    out = []
    while alive:
        succ, indeg = adjacency(alive)
        best = None

        def walk(v, seq):
            nonlocal best
            seq = seq + [v]
            if not succ[v]:
                key = [(w[x], -x) for x in seq]
                if best is None or key > best[0]:
                    best = (key, seq)
                return
            for b, _ in succ[v]:
                walk(b, seq)

        for v in alive:
            if indeg[v] == 0:
                walk(v, [])
        out.append(best[1])
        alive -= set(best[1])
    return out


@pytest.mark.parametrize("seed", range(100))
def test_secondary_clusters_against_path_enumeration(seed):
    rng = np.random.default_rng(700 + seed)
    n = int(rng.integers(1, 11))
    g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.2, 0.7)),
                     max_weight=int(rng.integers(0, 9)), n_labels=1)
    K = int(rng.integers(0, 4))
    cluster, paths = slice_all(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    primary, _, _ = slice_primaries(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    brute = _brute_secondaries(n, g.src.tolist(), g.dst.tolist(), g.comp.tolist(),
                               g.edge_cost.tolist(), [v for v in range(n) if primary[v] < 0])
    assert [p.tolist() for p in paths[K:]] == brute
    for j, p in enumerate(paths):
        assert (cluster[p] == j).all()
    assert (cluster >= 0).all() and sum(len(p) for p in paths) == n


def test_secondary_clusters_invariants():
    """On the tiny layered DAG after 8 primaries: the clusters partition the
    nodes; each secondary is a path of the graph; when it was taken its start
    had no remaining predecessor and its end no remaining successor."""
    g = W.make_config(0)
    K = 8
    cluster, paths = slice_all(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    assert (cluster >= 0).all() and sum(len(p) for p in paths) == g.n_nodes
    edges = set(zip(g.src.tolist(), g.dst.tolist()))
    gone = np.zeros(g.n_nodes, bool)
    for p in paths[:K]:
        gone[p] = True
    for p in paths[K:]:
        assert all((int(a), int(b)) in edges for a, b in zip(p[:-1], p[1:]))
        live = ~gone[g.src] & ~gone[g.dst]
        assert not (live & (g.dst == p[0])).any()       # start: no remaining predecessor
        assert not (live & (g.src == p[-1])).any()      # end: a dead end
        gone[p] = True
    assert len(paths) > K + 1


def test_slicing_chain_and_exhaustion():
    rng = np.random.default_rng(9)
    g = W.chain_graph(rng, 12)
    primary, paths, ms = slice_primaries(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, 3)
    # a chain is one path: its length is the sum of all weights, then nothing remains
    assert sorted(paths[0].tolist()) == list(range(12))
    assert ms[0] == int(g.comp.sum() + g.edge_cost.sum())
    assert paths[1].size == 0 and paths[2].size == 0 and ms[1] == ms[2] == 0
    assert (primary == 0).all()


# ---------------------------------------------------------------------------
# Cluster criticality (Sec. 3.1.2)
# ---------------------------------------------------------------------------
from oracle.clusters import cluster_criticality  # noqa: E402


def _brute_criticality(n, src, dst, comp, cost, cluster, C):
    """Enumerate every source-to-sink path; an edge inside one cluster is free.
    Each cluster takes the longest path on which all of its nodes appear as
    one contiguous run (-1 when no path does)."""
    succ = [[] for _ in range(n)]
    indeg = [0] * n
    for a, b, c in zip(src, dst, cost):
        succ[a].append((b, 0 if cluster[a] == cluster[b] else c))
        indeg[b] += 1
    size = [0] * C
    for v in range(n):
        size[cluster[v]] += 1
    crit = [-1] * C

    def runs(path):
        # clusters whose every node lies in one contiguous run of the path
        out, i = set(), 0
        while i < len(path):
            j = i
            while j + 1 < len(path) and cluster[path[j + 1]] == cluster[path[i]]:
                j += 1
            if j - i + 1 == size[cluster[path[i]]]:
                out.add(cluster[path[i]])
            i = j + 1
        return out

    def walk(v, path, length):
        length += comp[v]
        path = path + [v]
        if not succ[v]:
            for c in runs(path):
                crit[c] = max(crit[c], length)
            return
        for b, c in succ[v]:
            walk(b, path, length + c)

    for v in range(n):
        if indeg[v] == 0:
            walk(v, [], 0)
    return crit


@pytest.mark.parametrize("seed", range(40))
def test_cluster_criticality_against_path_enumeration(seed):
    rng = np.random.default_rng(500 + seed)
    n = int(rng.integers(1, 13))
    g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.1, 0.6)),
                     max_weight=int(rng.integers(0, 5)), n_labels=1)
    cl, C = W.path_clusters(rng, g)
    crit, order = cluster_criticality(n, g.src, g.dst, g.comp, g.edge_cost, cl, C)
    brute = _brute_criticality(n, g.src.tolist(), g.dst.tolist(), g.comp.tolist(),
                               g.edge_cost.tolist(), cl.tolist(), C)
    assert crit.tolist() == brute
    assert order.tolist() == sorted(range(C), key=lambda c: (-brute[c], c))


def test_cluster_criticality_hand_example():
    d = json.load(open(os.path.join(GOLDEN, "criticality_whole_cluster.json")))
    crit, order = cluster_criticality(d["n_nodes"], d["src"], d["dst"], d["comp"],
                                      d["edge_cost"], d["cluster"], d["n_clusters"])
    assert crit.tolist() == d["expect"]["criticality"]
    assert order.tolist() == d["expect"]["order"]
    # the brute force agrees, and the largest w over the cluster would not
    assert _brute_criticality(d["n_nodes"], d["src"], d["dst"], d["comp"], d["edge_cost"],
                              d["cluster"], d["n_clusters"]) == d["expect"]["criticality"]


def test_cluster_criticality_special_cases():
    rng = np.random.default_rng(11)
    g = W.chain_graph(rng, 10)
    # one cluster holding a whole chain: all communication is internal, so the
    # criticality is the sum of the computation weights
    crit, order = cluster_criticality(10, g.src, g.dst, g.comp, g.edge_cost, np.zeros(10, int), 1)
    assert crit.tolist() == [int(g.comp.sum())]
    # every node its own cluster: every node of a chain lies on the one path,
    # whose length counts every edge
    crit, _ = cluster_criticality(10, g.src, g.dst, g.comp, g.edge_cost, np.arange(10), 10)
    assert (crit == int(g.comp.sum() + g.edge_cost.sum())).all()
    # two isolated nodes, one empty cluster: order by criticality, empty last
    crit, order = cluster_criticality(2, [], [], [5, 9], [], [2, 0], 3)
    assert crit.tolist() == [9, -1, 5] and order.tolist() == [0, 2, 1]
    # ties keep ascending ids
    crit, order = cluster_criticality(3, [], [], [4, 4, 4], [], [2, 1, 0], 3)
    assert order.tolist() == [0, 1, 2]
    with pytest.raises(ValueError):
        cluster_criticality(2, [], [], [1, 1], [], [0, 2], 2)


def test_cluster_criticality_of_slicing_clusters():
    """The primary clusters of slicing (each a path): a cluster is at least as
    critical as its own path with the path's edges now free (the sum of its
    computation weights), and no cluster exceeds the makespan of the whole
    graph, since making edges free never lengthens a path."""
    g = W.make_config(0)
    K = 8
    primary, paths, ms = slice_primaries(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    cl = np.where(primary >= 0, primary, K + np.arange(g.n_nodes))
    C = K + g.n_nodes
    crit, order = cluster_criticality(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, cl, C)
    assert crit.max() <= ms[0]
    assert all(crit[j] >= int(g.comp[paths[j]].sum()) for j in range(K))


# ---------------------------------------------------------------------------
# Eq. 2 span-work terms (Sec. 3.1.2)
# ---------------------------------------------------------------------------
from oracle.span_work import span_work  # noqa: E402
from oracle import tb_levels  # noqa: E402


def test_eq2_hand_example():
    d = json.load(open(os.path.join(GOLDEN, "eq2_hand_example.json")))
    n = d["n_nodes"]
    # the fixture's tl is the top level with every edge paying
    tl, _, m = tb_levels(n, d["src"], d["dst"], d["comp"], d["edge_cost"], list(range(n)))
    assert tl.tolist() == d["tl"] and m == 17
    r = span_work(n, d["src"], d["dst"], d["comp"], d["edge_cost"], d["label"], d["K"],
                  d["cluster"], d["n_clusters"], d["tl"])
    for key, exp in d["expect"].items():
        assert r[key].tolist() == exp, key


class Fenwick:
    """The paper's range-sum structure over per-level weights (binary indexed
    tree, 1-based), written here as an independent check of the work sums."""

    def __init__(self, n):
        self.t = [0] * (n + 1)

    def add(self, i, w):
        i += 1
        while i < len(self.t):
            self.t[i] += w
            i += i & -i

    def prefix(self, i):        # sum of positions [0, i)
        s = 0
        while i > 0:
            s += self.t[i]
            i -= i & -i
        return s


def _fenwick_work(levels, tl, comp, label, K, lo, hi):
    import bisect
    trees = [Fenwick(len(levels)) for _ in range(K)]
    for v in range(len(tl)):
        if label[v] >= 0:
            trees[label[v]].add(levels.index(tl[v]), int(comp[v]))
    out = []
    for a, b in zip(lo, hi):
        i, j = bisect.bisect_left(levels, a), bisect.bisect_right(levels, b)
        out.append([trees[k].prefix(j) - trees[k].prefix(i) if a <= b else 0 for k in range(K)])
    return trees, out


@pytest.mark.parametrize("seed", range(6))
def test_eq2_work_matches_fenwick_trees_through_a_mapping_loop(seed):
    """Level-aware load balancing as the paper runs it: per-partition Fenwick
    trees over the distinct top levels, one cluster merged at a time into its
    Eq. 2 choice (the trees updated with its nodes). After every merge the
    oracle, re-run on the new placement, gives the trees' span sums."""
    rng = np.random.default_rng(700 + seed)
    n = int(rng.integers(20, 80))
    g = W.random_dag(rng, n, p_edge=0.08, max_weight=9, n_labels=1)
    K = int(rng.integers(2, 5))
    tl, _, _ = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))
    label = np.where(rng.random(n) < 0.4, rng.integers(0, K, n), -1)
    C = int(rng.integers(1, 12))
    cluster = np.where(label < 0, rng.integers(-1, C, n), -1)
    levels = sorted(set(tl.tolist()))
    for step in range(C):
        r = span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C, tl)
        _, fw = _fenwick_work(levels, tl.tolist(), g.comp, label, K, r["span_lo"], r["span_hi"])
        assert r["work"].tolist() == fw, step
        c = step
        if r["choice"][c] >= 0:
            label = np.where(cluster == c, r["choice"][c], label)
            cluster = np.where(cluster == c, -1, cluster)


def test_eq2_invariants():
    rng = np.random.default_rng(17)
    g = W.make_config(0)
    n = g.n_nodes
    K = 4
    tl, _, m = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))
    label = np.where(rng.random(n) < 0.5, rng.integers(0, K, n), -1)
    C = 300
    cluster = np.where(label < 0, rng.integers(-1, C, n), -1)
    rows = list(range(0, C, 7))
    r = span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C, tl, clusters=rows)
    total = np.array([g.comp[label == k].sum() for k in range(K)])
    assert (r["work"] <= total).all() and (r["span_lo"] <= m).all()
    # a cluster spanning the whole run sees all mapped work
    whole = (r["span_lo"] == 0) & (r["span_hi"] == m)
    assert (r["work"][whole] == total).all()
    # renaming the partitions permutes the columns
    perm = rng.permutation(K)
    r2 = span_work(n, g.src, g.dst, g.comp, g.edge_cost, np.where(label >= 0, perm[label], -1), K,
                   cluster, C, tl, clusters=rows)
    assert (r2["work"][:, perm] == r["work"]).all() and (r2["comm"][:, perm] == r["comm"]).all()
    # the choice minimises Eq. 2
    tot = r["comm"].sum(axis=1, keepdims=True)
    cost = r["work"] + tot - r["comm"]
    ok = r["choice"] >= 0
    assert (cost[ok, r["choice"][ok]] == cost[ok].min(axis=1)).all()
    # a single partition takes every cluster that has nodes
    r1 = span_work(n, g.src, g.dst, g.comp, g.edge_cost, np.where(label >= 0, 0, -1), 1,
                   cluster, C, tl, clusters=rows)
    assert set(r1["choice"].tolist()) <= {0, -1}


def test_eq2_comm_ignores_the_clusters_own_partitions():
    """Members of a cluster may already sit on a partition (a placed cluster
    re-evaluated). An edge inside the cluster carries no communication, so a
    cluster's comm row cannot depend on where its own members sit, while its
    work row grows by exactly their weight where their tl lies in the span."""
    rng = np.random.default_rng(23)
    for t in range(12):
        n = int(rng.integers(10, 70))
        g = W.random_dag(rng, n, p_edge=0.12, max_weight=9, n_labels=1)
        K = int(rng.integers(2, 5))
        tl, _, _ = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))
        C = int(rng.integers(1, 6))
        cluster = rng.integers(-1, C, n)
        label = np.where(rng.random(n) < 0.5, rng.integers(0, K, n), -1)
        r1 = span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C, tl)
        for c in range(C):
            free = np.where(cluster == c, -1, label)
            r0 = span_work(n, g.src, g.dst, g.comp, g.edge_cost, free, K, cluster, C, tl,
                           clusters=[c])
            assert (r1["comm"][c] == r0["comm"][0]).all(), (t, c)
            assert r1["span_lo"][c] == r0["span_lo"][0] and r1["span_hi"][c] == r0["span_hi"][0]
            inside = (tl >= r0["span_lo"][0]) & (tl <= r0["span_hi"][0]) & (cluster == c)
            for k in range(K):
                extra = int(g.comp[inside & (label == k)].sum())
                assert r1["work"][c, k] == r0["work"][0, k] + extra, (t, c, k)
        # with every edge inside one cluster there is no communication at all
        one = np.zeros(n, np.int64)
        r2 = span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, one, 1, tl)
        assert (r2["comm"] == 0).all()


def test_eq2_rejects_bad_ids():
    with pytest.raises(ValueError):
        span_work(2, [0], [1], [1, 1], [1], [0, 2], 2, [-1, 0], 1, [0, 2])
    with pytest.raises(ValueError):
        span_work(2, [0], [1], [1, 1], [1], [0, 1], 2, [-1, 1], 1, [0, 2])
