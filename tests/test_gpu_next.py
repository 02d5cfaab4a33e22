"""GPU parity for the rows after the core path, through the C ABI, against the
oracle: Memory Heuristic II evaluation (pardnn_memory_balance). All values are
integers, so every comparison is exact. Each case prints its name first.
"""
import json
import os
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle.memory_balance import memory_balance

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "next")


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def P():
    import paper_2008_08636_amd as P
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    P.load_library()
    return P


def dev(x, dt):
    return torch.as_tensor(np.ascontiguousarray(x), dtype=dt).cuda()


def check_balance(g_nodes, mem, kind, tgt, pl_vp, K, out, cols):
    for p in cols:
        e = memory_balance(g_nodes, mem, kind, tgt, pl_vp[:, p], K)
        assert (out["res_mem"][p] == e["res_mem"]).all(), p
        assert (out["nor_mem"][p] == e["nor_mem"]).all(), p
        assert (out["balanced"][p] == e["balanced"]).all(), p
        assert int(out["ref_misplaced"][p]) == e["ref_misplaced"], p


def run_balance(G, pl_vp, kind, tgt, K):
    out = G.memory_balance(dev(pl_vp, torch.int32), dev(kind, torch.int32),
                           dev(tgt, torch.int32), K)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def test_memory_balance_paper_example(P):
    say("heuristic II paper example")
    d = json.load(open(os.path.join(GOLDEN, "heuristic2_paper_example.json")))
    G = P.Graph(d["n_nodes"], np.array(d["src"], np.int32), np.array(d["dst"], np.int32),
                np.array(d["comp"], np.int64), np.array(d["edge_cost"], np.int64),
                np.array(d["mem"], np.int64))
    pl = np.stack([d["placements"]["before"], d["placements"]["after"]], axis=1)
    out = run_balance(G, pl, d["node_type"], d["ref_target"], d["n_labels"])
    for p, name in enumerate(["before", "after"]):
        exp = d["expect"][name]
        assert out["res_mem"][p].tolist() == exp["res_mem"]
        assert out["nor_mem"][p].tolist() == exp["nor_mem"]
        assert out["balanced"][p].tolist() == exp["balanced"]
        assert int(out["ref_misplaced"][p]) == exp["ref_misplaced"]
    G.close()


@pytest.mark.parametrize("K,n_place", [(1, 3), (2, 1), (16, 37), (33, 5), (100, 70)])
def test_memory_balance_random(P, K, n_place):
    """K = 33 and 100 take the global-atomic path (more labels than LDS bins);
    70 placements span two placement tiles with a ragged tail."""
    say(f"heuristic II random K={K} P={n_place}")
    rng = np.random.default_rng(1000 + K)
    g = W.random_dag(rng, 700, p_edge=0.01, max_weight=9, n_labels=min(K, 4))
    kind, tgt = W.node_kinds(g, seed=K)
    pl = rng.integers(0, K, (g.n_nodes, n_place)).astype(np.int32)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_balance(G, pl, kind, tgt, K)
    check_balance(g.n_nodes, g.mem, kind, tgt, pl, K, out, range(n_place))
    G.close()


def test_memory_balance_degenerate(P):
    say("heuristic II degenerate kinds")
    rng = np.random.default_rng(5)
    g = W.random_dag(rng, 200, p_edge=0.02, max_weight=5, n_labels=3)
    pl = rng.integers(0, 3, (g.n_nodes, 4)).astype(np.int32)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    none = np.full(g.n_nodes, -1, np.int32)
    for kind in (np.zeros(g.n_nodes, np.int32), np.ones(g.n_nodes, np.int32),
                 np.full(g.n_nodes, 2, np.int32)):
        out = run_balance(G, pl, kind, none, 3)
        check_balance(g.n_nodes, g.mem, kind, none, pl, 3, out, range(4))
    G.close()
    # no memory at all
    z = np.zeros(g.n_nodes, np.int64)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, z)
    kind, tgt = W.node_kinds(g)
    out = run_balance(G, pl, kind, tgt, 3)
    assert out["balanced"].all()
    check_balance(g.n_nodes, z, kind, tgt, pl, 3, out, range(4))
    G.close()


def test_memory_balance_errors(P):
    say("heuristic II errors")
    rng = np.random.default_rng(6)
    g = W.random_dag(rng, 50, p_edge=0.1, max_weight=5, n_labels=2)
    kind, tgt = W.node_kinds(g)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    pl = np.zeros((g.n_nodes, 2), np.int32)
    bad = pl.copy()
    bad[3, 1] = 2
    with pytest.raises(P.PardnnError) as e:
        run_balance(G, bad, kind, tgt, 2)
    assert e.value.status == P.E_INVAL
    k2 = kind.copy()
    k2[7] = 3
    with pytest.raises(P.PardnnError) as e:
        run_balance(G, pl, k2, tgt, 2)
    assert e.value.status == P.E_INVAL
    k3, t3 = kind.copy(), tgt.copy()
    k3[9], t3[9] = 2, g.n_nodes
    with pytest.raises(P.PardnnError) as e:
        run_balance(G, pl, k3, t3, 2)
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        run_balance(G, pl, kind, tgt, 0)
    assert e.value.status == P.E_INVAL
    G.close()


def test_memory_balance_refinement_loop_full_size(P):
    """The 1000 placements of the refinement loop on the transformer graph, with
    the graph's own memory kinds (variables residual, their optimiser updates
    reference nodes): every placement against the oracle, element by element."""
    g = W.make_config(2)
    say(f"heuristic II full size V={g.n_nodes} P=1000")
    kind, tgt = W.node_kinds(g)
    sched = W.config4_moves(g, n_place=1000)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    pl = G.build_placements(dev(sched.base, torch.int32), dev(sched.ptr, torch.int64),
                            dev(sched.node, torch.int32), dev(sched.label, torch.int32))
    out = G.memory_balance(pl, dev(kind, torch.int32), dev(tgt, torch.int32), g.n_labels)
    torch.cuda.synchronize()
    res_total = int(g.mem[kind == 1].sum())
    nor_total = int(g.mem[kind == 0].sum())
    assert bool((out["res_mem"].sum(dim=1) == res_total).all())
    assert bool((out["nor_mem"].sum(dim=1) == nor_total).all())
    assert bool((out["balanced"].sum(dim=1) >= 1).all())
    host = {k: v.cpu().numpy() for k, v in out.items()}
    exp_pl = W.materialize_placements(sched)
    check_balance(g.n_nodes, g.mem, kind, tgt, exp_pl.T.copy(), g.n_labels, host, range(1000))
    G.close()


# ---------------------------------------------------------------------------
# Graph slicing primaries (Alg. 1): pardnn_slice_primaries
# ---------------------------------------------------------------------------
from oracle.slicing import slice_primaries  # noqa: E402


def check_slicing(P, g, K):
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = G.slice_primaries(K)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    G.close()
    primary, paths, ms = slice_primaries(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    assert (got["primary"] == primary).all()
    assert (got["makespan"] == ms).all(), (got["makespan"], ms)
    for j in range(K):
        n = int(got["path_len"][j])
        assert n == len(paths[j]), j
        assert (got["paths"][j, :n] == paths[j]).all(), j


@pytest.mark.parametrize("i,K", [(0, 16), (1, 8), (2, 16)])
def test_slicing_configs(P, i, K):
    g = W.make_config(i)
    say(f"slicing config{i} K={K} V={g.n_nodes}")
    check_slicing(P, g, K)


def test_slicing_small_and_exhausted(P):
    """Random small DAGs (zero weights and ties included) with K up to past the
    point where no node remains."""
    say("slicing small random DAGs")
    rng = np.random.default_rng(77)
    for t in range(25):
        n = int(rng.integers(1, 40))
        g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.05, 0.5)),
                         max_weight=int(rng.integers(0, 6)), n_labels=1)
        check_slicing(P, g, int(rng.integers(1, n + 3)))
    rng = np.random.default_rng(78)
    g = W.chain_graph(rng, 50)
    check_slicing(P, g, 3)


# ---------------------------------------------------------------------------
# Cluster criticality (Sec. 3.1.2): pardnn_cluster_criticality
# ---------------------------------------------------------------------------
from oracle.clusters import cluster_criticality  # noqa: E402


def check_clusters(P, g, cl, C):
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    crit, order = G.cluster_criticality(dev(cl, torch.int32), C)
    torch.cuda.synchronize()
    crit, order = crit.cpu().numpy(), order.cpu().numpy()
    G.close()
    ec, eo = cluster_criticality(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, cl, C)
    assert (crit == ec).all()
    assert (order == eo).all()


def test_clusters_small_random(P):
    """Random DAGs with clusters made of random paths (a few groupings that
    are no path among them) and with arbitrary groupings (mostly no path)."""
    say("cluster criticality small random DAGs")
    rng = np.random.default_rng(91)
    for t in range(40):
        n = int(rng.integers(1, 60))
        g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.05, 0.4)),
                         max_weight=int(rng.integers(0, 6)), n_labels=1)
        if t % 4 == 3:
            C = int(rng.integers(1, n + 5))
            cl = rng.integers(0, C, n)
        else:
            cl, C = W.path_clusters(rng, g, max_extra=int(rng.integers(1, 12)))
        check_clusters(P, g, cl.astype(np.int32), C)


def test_clusters_hand_example(P):
    say("cluster criticality hand example")
    d = json.load(open(os.path.join(GOLDEN, "criticality_whole_cluster.json")))
    n = d["n_nodes"]
    G = P.Graph(n, np.array(d["src"], np.int32), np.array(d["dst"], np.int32),
                np.array(d["comp"], np.int64), np.array(d["edge_cost"], np.int64),
                np.zeros(n, np.int64))
    crit, order = G.cluster_criticality(dev(d["cluster"], torch.int32), d["n_clusters"])
    torch.cuda.synchronize()
    assert crit.cpu().numpy().tolist() == d["expect"]["criticality"]
    assert order.cpu().numpy().tolist() == d["expect"]["order"]
    G.close()


@pytest.mark.parametrize("i", [0, 1, 2])
def test_clusters_of_slicing(P, i):
    """Clusters as the mapping stage sees them: the primaries of 16 slicing
    rounds, every other node a cluster of its own (tens of thousands of
    clusters on the transformer graph: several sort tiles)."""
    g = W.make_config(i)
    say(f"cluster criticality config{i} V={g.n_nodes}")
    K = 16
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    primary = G.slice_primaries(K)["primary"].cpu().numpy()
    G.close()
    cl = np.where(primary >= 0, primary, K + np.arange(g.n_nodes)).astype(np.int32)
    check_clusters(P, g, cl, K + g.n_nodes)


def test_clusters_label_paths(P):
    """The three ways the sweep gets its labels: levels and cluster ranks
    (usual), the cluster ids themselves (more than 2^16 levels, few
    clusters), the single-placement sweep (many levels and many clusters)."""
    rng = np.random.default_rng(93)
    g = W.chain_graph(rng, 70000)
    n = g.n_nodes
    say(f"cluster criticality label paths, chain V={n}")
    two = (np.arange(n) >= n // 2).astype(np.int32)      # ids fit: 2 clusters
    check_clusters(P, g, two, 2)
    alone = np.arange(n, dtype=np.int32)                 # neither fits
    check_clusters(P, g, alone, n)
    mixed = np.where(np.arange(n) % 3 == 0, np.arange(n) // 3, n).astype(np.int32)
    check_clusters(P, g, mixed, n + 1)                   # one large cluster + lone nodes
    runs = (np.arange(n) // 7).astype(np.int32)          # paths of 7 chain nodes
    check_clusters(P, g, runs, int(runs.max()) + 1)


def test_clusters_errors(P):
    say("cluster criticality errors")
    rng = np.random.default_rng(92)
    g = W.random_dag(rng, 40, p_edge=0.1, max_weight=5, n_labels=1)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    cl = np.zeros(g.n_nodes, np.int32)
    cl[5] = 3
    with pytest.raises(P.PardnnError) as e:
        G.cluster_criticality(dev(cl, torch.int32), 3)
    assert e.value.status == P.E_INVAL
    cl[5] = -1
    with pytest.raises(P.PardnnError) as e:
        G.cluster_criticality(dev(cl, torch.int32), 3)
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        G.cluster_criticality(dev(np.zeros(g.n_nodes, np.int32), torch.int32), 0)
    assert e.value.status == P.E_INVAL
    # still usable after an error
    check_clusters(P, g, np.arange(g.n_nodes, dtype=np.int32) % 7, 7)
    G.close()


# ---------------------------------------------------------------------------
# Eq. 2 span-work terms (Sec. 3.1.2): pardnn_span_work
# ---------------------------------------------------------------------------
from oracle.span_work import span_work  # noqa: E402
from oracle import tb_levels  # noqa: E402


def run_span(G, label, K, cluster, C, tl):
    out = G.span_work(dev(label, torch.int32), K, dev(cluster, torch.int32), C,
                      dev(tl, torch.int64))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def check_span(got, exp, rows=None):
    for key in ("span_lo", "span_hi", "work", "comm", "choice"):
        g = got[key] if rows is None else got[key][rows]
        assert (g == exp[key]).all(), key


def test_span_work_hand_example(P):
    say("eq2 hand example")
    d = json.load(open(os.path.join(GOLDEN, "eq2_hand_example.json")))
    G = P.Graph(d["n_nodes"], np.array(d["src"], np.int32), np.array(d["dst"], np.int32),
                np.array(d["comp"], np.int64), np.array(d["edge_cost"], np.int64),
                np.zeros(d["n_nodes"], np.int64))
    got = run_span(G, d["label"], d["K"], d["cluster"], d["n_clusters"], d["tl"])
    for key, exp in d["expect"].items():
        assert got[key].tolist() == exp, key
    G.close()


def test_span_work_small_random(P):
    """Random DAGs, partial placements and clusters (in some cases with members
    already placed); tl either the graph's top levels or arbitrary values with
    many duplicates (negative ones included)."""
    say("eq2 small random")
    rng = np.random.default_rng(801)
    for t in range(24):
        n = int(rng.integers(1, 300))
        g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.005, 0.1)),
                         max_weight=int(rng.integers(0, 9)), n_labels=1)
        K = int(rng.integers(1, 9))
        C = int(rng.integers(0, n + 4))
        label = np.where(rng.random(n) < 0.5, rng.integers(0, K, n), -1).astype(np.int32)
        if C and t % 4 == 1:    # members already placed: edges inside stay free
            cluster = rng.integers(-1, C, n).astype(np.int32)
        else:
            cluster = (np.where(label < 0, rng.integers(-1, C, n), -1) if C else
                       np.full(n, -1)).astype(np.int32)
        if t % 3 == 2:
            tl = rng.integers(-5, 12, n).astype(np.int64)
        else:
            tl = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))[0]
        G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
        got = run_span(G, label, K, cluster, C, tl)
        G.close()
        exp = span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C, tl)
        check_span(got, exp)


def test_span_work_wide_cases(P):
    """More than 64 partitions (the choice in its own pass) and a tl range too
    wide for one (partition, tl) sort key (two sorts instead of one)."""
    say("eq2 wide cases")
    rng = np.random.default_rng(803)
    for K, wide in [(100, False), (3, True), (70, True)]:
        n = 400
        g = W.random_dag(rng, n, p_edge=0.01, max_weight=9, n_labels=1)
        label = np.where(rng.random(n) < 0.6, rng.integers(0, K, n), -1).astype(np.int32)
        C = 90
        cluster = np.where(label < 0, rng.integers(-1, C, n), -1).astype(np.int32)
        if wide:
            tl = rng.integers(-2 ** 62, 2 ** 62, n).astype(np.int64)
            tl[:5] = [-2 ** 62, 2 ** 62 - 1, 0, 0, 7]
        else:
            tl = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))[0]
        # comp is small, so tl + comp stays inside int64
        G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
        got = run_span(G, label, K, cluster, C, tl)
        G.close()
        check_span(got, span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C, tl))


@pytest.mark.parametrize("i", [0, 1, 2])
def test_span_work_mapping_state(P, i):
    """The mapping stage's state on each graph: the primaries of 16 slicing
    rounds mapped to 16 partitions, every other node a secondary cluster of
    its own; tl with every edge paying. All clusters on C0-C1; on the
    transformer graph 1,000 seeded random rows and both ends (each row
    computed by the oracle alone) and the Eq. 2 choice rule on every row."""
    g = W.make_config(i)
    n = g.n_nodes
    say(f"eq2 mapping state config{i} V={n}")
    K = 16
    G = P.Graph(n, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    primary = G.slice_primaries(K)["primary"].cpu().numpy()
    label = primary.astype(np.int32)
    free = np.nonzero(primary < 0)[0]
    cluster = np.full(n, -1, np.int32)
    cluster[free] = np.arange(free.size)
    C = int(free.size)
    tl = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))[0]
    got = run_span(G, label, K, cluster, C, tl)
    G.close()
    rows = None
    if n >= 50000:
        pick = np.random.default_rng(900 + i).choice(C, 1000, replace=False)
        rows = sorted(set(pick.tolist()) | {0, 1, C - 2, C - 1})
    exp = span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C, tl,
                    clusters=rows)
    check_span(got, exp, rows)
    if rows is not None:
        # every row: the choice minimises Eq. 2 with the tie rules
        tot = got["comm"].sum(axis=1, keepdims=True)
        cost = got["work"] + tot - got["comm"]
        best = cost.min(axis=1)
        assert (cost[np.arange(C), got["choice"]] == best).all()


def test_span_work_cached_tl_order(P):
    """Calls with the same tl and new partitions reuse the tl order kept on
    the handle; a tl changed in place (same buffer) or a new buffer with equal
    contents must give the oracle's answer every time."""
    g = W.make_config(1)
    n = g.n_nodes
    say(f"eq2 cached tl order config1 V={n}")
    rng = np.random.default_rng(805)
    K, C = 8, 500
    tl_np = tb_levels(n, g.src, g.dst, g.comp, g.edge_cost, np.arange(n))[0]
    tl = dev(tl_np, torch.int64)
    G = P.Graph(n, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    for t in range(5):
        label = np.where(rng.random(n) < 0.5, rng.integers(0, K, n), -1).astype(np.int32)
        cluster = np.where(label < 0, rng.integers(-1, C, n), -1).astype(np.int32)
        if t == 2:      # changed in place: the same device buffer, new contents
            tl_np = tl_np.copy()
            tl_np[rng.integers(0, n, 50)] += 3
            tl.copy_(dev(tl_np, torch.int64))
        if t == 3:      # a new buffer with the same contents
            tl = dev(tl_np, torch.int64)
        out = G.span_work(dev(label, torch.int32), K, dev(cluster, torch.int32), C, tl)
        torch.cuda.synchronize()
        got = {k: v.cpu().numpy() for k, v in out.items()}
        check_span(got, span_work(n, g.src, g.dst, g.comp, g.edge_cost, label, K, cluster, C,
                                  tl_np))
    G.close()


def test_span_work_errors(P):
    say("eq2 errors")
    rng = np.random.default_rng(802)
    g = W.random_dag(rng, 30, p_edge=0.1, max_weight=5, n_labels=1)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    lab = np.zeros(30, np.int32)
    cl = np.full(30, -1, np.int32)
    tl = np.zeros(30, np.int64)
    bad = lab.copy()
    bad[4] = 2
    with pytest.raises(P.PardnnError) as e:
        run_span(G, bad, 2, cl, 3, tl)
    assert e.value.status == P.E_INVAL
    bad = cl.copy()
    bad[4] = 3
    with pytest.raises(P.PardnnError) as e:
        run_span(G, lab, 2, bad, 3, tl)
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        run_span(G, lab, 0, cl, 3, tl)
    assert e.value.status == P.E_INVAL
    # still usable after an error
    cl2 = (np.arange(30) % 4 - 1).astype(np.int32)
    lab2 = np.where(cl2 < 0, 1, -1).astype(np.int32)
    got = run_span(G, lab2, 2, cl2, 3, tl)
    check_span(got, span_work(30, g.src, g.dst, g.comp, g.edge_cost, lab2, 2, cl2, 3, tl))
    G.close()


def test_slicing_beyond_packed_levels(P):
    """More than 2^16 levels: the rounds take the single-placement sweep
    instead of the pair sweep (labels = levels no longer fit 16 bits)."""
    rng = np.random.default_rng(79)
    g = W.chain_graph(rng, 70000)
    say(f"slicing deep chain V={g.n_nodes}")
    check_slicing(P, g, 2)


def test_next_rows_on_empty_and_single_node_graphs(P):
    """V = 0 and V = 1 through every entry point after the core path, against
    the oracle."""
    say("next rows: empty and single-node graphs")
    e32, e64 = np.zeros(0, np.int32), np.zeros(0, np.int64)
    for n in (0, 1):
        comp = np.full(n, 5, np.int64)
        mem = np.full(n, 7, np.int64)
        G = P.Graph(n, e32, e32, comp, e64, mem)
        # Heuristic II
        pl = np.zeros((n, 3), np.int32)
        kind = np.ones(n, np.int32)
        tgt = np.full(n, -1, np.int32)
        out = run_balance(G, pl, kind, tgt, 2)
        check_balance(n, mem, kind, tgt, pl, 2, out, range(3))
        # cluster criticality
        crit, order = G.cluster_criticality(dev(np.zeros(n, np.int32), torch.int32), 3)
        ec, eo = cluster_criticality(n, e32, e32, comp, e64, np.zeros(n, np.int64), 3)
        assert crit.cpu().numpy().tolist() == ec.tolist() and order.cpu().numpy().tolist() == eo.tolist()
        # span work
        lab = np.full(n, -1, np.int32)
        cl = np.zeros(n, np.int32)
        tl = np.zeros(n, np.int64)
        got = run_span(G, lab, 2, cl, 2, tl)
        check_span(got, span_work(n, e32, e32, comp, e64, lab, 2, cl, 2, tl))
        # slicing
        out = G.slice_primaries(2)
        torch.cuda.synchronize()
        primary, paths, ms = slice_primaries(n, e32, e32, comp, e64, 2)
        assert out["makespan"].cpu().numpy().tolist() == ms.tolist()
        assert out["primary"].cpu().numpy().tolist() == primary.tolist()
        for j in range(2):
            k = int(out["path_len"][j])
            assert out["paths"][j, :k].cpu().numpy().tolist() == paths[j].tolist()
        G.close()


def test_binding_rejects_short_buffers(P):
    """The binding checks buffer sizes before the C call, so a short output
    never reaches a kernel."""
    say("binding: short buffers")
    rng = np.random.default_rng(804)
    g = W.random_dag(rng, 50, p_edge=0.1, max_weight=5, n_labels=2)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    lab = dev(np.zeros(g.n_nodes, np.int32), torch.int32)
    short64 = torch.empty(g.n_nodes - 1, dtype=torch.int64, device="cuda")
    ok64 = torch.empty(g.n_nodes, dtype=torch.int64, device="cuda")
    m = torch.empty(1, dtype=torch.int64, device="cuda")
    with pytest.raises(ValueError):
        P.pardnn_tb_levels(G.handle, lab, short64, ok64, m)
    with pytest.raises(ValueError):
        P.pardnn_span_work(G.handle, lab, 2, lab, 3, ok64, torch.empty(3, dtype=torch.int64,
                           device="cuda"), torch.empty(3, dtype=torch.int64, device="cuda"),
                           torch.empty(5, dtype=torch.int64, device="cuda"),
                           torch.empty(6, dtype=torch.int64, device="cuda"),
                           torch.empty(3, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        P.pardnn_cluster_criticality(G.handle, lab, 4, torch.empty(3, dtype=torch.int64,
                                     device="cuda"), torch.empty(4, dtype=torch.int32,
                                                                 device="cuda"))
    G.close()


# ---------------------------------------------------------------------------
# Graph slicing in full (Alg. 1): primaries and secondaries, pardnn_slice_graph
# ---------------------------------------------------------------------------
from oracle.slicing import slice_all  # noqa: E402


def check_slice_all(P, g, K):
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = G.slice_graph(K)
    torch.cuda.synchronize()
    cluster = out["cluster"].cpu().numpy()
    paths = [p.cpu().numpy() for p in out["paths"]]
    G.close()
    ecl, epaths = slice_all(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, K)
    assert len(paths) == len(epaths), (len(paths), len(epaths))
    for j, (a, b) in enumerate(zip(paths, epaths)):
        assert a.tolist() == b.tolist(), j
    assert (cluster == ecl).all()


def test_slice_graph_small_random(P):
    say("slice_graph small random DAGs")
    rng = np.random.default_rng(710)
    for t in range(40):
        n = int(rng.integers(0, 60)) if t > 1 else t
        g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.02, 0.5)),
                         max_weight=int(rng.integers(0, 6)), n_labels=1)
        check_slice_all(P, g, int(rng.integers(0, 6)))


def test_slice_graph_hubs_and_long_lists(P):
    """Nodes with more successors than a record holds inline, and with
    hundreds of them (the walk's list path)."""
    say("slice_graph hubs")
    rng = np.random.default_rng(711)
    g = level_hub_graph(rng)
    for K in (0, 1, 3):
        check_slice_all(P, g, K)


def level_hub_graph(rng):
    widths = [1, 300, 2, 40, 1, 200, 7]
    fan = [1, 1, 300, 2, 40, 1, 150]
    return W.layered_dag(rng, widths, fan, max_span=3, n_labels=1)


@pytest.mark.parametrize("i,K", [(0, 8), (1, 8), (2, 16)])
def test_slice_graph_configs(P, i, K):
    g = W.make_config(i)
    say(f"slice_graph config{i} K={K} V={g.n_nodes}")
    check_slice_all(P, g, K)


def test_slice_graph_maps_in_device_memory(P):
    """The walk with its bit maps in device memory (as for graphs too large
    for LDS) gives the same clusters."""
    g = W.make_config(1)
    say(f"slice_graph config1 maps in device memory V={g.n_nodes}")
    os.environ["PARDNN_PEEL_GLOBAL_MAPS"] = "1"
    try:
        check_slice_all(P, g, 4)
    finally:
        del os.environ["PARDNN_PEEL_GLOBAL_MAPS"]


def test_slicing_and_criticality_with_grid_levels(P, monkeypatch):
    """Slicing rounds and cluster criticality run single-placement sweeps;
    with every level above 65 nodes computed grid-wide they are unchanged."""
    monkeypatch.setenv("PARDNN_WIDE_LEVEL", "65")
    g = W.make_config(1)
    say(f"slicing and criticality, grid-wide levels, config1 V={g.n_nodes}")
    check_slice_all(P, g, 6)
    rng = np.random.default_rng(95)
    cl, C = W.path_clusters(rng, g, max_extra=20)
    check_clusters(P, g, cl.astype(np.int32), C)
