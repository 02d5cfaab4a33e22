"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

All values are int64/int32/uint8, so every comparison is bit-exact. Inputs
come from the seeded generators in ``workloads``; expected values come only
from ``oracle``. Each case prints its name before touching the GPU.
"""
import functools
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


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


@functools.lru_cache(maxsize=None)
def cfg(i):
    return W.make_config(i)


def dev(x, dt):
    return torch.as_tensor(np.ascontiguousarray(x), dtype=dt).cuda()


def gpu_single(P, g, placement=None):
    lab_np = g.placement if placement is None else placement
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    level, order, lptr, n = G.levelize()
    lab = dev(lab_np, torch.int32)
    tl, bl, m = G.tb_levels(lab)
    crit, path, plen = G.critical_path(lab, tl, bl, m)
    sums, over = G.label_memory(lab, g.n_labels, dev(g.capacity, torch.int64))
    torch.cuda.synchronize()
    out = {
        "level": level.cpu().numpy(), "order": order.cpu().numpy(),
        "level_ptr": lptr.cpu().numpy(), "n_levels": n,
        "tl": tl.cpu().numpy(), "bl": bl.cpu().numpy(), "makespan": int(m.item()),
        "is_critical": crit.cpu().numpy(), "path": path[: int(plen.item())].cpu().numpy(),
        "label_mem": sums.cpu().numpy(), "overflow": over.cpu().numpy(),
    }
    G.close()
    return out


def oracle_single(g, placement=None):
    lab = g.placement if placement is None else placement
    level, order, lptr, n = oracle.levelize(g.n_nodes, g.src, g.dst)
    r = oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem, lab,
                        g.n_labels, g.capacity)
    r.update(level=level, order=order, level_ptr=lptr, n_levels=n)
    return r


def assert_same(got, exp, keys=None):
    keys = keys or ["level", "order", "level_ptr", "n_levels", "tl", "bl", "makespan",
                    "is_critical", "path", "label_mem", "overflow"]
    for k in keys:
        a, b = got[k], exp[k]
        if isinstance(b, np.ndarray):
            assert a.shape == b.shape, (k, a.shape, b.shape)
            bad = np.nonzero(a != b)[0]
            assert bad.size == 0, f"{k}: {bad.size} mismatches, first at {bad[:5]}: {a[bad[:5]]} vs {b[bad[:5]]}"
        else:
            assert a == b, (k, a, b)


# ------------------------------------------------------------ single placement --

@pytest.mark.parametrize("i", [0, 1, 2, 3])
def test_config_single(P, i):
    g = cfg(i)
    say(f"config{i} single V={g.n_nodes} E={g.n_edges}")
    got = gpu_single(P, g)
    exp = oracle_single(g)
    assert_same(got, exp)


def test_random_small_graphs(P):
    say("random small DAGs")
    rng = np.random.default_rng(20080863)
    for t in range(150):
        n = int(rng.integers(0, 40)) if t > 2 else t  # includes V = 0, 1, 2
        g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.0, 0.5)),
                         max_weight=int(rng.integers(0, 5)), n_labels=int(rng.integers(1, 4)))
        got = gpu_single(P, g)
        exp = oracle_single(g)
        assert_same(got, exp)


def test_single_labels_beyond_16_bits(P):
    """Labels outside [0, 2^16) -- one stray label is enough -- send a single
    evaluation to the single-placement sweep instead of the batched one; the
    results must not depend on which ran."""
    say("single placement, labels beyond 16 bits")
    rng = np.random.default_rng(65536)
    for t, g in enumerate([W.random_dag(rng, 600, p_edge=0.01, max_weight=9, n_labels=3),
                           cfg(0)]):
        pools = [np.array([-5, 65536, 70000, 2 ** 30, 123456789]), np.arange(4)]
        for pool in pools:
            lab = pool[rng.integers(0, pool.size, g.n_nodes)].astype(np.int32)
            if pool.size == 4:
                lab[g.n_nodes // 2] = 65536   # a single label out of range
            G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
            tl, bl, m = G.tb_levels(dev(lab, torch.int32))
            crit, path, plen = G.critical_path(dev(lab, torch.int32), tl, bl, m)
            torch.cuda.synchronize()
            etl, ebl, em = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab)
            ecrit, epath = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab,
                                                etl, ebl, em)
            assert (tl.cpu().numpy() == etl).all() and (bl.cpu().numpy() == ebl).all()
            assert int(m.item()) == em
            assert (crit.cpu().numpy() == ecrit).all()
            assert (path[: int(plen.item())].cpu().numpy() == epath).all()
            G.close()


def test_all_zero_weights_ties(P):
    # every path has length 0: every node critical, path = lexicographic minimum
    say("all-zero weights")
    rng = np.random.default_rng(5)
    g = W.random_dag(rng, 300, p_edge=0.02, max_weight=0, n_labels=2)
    assert_same(gpu_single(P, g), oracle_single(g))


def test_unit_weights_give_levels(P):
    say("unit weights")
    g = cfg(1)
    g1 = W.SynthGraph("unit", g.n_nodes, g.src, g.dst, np.ones(g.n_nodes, np.int64),
                      np.zeros(g.n_edges, np.int64), g.mem, g.placement, g.n_labels,
                      g.capacity, {})
    got = gpu_single(P, g1)
    assert (got["tl"] == got["level"]).all()


def test_critical_path_arbitrary_inputs(P):
    # the path definition holds for any tl/bl/M, not only consistent ones
    say("critical_path on perturbed inputs")
    g = cfg(0)
    rng = np.random.default_rng(3)
    tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.placement)
    tl2 = tl.copy()
    bl2 = bl.copy()
    idx = rng.choice(g.n_nodes, 200, replace=False)
    tl2[idx] += rng.integers(-5, 6, 200)
    bl2[idx[::2]] -= 3
    exp_crit, exp_path = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost,
                                              g.placement, tl2, bl2, m)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    lab = dev(g.placement, torch.int32)
    crit, path, plen = G.critical_path(lab, dev(tl2, torch.int64), dev(bl2, torch.int64),
                                       dev([m], torch.int64))
    torch.cuda.synchronize()
    assert (crit.cpu().numpy() == exp_crit).all()
    assert (path[: int(plen.item())].cpu().numpy() == exp_path).all()
    G.close()


def test_critical_path_walk_leaves_critical_set(P):
    """Inconsistent tl / bl on which the walk passes a non-critical node: the
    hand-derived 4-node case (path [0, 1, 3], node 1 not critical), then seeded
    random DAGs with tl, bl drawn from a small range so that tight edges out of
    non-critical nodes are common; expected values from the oracle."""
    say("critical_path through non-critical nodes")
    cases = [(4, [0, 1, 1], [1, 2, 3], [1] * 4, [0] * 3, [0] * 4, [0, 2, 2, 2], [3, 2, 1, 0], 3)]
    rng = np.random.default_rng(77)
    for t in range(120):
        n = int(rng.integers(1, 48))
        g = W.random_dag(rng, n, p_edge=float(rng.uniform(0.05, 0.4)),
                         max_weight=int(rng.integers(0, 3)), n_labels=int(rng.integers(1, 3)))
        tl = rng.integers(0, 5, n).astype(np.int64)
        bl = rng.integers(0, 5, n).astype(np.int64)
        m = int((tl + bl)[int(rng.integers(0, n))])
        cases.append((n, g.src, g.dst, g.comp, g.edge_cost, g.placement, tl, bl, m))
    walked_off = 0
    for (n, src, dst, comp, cost, lab, tl, bl, m) in cases:
        src = np.asarray(src, np.int32)
        dst = np.asarray(dst, np.int32)
        comp = np.asarray(comp, np.int64)
        cost = np.asarray(cost, np.int64)
        lab = np.asarray(lab, np.int32)
        tl = np.asarray(tl, np.int64)
        bl = np.asarray(bl, np.int64)
        ecrit, epath = oracle.critical_path(n, src, dst, comp, cost, lab, tl, bl, m)
        walked_off += int((ecrit[epath] == 0).any())
        G = P.Graph(n, src, dst, comp, cost, np.zeros(n, np.int64))
        crit, path, plen = G.critical_path(dev(lab, torch.int32), dev(tl, torch.int64),
                                           dev(bl, torch.int64), dev([m], torch.int64))
        torch.cuda.synchronize()
        assert (crit.cpu().numpy() == ecrit).all()
        assert path[: int(plen.item())].cpu().numpy().tolist() == epath.tolist()
        G.close()
    assert walked_off >= 10   # the cases do exercise the walk off the critical set


def test_determinism_and_stream(P):
    say("determinism on a side stream")
    g = cfg(2)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    lab = dev(g.placement, torch.int32)
    s = torch.cuda.Stream()
    outs = []
    for _ in range(2):
        with torch.cuda.stream(s):
            P.pardnn_set_stream(G.handle, s)
            tl, bl, m = G.tb_levels(lab)
        s.synchronize()
        outs.append((tl.cpu().numpy(), bl.cpu().numpy(), int(m.item())))
    assert (outs[0][0] == outs[1][0]).all() and (outs[0][1] == outs[1][1]).all()
    assert outs[0][2] == outs[1][2]
    G.close()


# --------------------------------------------------------------------- errors --

def test_alloc_failure_injection(P, monkeypatch):
    """Each allocation of a create -> levelize -> tb_levels -> critical path ->
    label memory -> batch sequence fails once in turn (PARDNN_FAULT_ALLOC=n,
    n = 1, 2, ...): the call that meets the failure returns E_NOMEM, the same
    handle then finishes the sequence (the retried call allocates only what is
    missing), and every result equals the oracle's."""
    g = cfg(0)
    exp = oracle_single(g)
    pls_np = np.stack([g.placement, (g.placement + 1) % g.n_labels], axis=1).astype(np.int32)
    exp_b = [oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem,
                             pls_np[:, p].copy(), g.n_labels, g.capacity) for p in range(2)]
    lab = dev(g.placement, torch.int32)
    pls = dev(pls_np, torch.int32)
    cap = dev(g.capacity, torch.int64)
    hits = []
    for n in range(1, 400):
        say(f"allocation failure at attempt {n}")
        monkeypatch.setenv("PARDNN_FAULT_ALLOC", str(n))
        hit = []

        def attempt(name, fn):
            try:
                return fn()
            except P.PardnnError as e:
                assert e.status == P.E_NOMEM, (n, name, str(e))
                assert not hit, (n, name, hit)   # one failure per value
                hit.append(name)
                return fn()

        G = attempt("create", lambda: P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost,
                                              g.mem))
        level, order, lptr, nl = attempt("levelize", G.levelize)
        tl, bl, m = attempt("tb_levels", lambda: G.tb_levels(lab))
        crit, path, plen = attempt("critical_path", lambda: G.critical_path(lab, tl, bl, m))
        sums, over = attempt("label_memory", lambda: G.label_memory(lab, g.n_labels, cap))
        out = attempt("batch", lambda: G.evaluate_batch(pls, g.n_labels, cap))
        torch.cuda.synchronize()
        got = {"level": level.cpu().numpy(), "order": order.cpu().numpy(),
               "level_ptr": lptr.cpu().numpy(), "n_levels": nl, "tl": tl.cpu().numpy(),
               "bl": bl.cpu().numpy(), "makespan": int(m.item()),
               "is_critical": crit.cpu().numpy(), "path": path[: int(plen.item())].cpu().numpy(),
               "label_mem": sums.cpu().numpy(), "overflow": over.cpu().numpy()}
        assert_same(got, exp)
        for p in range(2):
            e = exp_b[p]
            assert (out["tl"][:, p].cpu().numpy() == e["tl"]).all(), (n, p)
            assert (out["bl"][:, p].cpu().numpy() == e["bl"]).all(), (n, p)
            assert int(out["makespan"][p]) == e["makespan"]
            assert (out["is_critical"][:, p].cpu().numpy() == e["is_critical"]).all()
            k = int(out["path_len"][p])
            assert out["path"][p, :k].cpu().numpy().tolist() == e["path"].tolist()
            assert (out["label_mem"][p].cpu().numpy() == e["label_mem"]).all()
            assert (out["overflow"][p].cpu().numpy() == e["overflow"]).all()
        G.close()
        if not hit:
            break
        hits.append(hit[0])
    assert not hit, "the sequence never ran without a failure"
    # every call of the sequence met a failure at least once
    assert {"create", "levelize", "tb_levels", "batch"} <= set(hits), hits


def test_fixed_entry_point_attempts_no_allocation(P, monkeypatch):
    """pardnn_evaluate_batch_fixed on a levelized handle makes no allocation
    attempt: with PARDNN_FAULT_ALLOC=1 set just before it, it succeeds, and
    the failure lands on the next call that allocates (the first batch
    workspace of the allocating entry point)."""
    say("fixed entry point under allocation-failure injection")
    g = cfg(0)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    L = P.pardnn_levelize(G.handle)
    pls_np = np.stack([g.placement, (g.placement + 2) % g.n_labels], axis=1).astype(np.int32)
    pls = dev(pls_np, torch.int32)
    cap = dev(g.capacity, torch.int64)
    V, K = g.n_nodes, g.n_labels
    i64 = dict(dtype=torch.int64, device="cuda")
    o = {"tl": torch.empty((V, 2), **i64), "bl": torch.empty((V, 2), **i64),
         "m": torch.empty(2, **i64), "crit": torch.empty((V, 2), dtype=torch.uint8, device="cuda"),
         "path": torch.empty((2, max(L, 1)), dtype=torch.int32, device="cuda"),
         "plen": torch.empty(2, dtype=torch.int32, device="cuda"),
         "lm": torch.empty((2, K), **i64), "ov": torch.empty((2, K), **i64)}
    monkeypatch.setenv("PARDNN_FAULT_ALLOC", "1")
    P.pardnn_evaluate_batch_fixed(G.handle, 2, pls, K, cap, o["tl"], o["bl"], o["m"], o["crit"],
                                  o["path"], max(L, 1), o["plen"], o["lm"], o["ov"])
    with pytest.raises(P.PardnnError) as ei:
        G.evaluate_batch(pls, K, cap)
    assert ei.value.status == P.E_NOMEM
    monkeypatch.delenv("PARDNN_FAULT_ALLOC")
    torch.cuda.synchronize()
    for p in range(2):
        e = oracle.evaluate(V, g.src, g.dst, g.comp, g.edge_cost, g.mem, pls_np[:, p].copy(), K,
                            g.capacity)
        assert (o["tl"][:, p].cpu().numpy() == e["tl"]).all()
        assert (o["bl"][:, p].cpu().numpy() == e["bl"]).all()
        assert int(o["m"][p]) == e["makespan"]
        assert (o["lm"][p].cpu().numpy() == e["label_mem"]).all()
    G.close()


def test_error_paths(P):
    say("error paths")
    def mk(n, src, dst, comp=None, cost=None, mem=None):
        comp = np.ones(n, np.int64) if comp is None else np.asarray(comp, np.int64)
        cost = np.ones(len(src), np.int64) if cost is None else np.asarray(cost, np.int64)
        mem = np.ones(n, np.int64) if mem is None else np.asarray(mem, np.int64)
        return P.Graph(n, np.asarray(src, np.int32), np.asarray(dst, np.int32), comp, cost, mem)

    with pytest.raises(P.PardnnError) as e:
        mk(3, [0, 5], [1, 2])
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        mk(3, [0], [-1])
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        mk(2, [0], [1], comp=[1, -1])
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        mk(2, [0], [1], cost=[-7])
    assert e.value.status == P.E_INVAL
    big = np.iinfo(np.int64).max
    with pytest.raises(P.PardnnError) as e:
        mk(2, [0], [1], comp=[big - 5, 0], cost=[10])
    assert e.value.status == P.E_OVERFLOW
    with pytest.raises(P.PardnnError) as e:
        mk(2, [0], [1], mem=[big, 1])
    assert e.value.status == P.E_OVERFLOW
    ok = mk(2, [0], [1], comp=[big - 11, 0], cost=[10])  # exactly at the bound minus one
    ok.close()
    # cycles and self-loops
    for src, dst in [([0, 1, 2], [1, 2, 0]), ([1], [1]), ([0, 1, 1], [1, 2, 1])]:
        G = mk(3, src, dst)
        with pytest.raises(P.PardnnError) as e:
            G.levelize()
        assert e.value.status == P.E_CYCLE
        lab = dev([0, 0, 0], torch.int32)
        with pytest.raises(P.PardnnError) as e:
            G.tb_levels(lab)
        assert e.value.status == P.E_CYCLE
        G.close()
    # labels out of range, negative capacity, bad move ids
    G = mk(3, [0, 1], [1, 2])
    with pytest.raises(P.PardnnError) as e:
        G.label_memory(dev([0, 3, 1], torch.int32), 3)
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        G.label_memory(dev([0, 1, 1], torch.int32), 2, dev([5, -1], torch.int64))
    assert e.value.status == P.E_INVAL
    place = dev([0, 0, 0], torch.int32)
    with pytest.raises(P.PardnnError) as e:
        G.apply_moves(place, dev([1, 7], torch.int32), dev([2, 2], torch.int32))
    assert e.value.status == P.E_INVAL
    assert place.cpu().tolist() == [0, 0, 0]  # nothing applied
    G.close()


# ---------------------------------------------------------------- moves --

def test_apply_moves(P):
    say("apply_moves")
    rng = np.random.default_rng(11)
    g = cfg(0)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    place = g.placement.copy()
    node = rng.integers(0, g.n_nodes, 500).astype(np.int32)  # with repeats
    label = rng.integers(-3, 9, 500).astype(np.int32)
    d = dev(place, torch.int32)
    G.apply_moves(d, dev(node, torch.int32), dev(label, torch.int32))
    for a, b in zip(node, label):  # in order, later wins
        place[a] = b
    assert (d.cpu().numpy() == place).all()
    G.close()


def test_build_placements(P):
    say("build_placements")
    g = cfg(0)
    sched = W.config4_moves(g, n_place=70, frac=0.05, seed=77)
    # add a repeated node inside one step and an empty step
    node = sched.node.copy()
    node[sched.ptr[3] + 1] = node[sched.ptr[3]]
    ptr = sched.ptr.copy()
    ptr[5] = ptr[4]  # step 4 now empty, step 5 gets its moves
    sched2 = W.MoveSchedule(sched.base, ptr, node, sched.label, sched.n_labels)
    exp = W.materialize_placements(sched2).T.copy()  # [V][P]
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    got = G.build_placements(dev(sched2.base, torch.int32), dev(ptr, torch.int64),
                             dev(node, torch.int32), dev(sched2.label, torch.int32))
    torch.cuda.synchronize()
    assert (got.cpu().numpy() == exp).all()
    G.close()


# ---------------------------------------------------------------- batches --

def check_batch(g, placements_vp, out, cols):
    for p in cols:
        lab = placements_vp[:, p].copy()
        exp = oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem, lab,
                              g.n_labels, g.capacity)
        assert (out["tl"][:, p] == exp["tl"]).all(), p
        assert (out["bl"][:, p] == exp["bl"]).all(), p
        assert out["makespan"][p] == exp["makespan"], p
        assert (out["is_critical"][:, p] == exp["is_critical"]).all(), p
        plen = out["path_len"][p]
        assert (out["path"][p, :plen] == exp["path"]).all(), p
        assert (out["label_mem"][p] == exp["label_mem"]).all(), p
        assert (out["overflow"][p] == exp["overflow"]).all(), p


def run_batch(P, G, placements_vp, g):
    out = G.evaluate_batch(dev(placements_vp, torch.int32), g.n_labels,
                           dev(g.capacity, torch.int64))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


@pytest.mark.parametrize("i,n_place", [(0, 37), (1, 5), (2, 9)])
def test_batch_random_placements(P, i, n_place):
    g = cfg(i)
    say(f"batch config{i} P={n_place}")
    rng = np.random.default_rng(100 + i)
    pl = rng.integers(0, g.n_labels, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 0] = g.placement
    pl[:, -1] = 0  # a single label: no communication at all
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_batch(P, G, pl, g)
    check_batch(g, pl, out, range(n_place))
    # the batched tl/bl/M agree with the single-placement entry point
    lab = dev(pl[:, 1].copy(), torch.int32)
    tl, bl, m = G.tb_levels(lab)
    torch.cuda.synchronize()
    assert (tl.cpu().numpy() == out["tl"][:, 1]).all() and int(m.item()) == out["makespan"][1]
    G.close()


def _long_edge_coverage(g):
    """How a graph exercises the batch sweep's long-edge machinery, from its
    shape alone (blocks of 8 steps; an edge is long when its neighbour's step
    is at most 8 k - 12 for the owner's block k; at most 512 neighbours per
    block get LDS entries; a level of the fast shape -- at most 64 nodes, 128
    span-1 and 192 longer edges -- with more than 64 longer edges left to
    gather from the workspace takes the general path). Per direction: blocks
    past 512 neighbours, fast-shaped levels past 64 gathers, fast levels
    with some gathers."""
    src, dst = np.asarray(g.src, np.int64), np.asarray(g.dst, np.int64)
    lvl = oracle.levelize(g.n_nodes, src, dst)[0].astype(np.int64)
    L = int(lvl.max() + 1)
    span, w = lvl[dst] - lvl[src], np.bincount(lvl, minlength=L)
    out = {}
    for fwd in (True, False):
        own, nb = (dst, src) if fwd else (src, dst)
        step = lvl[own] if fwd else L - 1 - lvl[own]
        nstep = lvl[nb] if fwd else L - 1 - lvl[nb]
        nn = np.bincount(step[span == 1], minlength=L)
        nf = np.bincount(step[span >= 2], minlength=L)
        shape = ((w if fwd else w[::-1]) <= 64) & (nn <= 128) & (nf <= 192)
        slot, over = np.zeros(src.shape[0], bool), 0
        for k in range((L + 7) // 8):
            m = (step // 8 == k) & shape[step] & (span > 4) & (nstep <= 8 * k - 12)
            u = np.unique(nb[m])
            over += len(u) > 512
            slot |= m & np.isin(nb, u[:512])
        gathered = np.bincount(step[(span > 4) & ~slot], minlength=L)
        out["t" if fwd else "b"] = (over, int(((gathered > 64) & shape).sum()),
                                    int((shape & (gathered > 0) & (gathered <= 64)).sum()))
    return out


def test_batch_long_edge_blocks(P):
    """A layered DAG whose long edges overflow the per-block LDS lists (more
    than 512 distinct neighbours in a block of 8 levels), with levels that
    gather more than 64 values from the workspace (general path) and levels
    that mix gathered and LDS-served records, in both directions: the batch
    with and without label sums and the one-placement sweep, against the
    oracle for every placement."""
    g = W.long_edge_dag(np.random.default_rng(5))
    cov = _long_edge_coverage(g)
    say(f"long-edge blocks V={g.n_nodes} E={g.n_edges} coverage={cov}")
    for d in ("t", "b"):
        assert all(x > 0 for x in cov[d]), cov   # every case present
    rng = np.random.default_rng(6)
    n_place = 7
    pl = rng.integers(0, g.n_labels, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 0] = g.placement
    pl[:, -1] = 0
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_batch(P, G, pl, g)
    check_batch(g, pl, out, range(n_place))
    for p in (1, 4):   # one placement per chain reads the same lists
        tl, bl, m = G.tb_levels(dev(pl[:, p].copy(), torch.int32))
        torch.cuda.synchronize()
        etl, ebl, em = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost,
                                        pl[:, p].copy())
        assert (tl.cpu().numpy() == etl).all() and (bl.cpu().numpy() == ebl).all(), p
        assert int(m.item()) == em, p
    G.close()
    _tb_batch_case(P, g, pl)


@pytest.mark.parametrize("shift", [18, 20])
def test_batch_large_weights_successor_links(P, shift):
    """Weights scaled by 2^shift on config 0 (4 labels: 2 label bits; 2050
    nodes: 12 successor bits). 2^18 keeps the weight bound below 2^48, where
    the successor links ride in the packed b values; 2^20 puts it between 2^48
    and 2^50, where the values are still packed but the links need their own
    array. Both give the oracle's results, paths included."""
    import types
    g0 = cfg(0)
    f = 1 << shift
    g = types.SimpleNamespace(n_nodes=g0.n_nodes, src=g0.src, dst=g0.dst, comp=g0.comp * f,
                              edge_cost=g0.edge_cost * f, mem=g0.mem, n_labels=g0.n_labels,
                              capacity=g0.capacity, placement=g0.placement)
    wb = int(g.comp.sum()) + int(g.edge_cost.sum())
    assert (wb < 2 ** 48) == (shift == 18) and wb < 2 ** 50
    say(f"batch config0 weights x 2^{shift}")
    rng = np.random.default_rng(300 + shift)
    pl = rng.integers(0, g.n_labels, (g.n_nodes, 11)).astype(np.int32)
    pl[:, 0] = g.placement
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_batch(P, G, pl, g)
    check_batch(g, pl, out, range(11))
    G.close()


def test_batch_wide_resnet(P):
    """The batched pair sweep on the largest graph (1.05M nodes, 100,270
    levels, about 90 levels of 9,500 nodes: the general level path and the
    early folds of wide levels on every chain; its weights leave no room for
    the successor links in the b values, so they take their own array),
    element by element against the oracle."""
    g = cfg(3)
    say(f"batch config3 V={g.n_nodes} P=3")
    rng = np.random.default_rng(33)
    pl = np.stack([g.placement, rng.integers(0, g.n_labels, g.n_nodes),
                   np.zeros(g.n_nodes)], axis=1).astype(np.int32)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_batch(P, G, pl, g)
    check_batch(g, pl, out, range(3))
    G.close()


def test_batch_small_graphs(P):
    say("batch on small random DAGs")
    rng = np.random.default_rng(4242)
    for t in range(40):
        n = int(rng.integers(0, 30)) if t > 1 else t
        g = W.random_dag(rng, n, p_edge=0.3, max_weight=3, n_labels=3)
        n_place = int(rng.integers(1, 6))
        pl = rng.integers(0, 3, (n, n_place)).astype(np.int32)
        G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
        out = run_batch(P, G, pl, g)
        check_batch(g, pl, out, range(n_place))
        G.close()


def level_shapes(seed):
    """A level schedule that drives every path of the batched sweep: a chain,
    a 100-wide level read back at spans 1..3, levels of exactly 64 and 65
    nodes, a 36-node level with about 300 in-edges, a 10-node level with about
    300 out-edges, a node with up to 64 predecessors, and a chain tail."""
    sched = [(1, 1)] + [(1, 2)] * 5
    sched += [(100, 3)]
    sched += [(3, 6), (64, 4), (65, 3)]
    sched += [(36, 16)]
    sched += [(10, 2), (300, 1)]
    sched += [(2, 4), (1, 3), (50, 5), (1, 64), (20, 3)]
    sched += [(1, 2)] * 7
    widths, fan = zip(*sched)
    return W.layered_dag(np.random.default_rng(seed), widths, fan, max_span=4, n_labels=4)


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_batch_level_shapes(P, seed):
    g = level_shapes(seed)
    say(f"batch level shapes seed={seed} V={g.n_nodes} E={g.n_edges}")
    rng = np.random.default_rng(seed)
    n_place = 7
    pl = rng.integers(0, g.n_labels, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 0] = 0
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_batch(P, G, pl, g)
    check_batch(g, pl, out, range(n_place))
    G.close()


def test_batch_tie_rows_next_to_chains(P):
    """Placements whose critical set is far larger than the number of levels
    (zero node weights and one label: every node is critical) interleaved with
    placements whose critical set is a single path. The path rows are exactly
    as long as the number of levels, so a row that wrote past its end would
    corrupt its neighbour's path."""
    rng = np.random.default_rng(31)
    base = W.layered_dag(rng, [1] + [24] * 20 + [1], [1] + [3] * 20 + [24], max_span=3,
                         n_labels=4)
    g = W.SynthGraph("ties", base.n_nodes, base.src, base.dst,
                     np.zeros(base.n_nodes, np.int64), base.edge_cost + 1, base.mem,
                     base.placement, 4, base.capacity, {})
    say(f"batch tie rows V={g.n_nodes} E={g.n_edges}")
    n_place = 12
    pl = rng.integers(0, 4, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 0::2] = 0
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = run_batch(P, G, pl, g)
    assert (out["path_len"][0::2] <= 22).all()
    assert out["is_critical"][:, 0::2].all()
    check_batch(g, pl, out, range(n_place))
    G.close()


@pytest.mark.parametrize("seed", [21, 22])
def test_batch_any_int32_labels(P, seed):
    """Without label sums the batch takes any int32 labels (only equality
    matters), so values are kept as full {value, label} pairs."""
    g = level_shapes(seed)
    say(f"batch int32 labels seed={seed}")
    rng = np.random.default_rng(seed)
    n_place = 5
    pool = np.array([-2**31, -7, 0, 3, 2**20 + 1, 2**31 - 1], np.int64)
    pl = pool[rng.integers(0, pool.size, (g.n_nodes, n_place))].astype(np.int32)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = G.evaluate_batch(dev(pl, torch.int32), 0, labels=False)
    torch.cuda.synchronize()
    out = {k: v.cpu().numpy() for k, v in out.items()}
    for p in range(n_place):
        lab = pl[:, p].copy()
        tl, bl, m = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab)
        crit, path = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab,
                                          tl, bl, m)
        assert (out["tl"][:, p] == tl).all(), p
        assert (out["bl"][:, p] == bl).all(), p
        assert out["makespan"][p] == m, p
        assert (out["is_critical"][:, p] == crit).all(), p
        assert (out["path"][p, : out["path_len"][p]] == path).all(), p
    G.close()


@pytest.mark.parametrize("K", [3000, 65536, 70000])
def test_batch_many_labels(P, K):
    """Label sums with many labels: 3,000 labels keep packed keys but sum by
    global atomics (more than the LDS bins hold); 65,536 labels are the most
    the 16-bit label layout holds (labels up to 65,535 must come back whole,
    not as negative 16-bit values); 70,000 labels no longer pack into 16 bits,
    so the batch keeps {value, label} pairs and 32-bit labels."""
    say(f"batch with K={K} labels")
    rng = np.random.default_rng(K)
    g = W.random_dag(rng, 900, p_edge=0.01, max_weight=9, n_labels=1)
    n_place = 5
    pl = rng.integers(0, K, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 1] = rng.integers(0, 3, g.n_nodes)      # a few labels in use, many idle
    pl[:, 2] = K - 1 - rng.integers(0, 3, g.n_nodes)   # the top labels
    cap = rng.integers(0, 2000, K).astype(np.int64)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    out = G.evaluate_batch(dev(pl, torch.int32), K, dev(cap, torch.int64))
    torch.cuda.synchronize()
    out = {k: v.cpu().numpy() for k, v in out.items()}
    G.close()
    for p in range(n_place):
        exp = oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem,
                              pl[:, p].copy(), K, cap)
        assert (out["tl"][:, p] == exp["tl"]).all(), p
        assert (out["bl"][:, p] == exp["bl"]).all(), p
        assert out["makespan"][p] == exp["makespan"], p
        assert (out["is_critical"][:, p] == exp["is_critical"]).all(), p
        assert (out["path"][p, : out["path_len"][p]] == exp["path"]).all(), p
        assert (out["label_mem"][p] == exp["label_mem"]).all(), p
        assert (out["overflow"][p] == exp["overflow"]).all(), p


def test_labels_checked_before_16_bit_storage(P):
    """The batch with label sums stores labels as 16 bits; a label that is
    out of range only in its upper bits (K + 3 with K = 2^16, which 16 bits
    would read as 3) is still rejected, by the placements path and by the
    moves path, and the handle stays usable."""
    say("labels checked before 16-bit storage")
    rng = np.random.default_rng(77)
    g = W.random_dag(rng, 300, p_edge=0.02, max_weight=9, n_labels=1)
    K = 1 << 16
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    pl = rng.integers(0, 4, (g.n_nodes, 4)).astype(np.int32)
    bad = pl.copy()
    bad[7, 2] = K + 3
    with pytest.raises(P.PardnnError) as e:
        G.evaluate_batch(dev(bad, torch.int32), K)
    assert e.value.status == P.E_INVAL
    base = pl[:, 0].copy()
    ptr = np.array([0, 1, 2, 2], np.int64)
    node = np.array([5, 9], np.int32)
    with pytest.raises(P.PardnnError) as e:
        G.evaluate_moves(dev(base, torch.int32), dev(ptr, torch.int64), dev(node, torch.int32),
                         dev(np.array([1, K + 3], np.int32), torch.int32), K)
    assert e.value.status == P.E_INVAL
    # the same calls with the labels in range match the oracle
    out = G.evaluate_batch(dev(pl, torch.int32), K)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    for p in range(4):
        exp = oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem,
                              pl[:, p].copy(), K, None)
        assert (got["tl"][:, p] == exp["tl"]).all(), p
        assert (got["label_mem"][p] == exp["label_mem"]).all(), p
    G.close()


def test_evaluate_moves_without_values(P):
    """tl / bl may be left out: every other output is unchanged."""
    g = cfg(1)
    say("evaluate_moves without tl / bl")
    sched = W.config4_moves(g, n_place=37)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    margs = (dev(sched.base, torch.int32), dev(sched.ptr, torch.int64),
             dev(sched.node, torch.int32), dev(sched.label, torch.int32))
    cap = dev(g.capacity, torch.int64)
    full = G.evaluate_moves(*margs, g.n_labels, cap)
    lean = G.evaluate_moves(*margs, g.n_labels, cap, values=False)
    torch.cuda.synchronize()
    assert "tl" not in lean and "bl" not in lean
    for k in ("makespan", "is_critical", "path_len", "label_mem", "overflow"):
        assert torch.equal(full[k], lean[k]), k
    for p in range(37):
        n = int(full["path_len"][p])
        assert torch.equal(full["path"][p, :n], lean["path"][p, :n]), p
    G.close()


def test_evaluate_moves_small(P):
    """The fused moves entry point equals build_placements + evaluate_batch
    and the oracle, with repeated nodes, an empty step and an odd count."""
    g = cfg(0)
    say("evaluate_moves small")
    sched = W.config4_moves(g, n_place=53, frac=0.05, seed=5)
    node = sched.node.copy()
    node[sched.ptr[7] + 2] = node[sched.ptr[7]]
    ptr = sched.ptr.copy()
    ptr[10] = ptr[9]
    sched2 = W.MoveSchedule(sched.base, ptr, node, sched.label, sched.n_labels)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    args = (dev(sched2.base, torch.int32), dev(ptr, torch.int64), dev(node, torch.int32),
            dev(sched2.label, torch.int32))
    out = G.evaluate_moves(*args, g.n_labels, dev(g.capacity, torch.int64))
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    pl = W.materialize_placements(sched2).T.copy()
    check_batch(g, pl, got, range(53))
    ref = run_batch(P, G, pl, g)
    for k in ref:
        assert (ref[k] == got[k]).all(), k
    # no moves at all: every placement equals the base, label array may be empty
    zero_ptr = dev(np.zeros(4, np.int64), torch.int64)
    empty = torch.empty(0, dtype=torch.int32, device="cuda")
    out0 = G.evaluate_moves(args[0], zero_ptr, empty, empty, g.n_labels)
    torch.cuda.synchronize()
    g0 = {k: v.cpu().numpy() for k, v in out0.items()}
    check_batch(g, np.repeat(sched2.base[:, None], 3, axis=1), g0, range(3))
    with pytest.raises(P.PardnnError) as e:
        bad = node.copy()
        bad[3] = g.n_nodes + 7
        G.evaluate_moves(args[0], args[1], dev(bad, torch.int32), args[3], g.n_labels)
    assert e.value.status == P.E_INVAL
    with pytest.raises(P.PardnnError) as e:
        bad = node.copy()
        bad[-1] = -2
        G.evaluate_moves(args[0], args[1], dev(bad, torch.int32), args[3], g.n_labels)
    assert e.value.status == P.E_INVAL
    # still usable after the rejected calls
    out2 = G.evaluate_moves(*args, g.n_labels, dev(g.capacity, torch.int64))
    torch.cuda.synchronize()
    for k in ref:
        assert (ref[k] == out2[k].cpu().numpy()).all(), k
    G.close()


@pytest.mark.parametrize("n_moves,n_place,width", [(3584, 64, 256), (3585, 63, 256),
                                                   (6400, 64, 256), (6400, 63, 255)])
def test_evaluate_moves_label_build_forms(P, n_moves, n_place, width):
    """The labels built from the moves take one of three forms: one lane per
    node with the moves of a 256-node workgroup staged in LDS (up to 3,584
    entries), the same walk reading the moves from global memory (a workgroup
    with more), and one wave per 64-node tile (more than 11 moves per node on
    average). Two levels of 256 nodes, every move on a source, so the first
    workgroup holds all of them: 3,584 moves fit, 3,585 do not, and 6,400 on
    512 nodes exceed the average (with 511 nodes, the tile form's last node
    has no neighbour to share its store with). Each equals build +
    evaluate_batch and the oracle."""
    say(f"evaluate_moves label build forms: {n_moves} moves, {n_place} placements, {width}")
    rng = np.random.default_rng(4242 + n_moves)
    g = W.layered_dag(rng, [256, width], [0, 3], n_labels=4)
    sources = np.setdiff1d(np.arange(g.n_nodes), g.dst).astype(np.int32)
    assert sources.shape[0] == 256
    cuts = np.sort(rng.integers(0, n_moves + 1, n_place - 1))
    ptr = np.concatenate([[0], cuts, [n_moves]]).astype(np.int64)
    node = rng.choice(sources, n_moves).astype(np.int32)      # repeats within a step too
    label = rng.integers(0, g.n_labels, n_moves).astype(np.int32)
    sched = W.MoveSchedule(g.placement.copy(), ptr, node, label, g.n_labels)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    args = (dev(sched.base, torch.int32), dev(ptr, torch.int64), dev(node, torch.int32),
            dev(label, torch.int32))
    out = G.evaluate_moves(*args, g.n_labels, dev(g.capacity, torch.int64))
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    pl = W.materialize_placements(sched).T.copy()
    check_batch(g, pl, got, sorted({0, 1, n_place // 2, n_place - 2, n_place - 1}))
    ref = run_batch(P, G, pl, g)
    for k in ref:
        assert (ref[k] == got[k]).all(), k
    G.close()


def test_step_ptr_checks_and_deferred_errors(P):
    """step_ptr is checked against the number of moves on the device (no host
    read-back): one that does not start at 0, decreases or does not end at
    n_moves gives E_INVAL. With deferred errors the calls only enqueue and
    pardnn_take_errors reports what they found, once; valid calls give the
    same results in both modes."""
    say("step_ptr checks and deferred errors")
    g = cfg(0)
    sched = W.config4_moves(g, n_place=20, frac=0.05, seed=5)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    base, ptr = dev(sched.base, torch.int32), dev(sched.ptr, torch.int64)
    node, lab = dev(sched.node, torch.int32), dev(sched.label, torch.int32)
    cap = dev(g.capacity, torch.int64)
    ref = {k: v.cpu().numpy() for k, v in
           G.evaluate_moves(base, ptr, node, lab, g.n_labels, cap).items()}
    check_batch(g, W.materialize_placements(sched).T.copy(), ref, range(20))
    bads = []
    b = sched.ptr.copy(); b[-1] -= 1; bads.append(b)          # ends before n_moves
    b = sched.ptr.copy(); b[0] = 1; bads.append(b)            # does not start at 0
    b = sched.ptr.copy(); b[5], b[6] = b[6] + 1, b[5]; bads.append(b)   # decreases
    for b in bads:
        for call in (lambda: G.evaluate_moves(base, dev(b, torch.int64), node, lab, g.n_labels,
                                              cap),
                     lambda: G.build_placements(base, dev(b, torch.int64), node, lab)):
            with pytest.raises(P.PardnnError) as e:
                call()
            assert e.value.status == P.E_INVAL and "step_ptr" in str(e.value)
    # a shorter n_moves than step_ptr ends at
    with pytest.raises(P.PardnnError) as e:
        o, stride = G._outputs(20, g.n_labels, True, True, True)
        P.pardnn_evaluate_moves(G.handle, base, 20, ptr, node, lab, g.n_labels, cap, o["tl"],
                                o["bl"], o["makespan"], o["is_critical"], o["path"], stride,
                                o["path_len"], o["label_mem"], o["overflow"],
                                n_moves=node.numel() - 1)
    assert e.value.status == P.E_INVAL
    # deferred: the bad calls return at once, the take reports them once
    P.pardnn_set_deferred_errors(G.handle, True)
    bad_node = sched.node.copy()
    bad_node[2] = g.n_nodes + 3
    G.evaluate_moves(base, ptr, dev(bad_node, torch.int32), lab, g.n_labels, cap)
    G.build_placements(base, dev(bads[2], torch.int64), node, lab)
    out = G.evaluate_moves(base, ptr, node, lab, g.n_labels, cap)
    with pytest.raises(P.PardnnError) as e:
        P.pardnn_take_errors(G.handle)
    assert e.value.status == P.E_INVAL
    P.pardnn_take_errors(G.handle)   # cleared
    got = {k: v.cpu().numpy() for k, v in out.items()}
    for k in ref:
        assert (ref[k] == got[k]).all(), k
    bad_lab = dev(np.full(g.n_nodes, g.n_labels, np.int32), torch.int32)
    G.label_memory(bad_lab, g.n_labels, cap)
    with pytest.raises(P.PardnnError) as e:
        P.pardnn_take_errors(G.handle)
    assert e.value.status == P.E_INVAL
    P.pardnn_set_deferred_errors(G.handle, False)
    with pytest.raises(P.PardnnError) as e:
        G.label_memory(bad_lab, g.n_labels, cap)
    assert e.value.status == P.E_INVAL
    P.pardnn_take_errors(G.handle)   # not deferred: the call reported it itself
    G.close()


def test_c4_refinement_loop_full_size(P):
    """The 1000-placement refinement loop on the transformer graph, in the
    launch configuration the benchmark times (pardnn_evaluate_moves); sampled
    placements against the oracle, properties on all of them."""
    g = cfg(2)
    say(f"config4 full size V={g.n_nodes} P=1000")
    sched = W.config4_moves(g, n_place=1000)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    margs = (dev(sched.base, torch.int32), dev(sched.ptr, torch.int64),
             dev(sched.node, torch.int32), dev(sched.label, torch.int32))
    out = G.evaluate_moves(*margs, g.n_labels, dev(g.capacity, torch.int64))
    pl = G.build_placements(*margs)
    torch.cuda.synchronize()
    cols = [0, 1, 2, 499, 998, 999] + list(range(50, 1000, 97))
    exp_pl = W.materialize_placements(sched)  # [P][V]
    for p in cols:
        assert (pl[:, p].cpu().numpy() == exp_pl[p]).all(), p
    sub = {k: (v[:, cols] if v.dim() == 2 and v.shape[0] == g.n_nodes else
               v[cols]).cpu().numpy() for k, v in out.items()}
    check_batch(g, exp_pl[cols].T.copy(), sub, range(len(cols)))
    # properties on every placement, evaluated on the GPU in chunks
    M = out["makespan"]
    for c0 in range(0, 1000, 100):
        tl = out["tl"][:, c0:c0 + 100]
        bl = out["bl"][:, c0:c0 + 100]
        w = tl + bl
        assert bool((w <= M[c0:c0 + 100]).all())
        crit = out["is_critical"][:, c0:c0 + 100].bool()
        assert bool((crit == (w == M[c0:c0 + 100])).all())
    assert bool((out["path_len"] >= 1).all())
    total_mem = int(g.mem.sum())
    assert bool((out["label_mem"].sum(dim=1) == total_mem).all())
    G.close()


# Every placement of the refinement loop against the oracle, element by
# element: tl, bl, the critical flags and the path of each placement, its
# makespan, label sums and overflows. The outputs are copied back 100
# placements at a time; the oracle (C, called through ctypes, which releases
# the GIL) runs on host threads.
def _c4_oracle(g, sched, p):
    lab = W.materialize_placements(sched, p, 1)[0]
    return p, oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem, lab,
                              g.n_labels, g.capacity)


def test_c4_every_placement(P):
    g = cfg(2)
    say(f"config4 every placement element by element V={g.n_nodes} P=1000")
    sched = W.config4_moves(g, n_place=1000)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    margs = (dev(sched.base, torch.int32), dev(sched.ptr, torch.int64),
             dev(sched.node, torch.int32), dev(sched.label, torch.int32))
    out = G.evaluate_moves(*margs, g.n_labels, dev(g.capacity, torch.int64))
    torch.cuda.synchronize()
    small = {k: out[k].cpu().numpy() for k in ("makespan", "path", "path_len", "label_mem",
                                              "overflow")}
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        for c0 in range(0, 1000, 100):
            cols = range(c0, c0 + 100)
            res = ex.map(lambda p: _c4_oracle(g, sched, p), cols)
            tl = out["tl"][:, c0:c0 + 100].cpu().numpy()
            bl = out["bl"][:, c0:c0 + 100].cpu().numpy()
            cr = out["is_critical"][:, c0:c0 + 100].cpu().numpy()
            for p, e in res:
                j = p - c0
                assert (tl[:, j] == e["tl"]).all(), ("tl", p)
                assert (bl[:, j] == e["bl"]).all(), ("bl", p)
                assert (cr[:, j] == e["is_critical"]).all(), ("is_critical", p)
                assert small["makespan"][p] == e["makespan"], ("makespan", p)
                n = small["path_len"][p]
                assert n == len(e["path"]) and (small["path"][p, :n] == e["path"]).all(), p
                assert (small["label_mem"][p] == e["label_mem"]).all(), ("label_mem", p)
                assert (small["overflow"][p] == e["overflow"]).all(), ("overflow", p)
            say(f"config4 placements {c0}..{c0 + 99} equal")
    G.close()


# ------------------------------------------- batches without label sums --

def _tb_batch_case(P, g, pl):
    """pardnn_tb_levels_batch and pardnn_evaluate_batch without label sums on
    placements pl [V][P], against the oracle for every placement."""
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    n_place = pl.shape[1]
    d = dev(pl, torch.int32)
    tl = torch.empty((g.n_nodes, n_place), dtype=torch.int64, device="cuda")
    bl = torch.empty_like(tl)
    m = torch.empty(n_place, dtype=torch.int64, device="cuda")
    P.pardnn_tb_levels_batch(G.handle, n_place, d, tl, bl, m)
    full = G.evaluate_batch(d, 0)          # no label sums: path and flags still there
    torch.cuda.synchronize()
    tl, bl, m = tl.cpu().numpy(), bl.cpu().numpy(), m.cpu().numpy()
    full = {k: v.cpu().numpy() for k, v in full.items()}
    G.close()
    from concurrent.futures import ThreadPoolExecutor

    def one(p):
        lab = pl[:, p].copy()
        etl, ebl, em = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab)
        ecrit, epath = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab,
                                            etl, ebl, em)
        return p, etl, ebl, em, ecrit, epath

    with ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        for p, etl, ebl, em, ecrit, epath in ex.map(one, range(n_place)):
            assert (tl[:, p] == etl).all() and (bl[:, p] == ebl).all() and m[p] == em, p
            assert (full["tl"][:, p] == etl).all() and (full["bl"][:, p] == ebl).all(), p
            assert full["makespan"][p] == em, p
            assert (full["is_critical"][:, p] == ecrit).all(), p
            n = full["path_len"][p]
            assert n == len(epath) and (full["path"][p, :n] == epath).all(), p


@pytest.mark.parametrize("i,n_place", [(1, 64), (2, 64)])
def test_tb_levels_batch_labels_in_16_bits(P, i, n_place):
    """Labels in [0, 2^16) without label sums: the pair sweep, chosen on the
    device (labels drawn from the whole 16-bit range, plus the placement of
    the config and a single-label placement)."""
    g = cfg(i)
    say(f"tb_levels_batch config{i} P={n_place} labels < 2^16")
    rng = np.random.default_rng(640 + i)
    pl = rng.integers(0, 16, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 0] = g.placement
    pl[:, 1] = 0
    pl[:, 2] = rng.integers(0, 1 << 16, g.n_nodes)
    pl[:, 3] = (1 << 16) - 1
    _tb_batch_case(P, g, pl)


@pytest.mark.parametrize("i,n_place", [(1, 64), (2, 64)])
def test_tb_levels_batch_labels_beyond_16_bits(P, i, n_place):
    """One label outside [0, 2^16) anywhere in the batch sends every placement
    to the unpacked sweep; results do not depend on which sweep ran."""
    g = cfg(i)
    say(f"tb_levels_batch config{i} P={n_place} a label >= 2^16")
    rng = np.random.default_rng(650 + i)
    pl = rng.integers(0, 16, (g.n_nodes, n_place)).astype(np.int32)
    pl[:, 0] = g.placement
    pl[g.n_nodes // 3, n_place - 1] = 1 << 16
    pl[:, 5] = rng.choice(np.array([-7, 70000, 2 ** 31 - 1, 3], np.int32), g.n_nodes)
    _tb_batch_case(P, g, pl)


@pytest.mark.parametrize("hint", [0, 2])
def test_evaluate_moves_without_label_sums(P, hint):
    """The moves entry point without label sums takes the same device-side
    choice: labels outside 16 bits among the moves take the unpacked sweep,
    and so do labels past the caller's hint n_labels (hint 2 on this
    two-label graph: 1 label bit, room for the successor links in the b
    values; a moved label 5 breaks the hint)."""
    g = cfg(1)
    say(f"evaluate_moves without label sums, hint {hint}")
    sched = W.config4_moves(g, n_place=40)
    G = P.Graph(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    for wide in (0, 1 << 20, 5):
        label = sched.label.copy()
        if wide:
            label[len(label) // 2] = wide
        s2 = W.MoveSchedule(sched.base, sched.ptr, sched.node, label, sched.n_labels)
        out = G.evaluate_moves(dev(s2.base, torch.int32), dev(s2.ptr, torch.int64),
                               dev(s2.node, torch.int32), dev(label, torch.int32), hint,
                               labels=False)
        torch.cuda.synchronize()
        got = {k: v.cpu().numpy() for k, v in out.items()}
        pl = W.materialize_placements(s2).T.copy()
        for p in range(40):
            lab = pl[:, p].copy()
            etl, ebl, em = oracle.tb_levels(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, lab)
            ecrit, epath = oracle.critical_path(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost,
                                                lab, etl, ebl, em)
            assert (got["tl"][:, p] == etl).all() and (got["bl"][:, p] == ebl).all(), p
            assert got["makespan"][p] == em and (got["is_critical"][:, p] == ecrit).all(), p
            n = got["path_len"][p]
            assert (got["path"][p, :n] == epath).all(), p
    G.close()


# ------------------------------------------- segmented single-placement sweeps --

@pytest.fixture
def wide_level(monkeypatch):
    """Sets the width above which a single-placement sweep computes a level
    grid-wide between chain segments (read by the library at every call)."""
    def set_(n):
        monkeypatch.setenv("PARDNN_WIDE_LEVEL", str(n))
    return set_


@pytest.mark.parametrize("thr", [1, 65, 300, 0])
@pytest.mark.parametrize("i", [0, 1, 2])
def test_single_wide_level_thresholds(P, wide_level, thr, i):
    """Every level wider than thr nodes computed grid-wide between chain
    segments (thr = 1: nearly every level; 0: none): results unchanged."""
    wide_level(thr)
    g = cfg(i)
    say(f"config{i} single, wide levels above {thr} nodes grid-wide")
    assert_same(gpu_single(P, g), oracle_single(g))


def test_single_wide_levels_wide_resnet(P, wide_level):
    """The Wide-ResNet-shaped graph (90 levels of about 10k nodes between long
    one-wide chains) with the default threshold and with 65."""
    g = cfg(3)
    exp = oracle_single(g)
    for thr in (512, 65):
        wide_level(thr)
        say(f"config3 single, wide levels above {thr} nodes grid-wide")
        assert_same(gpu_single(P, g), exp)


def test_single_wide_levels_random_shapes(P, wide_level):
    """Level shapes that drive every path of the chain (level_shapes) and
    random DAGs, with the grid-wide pass for every level above 2 nodes."""
    wide_level(2)
    say("segmented sweeps on level shapes and random DAGs")
    for seed in (11, 12, 13):
        g = level_shapes(seed)
        assert_same(gpu_single(P, g), oracle_single(g))
    rng = np.random.default_rng(2121)
    for t in range(30):
        g = W.random_dag(rng, int(rng.integers(1, 80)), p_edge=float(rng.uniform(0.02, 0.3)),
                         max_weight=int(rng.integers(0, 6)), n_labels=int(rng.integers(1, 4)))
        assert_same(gpu_single(P, g), oracle_single(g))
