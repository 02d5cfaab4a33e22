"""Seeded synthetic stand-ins for the DNN training graphs of the paper.

The paper partitions TensorFlow graphs of 10.6k-205k ops (Sec. 5, Table 3) that
are not available here, so these generators build DAGs of the same shape from
a fixed seed. They only produce INPUTS: node weights, edge costs, memory and a
placement. All randomness is numpy PCG64 with ``seed = SEED_BASE + config``.

Sampling rules shared by every config:

* log-uniform on [a, b] means ``floor(exp(U(ln a, ln b)))`` clipped to [a, b];
* op cost ``comp`` is int64 ns, log-uniform on [1, 1e4];
* op memory ``mem`` is int64 bytes, log-uniform on [4 KiB, 64 MiB];
* tensor bytes per edge are log-uniform on [1 KiB, 16 MiB] (config 2:
  log-normal, median 2 MiB, sigma 1.0, clipped to [1 KiB, 1 GiB]);
* the raw edge cost is ``ceil(bytes / 12)`` ns, i.e. ``(bytes + 11) // 12``.
  The evaluator, not the generator, zeroes it when both ends share a label;
* node ids are a seeded random permutation of the construction order and the
  edge list is shuffled, so no input is handed over in topological order.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 200808636
KIB, MIB, GIB = 1 << 10, 1 << 20, 1 << 30
# Memory capacity per label: 90 % of a 32 GiB device (the paper keeps a 10 %
# reserve, Sec. 4, on 32 GB V100s, Sec. 5.1).
CAPACITY_32G_90 = (9 * 32 * GIB) // 10


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _log_uniform(rng, lo, hi, n) -> np.ndarray:
    x = np.floor(np.exp(rng.uniform(np.log(lo), np.log(hi), n)))
    return np.clip(x, lo, hi).astype(np.int64)


def _bytes_to_cost(nbytes: np.ndarray) -> np.ndarray:
    return (np.asarray(nbytes, np.int64) + 11) // 12


@dataclass
class SynthGraph:
    """One weighted DAG plus one placement.

    ``src[e] -> dst[e]`` are int32 node ids; ``comp``/``mem`` are int64[V];
    ``edge_cost`` is the int64 transfer cost of each edge when its endpoints sit
    on different labels; ``placement`` is int32[V] in [0, n_labels).
    """

    name: str
    n_nodes: int
    src: np.ndarray
    dst: np.ndarray
    comp: np.ndarray
    edge_cost: np.ndarray
    mem: np.ndarray
    placement: np.ndarray
    n_labels: int
    capacity: np.ndarray
    meta: dict = field(default_factory=dict)

    @property
    def n_edges(self) -> int:
        return int(self.src.shape[0])


@dataclass
class MoveSchedule:
    """Placements 1..n_place as cumulative moves over a base placement.

    Placement p (0-based, p = 0..n_place-1) is ``base`` with the moves of steps
    0..p applied in order; step p's moves are ``node[ptr[p]:ptr[p+1]]`` ->
    ``label[ptr[p]:ptr[p+1]]`` (distinct nodes within a step).
    """

    base: np.ndarray
    ptr: np.ndarray
    node: np.ndarray
    label: np.ndarray
    n_labels: int

    @property
    def n_place(self) -> int:
        return int(self.ptr.shape[0] - 1)


def _finish(name, rng, n, src, dst, comp, nbytes, mem, label, n_labels, meta,
            permute=True, kinds=None):
    """Convert to arrays, renumber nodes by a random permutation, shuffle edges.
    ``kinds`` (optional) is (node_type int[n], ref_target int[n]) in the
    pre-permutation ids; it is renumbered with the nodes into meta."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    comp = np.asarray(comp, np.int64)
    mem = np.asarray(mem, np.int64)
    label = np.asarray(label, np.int32)
    cost = _bytes_to_cost(nbytes)
    if permute:
        perm = rng.permutation(n)
        src, dst = perm[src], perm[dst]
        inv_comp, inv_mem, inv_label = (np.empty_like(comp), np.empty_like(mem),
                                        np.empty_like(label))
        inv_comp[perm], inv_mem[perm], inv_label[perm] = comp, mem, label
        comp, mem, label = inv_comp, inv_mem, inv_label
        eperm = rng.permutation(src.shape[0])
        src, dst, cost = src[eperm], dst[eperm], cost[eperm]
        if kinds is not None:
            kt, kr = np.asarray(kinds[0], np.int32), np.asarray(kinds[1], np.int64)
            nt, nr = np.empty_like(kt), np.empty(n, np.int32)
            nt[perm] = kt
            nr[perm] = np.where(kr >= 0, perm[np.maximum(kr, 0)], -1)
            meta = dict(meta, node_type=nt, ref_target=nr)
    elif kinds is not None:
        meta = dict(meta, node_type=np.asarray(kinds[0], np.int32),
                    ref_target=np.asarray(kinds[1], np.int32))
    cap = np.full(n_labels, CAPACITY_32G_90, np.int64)
    return SynthGraph(name, int(n), src.astype(np.int32), dst.astype(np.int32), comp,
                      cost.astype(np.int64), mem, label, int(n_labels), cap, meta)


# --------------------------------------------------------------------------
# Config 0: tiny layered DAG, 64 levels x 32 ops, plus a source and a sink.
# --------------------------------------------------------------------------

def config0(seed: int = SEED_BASE + 0) -> SynthGraph:
    rng = _rng(seed)
    L, W, K = 64, 32, 4
    n = L * W + 2
    source, sink = 0, n - 1

    def op(lvl, j):
        return 1 + lvl * W + j

    src, dst, nbytes = [], [], []
    for j in range(W):
        src.append(source); dst.append(op(0, j)); nbytes.append(0)
    for lvl in range(1, L):
        for j in range(W):
            k = int(rng.integers(1, 4))
            for p in rng.choice(W, k, replace=False):
                src.append(op(lvl - 1, int(p))); dst.append(op(lvl, j)); nbytes.append(-1)
            if lvl >= 2 and rng.random() < 0.05:
                back = int(rng.integers(2, 9))
                src.append(op(max(0, lvl - back), int(rng.integers(W))))
                dst.append(op(lvl, j)); nbytes.append(-1)
    outdeg = np.bincount(np.asarray(src), minlength=n)
    for v in range(1, n - 1):
        if outdeg[v] == 0:
            src.append(v); dst.append(sink); nbytes.append(0)
    nbytes = np.asarray(nbytes, np.int64)
    data = nbytes < 0
    nbytes[data] = _log_uniform(rng, KIB, 16 * MIB, int(data.sum()))
    comp = _log_uniform(rng, 1, 10_000, n)
    mem = _log_uniform(rng, 4 * KIB, 64 * MIB, n)
    comp[[source, sink]] = 0
    mem[[source, sink]] = 0
    label = rng.integers(0, K, n).astype(np.int32)
    return _finish("tiny_layered_2k", rng, n, src, dst, comp, nbytes, mem, label, K,
                   {"levels_expected": L + 2})


# --------------------------------------------------------------------------
# Config 1: stacked-LSTM training graph, 8 layers x 256 timesteps.
# --------------------------------------------------------------------------

def config1(seed: int = SEED_BASE + 1) -> SynthGraph:
    """Forward cell (l, t): projection P <- h(l-1, t), h(l, t-1); four gates
    G0..G3 <- P; update U <- G0..G3, c(l, t-1). Every forward op f gets three
    backward ops: A_f (gradient accumulation), X_f (input gradient) and W_f
    (weight gradient), with A_f -> X_f, A_f -> W_f, f -> X_f; each forward edge
    a -> f adds the reversed X_f -> A_a, the activation a -> W_f and, for the
    nonlinear gate/update ops, a -> X_f. Layers 0-3 carry label 0 and layers
    4-7 label 1; backward ops follow their forward op."""
    rng = _rng(seed)
    LAY, T, K = 8, 256, 2
    labels = []
    fwd_edges = []  # (a, f) between forward ops (a may be an embedding op)

    def new(lbl):
        labels.append(lbl)
        return len(labels) - 1

    embed = [new(0) for _ in range(T)]
    cell_ops = {}
    fwd_list = []
    nonlinear = set()
    for t in range(T):
        for lay in range(LAY):
            lbl = lay // 4
            P = new(lbl)
            G = [new(lbl) for _ in range(4)]
            U = new(lbl)
            cell_ops[(lay, t)] = (P, G, U)
            fwd_list += [P] + G + [U]
            nonlinear.update(G + [U])
            below = embed[t] if lay == 0 else cell_ops[(lay - 1, t)][2]
            fwd_edges.append((below, P))
            if t > 0:
                prevU = cell_ops[(lay, t - 1)][2]
                fwd_edges.append((prevU, P))
                fwd_edges.append((prevU, U))
            for g in G:
                fwd_edges.append((P, g))
                fwd_edges.append((g, U))
    loss = new(1)
    embed_set = set(embed)
    A, X, Wg = {}, {}, {}
    for f in fwd_list:
        lbl = labels[f]
        A[f], X[f], Wg[f] = new(lbl), new(lbl), new(lbl)
    src, dst = [], []

    def edge(a, b):
        src.append(a); dst.append(b)

    for a, f in fwd_edges:
        edge(a, f)
        edge(a, Wg[f])
        if f in nonlinear:
            edge(a, X[f])
        if a not in embed_set:
            edge(X[f], A[a])
    for f in fwd_list:
        edge(A[f], X[f]); edge(A[f], Wg[f]); edge(f, X[f])
    for t in range(T):
        U = cell_ops[(LAY - 1, t)][2]
        edge(U, loss)
        edge(loss, A[U])
    n = len(labels)
    nbytes = _log_uniform(rng, KIB, 16 * MIB, len(src))
    comp = _log_uniform(rng, 1, 10_000, n)
    mem = _log_uniform(rng, 4 * KIB, 64 * MIB, n)
    return _finish("lstm_8x256_50k", rng, n, src, dst, comp, nbytes, mem,
                   np.asarray(labels, np.int32), K, {})


# --------------------------------------------------------------------------
# Config 2: transformer-shaped training graph, 48 blocks.
# --------------------------------------------------------------------------

def _block_template(rng, n_ops=2000):
    """Random layered forward block. Local node 0 is the block input (the
    previous block's output), local node n_ops-1 the residual add that ends the
    block. Internal ops take one predecessor from the level above plus
    Poisson(1.5) more from the three levels above (mean in-degree 2.5), and 5 %
    also read the block input (residual edges)."""
    depth = int(rng.integers(40, 61))
    n_int = n_ops - 2
    widths = rng.multinomial(n_int - depth, np.full(depth, 1.0 / depth)) + 1
    lvl_nodes = [[0]]
    nid = 1
    for w in widths:
        lvl_nodes.append(list(range(nid, nid + int(w))))
        nid += int(w)
    out = nid
    assert out == n_ops - 1
    edges = set()
    for i in range(1, depth + 1):
        for v in lvl_nodes[i]:
            prev = lvl_nodes[i - 1]
            edges.add((prev[int(rng.integers(len(prev)))], v))
            extra = min(int(rng.poisson(1.5)), 5)
            pool = [u for j in range(max(0, i - 3), i) for u in lvl_nodes[j]]
            for u in rng.choice(pool, min(extra, len(pool)), replace=False):
                edges.add((int(u), v))
            if rng.random() < 0.05:
                edges.add((0, v))
    has_out = {a for a, _ in edges}
    for i in range(1, depth):
        for v in lvl_nodes[i]:
            if v not in has_out:
                nxt = lvl_nodes[i + 1]
                edges.add((v, nxt[int(rng.integers(len(nxt)))]))
    for v in lvl_nodes[depth]:
        edges.add((v, out))
    edges.add((0, out))
    e = np.array(sorted(edges), np.int64)
    param = rng.random(n_ops) < 0.10
    param[0] = param[out] = False
    return e[:, 0], e[:, 1], param, depth


def config2(seed: int = SEED_BASE + 2) -> SynthGraph:
    """48 copies of one random attention/MLP block template chained through
    their residual outputs, a token source and parametric embedding in front,
    a loss behind. Backward: every forward op f gets a gradient accumulation
    A_f and a local backward D_f with A_f -> D_f, f -> D_f, and for each forward
    edge a -> f the reversed D_f -> A_a plus (half of them) the activation
    a -> D_f. Each parametric op has a variable source var_f -> f and an
    optimiser op opt_f <- var_f, D_f, clip, where clip is a global gradient-norm
    op fed by every D_f of a parametric op. Three consecutive blocks share a
    label (16 labels); 2 % of all ops are then moved to another label."""
    rng = _rng(seed)
    NB, K = 48, 16
    t_src, t_dst, t_param, depth = _block_template(rng)
    F = int(t_param.shape[0])
    # keep half of the input-activation edges, fixed by the template
    t_act = rng.random(t_src.shape[0]) < 0.5

    labels = []

    def alloc(count, lbl):
        start = len(labels)
        labels.extend([lbl] * count)
        return start

    S, D = [], []
    token = alloc(1, 0)
    var_embed = alloc(1, 0)
    embed = alloc(1, 0)
    S += [token, var_embed]; D += [embed, embed]
    param_D = [None]  # filled with D ids of parametric ops
    param_pairs = []  # (var id, D id, label)
    A_embed = alloc(1, 0)
    D_embed = alloc(1, 0)
    S += [A_embed, embed]; D += [D_embed, D_embed]
    param_pairs.append((var_embed, D_embed, 0))
    block_in, A_in = embed, A_embed
    for b in range(NB):
        lbl = b // 3
        base = alloc(F - 1, lbl)           # forward ops, local 1..F-1
        A_base = alloc(F - 1, lbl)
        D_base = alloc(F - 1, lbl)
        g = np.concatenate([[block_in], base + np.arange(F - 1)])
        gA = np.concatenate([[A_in], A_base + np.arange(F - 1)])
        gD = np.concatenate([[-1], D_base + np.arange(F - 1)])
        a, f = g[t_src], g[t_dst]
        S += a.tolist(); D += f.tolist()                      # forward
        S += gD[t_dst].tolist(); D += gA[t_src].tolist()      # reversed grads
        S += a[t_act].tolist(); D += gD[t_dst][t_act].tolist()  # activations
        S += gA[1:].tolist(); D += gD[1:].tolist()            # A_f -> D_f
        S += g[1:].tolist(); D += gD[1:].tolist()             # f -> D_f
        for loc in np.nonzero(t_param)[0]:
            var = alloc(1, lbl)
            S.append(var); D.append(int(g[loc]))
            param_pairs.append((var, int(gD[loc]), lbl))
        block_in, A_in = int(g[F - 1]), int(gA[F - 1])
    loss = alloc(1, K - 1)
    D_loss = alloc(1, K - 1)
    S += [block_in, loss, D_loss]; D += [loss, D_loss, A_in]
    clip = alloc(1, K - 1)
    opt_of = []   # (optimiser op, the variable it updates)
    for var, dd, lbl in param_pairs:
        opt = alloc(1, lbl)
        S += [dd, var, dd, clip]; D += [clip, opt, opt, opt]
        opt_of.append((opt, var))
    del param_D
    n = len(labels)
    # memory kinds (Sec. 3.2.1): variables are residual, the optimiser op that
    # updates a variable in place is a reference node to it, the rest normal
    node_type = np.zeros(n, np.int32)
    ref_target = np.full(n, -1, np.int64)
    for opt, var in opt_of:
        node_type[var] = 1
        node_type[opt] = 2
        ref_target[opt] = var
    label = np.asarray(labels, np.int32)
    moved = rng.choice(n, int(round(0.02 * n)), replace=False)
    label[moved] = (label[moved] + rng.integers(1, K, moved.shape[0])) % K
    ne = len(S)
    nbytes = np.exp(rng.normal(np.log(2 * MIB), 1.0, ne))
    nbytes = np.clip(np.floor(nbytes), KIB, GIB).astype(np.int64)
    comp = _log_uniform(rng, 1, 10_000, n)
    mem = _log_uniform(rng, 4 * KIB, 64 * MIB, n)
    return _finish("transformer_48blk_300k", rng, n, S, D, comp, nbytes, mem, label, K,
                   {"template_depth": depth, "template_ops": F},
                   kinds=(node_type, ref_target))


# --------------------------------------------------------------------------
# Config 3: wide-ResNet-shaped DAG, ~1M ops, ~4M edges.
# --------------------------------------------------------------------------

def _powerlaw_degrees(rng, n, exponent=2.1, dmax=64):
    d = np.arange(1, dmax + 1, dtype=np.float64)
    p = d ** (-exponent)
    p /= p.sum()
    return rng.choice(dmax, n, p=p) + 1


def config3(seed: int = SEED_BASE + 3) -> SynthGraph:
    """Level schedule: 91 one-wide chains (100k levels in total) separated by
    90 wide segments. A wide segment fans out 1 -> 32 -> 1024 -> 9,500 so that
    no structural fan-out exceeds 64, and the next chain starts at a node fed by
    64 ops of the wide level. Every node then draws a total out-degree from a
    power law P(d) ~ d^-2.1 on [1, 64] whose extra edges go to uniform nodes of
    the next 20k positions; long skip edges (span up to 200k positions) top
    the edge count up to ~4M. Labels are uniform over 16."""
    rng = _rng(seed)
    K = 16
    n_wide, wide_w, chain_total, min_chain = 90, 9_500, 100_000, 600
    n_chain = n_wide + 1
    chain_lens = rng.multinomial(chain_total - n_chain * min_chain,
                                 np.full(n_chain, 1.0 / n_chain)) + min_chain
    widths = []
    for i in range(n_chain):
        widths += [1] * int(chain_lens[i])
        if i < n_wide:
            widths += [32, 1024, wide_w]
    widths = np.asarray(widths, np.int64)
    n_lvls = widths.shape[0]
    lptr = np.concatenate([[0], np.cumsum(widths)])
    n = int(lptr[-1])
    lvl = np.repeat(np.arange(n_lvls), widths)
    v = np.arange(n, dtype=np.int64)
    # structural predecessor at the previous level
    has_prev = lvl >= 1
    vv = v[has_prev]
    lv = lvl[has_prev]
    j = vv - lptr[lv]
    pw = widths[lv - 1]
    s_src = [lptr[lv - 1] + (j % pw)]
    s_dst = [vv]
    # chain starts after a wide level read 64 ops of that level
    starts = np.nonzero((widths[1:] == 1) & (widths[:-1] > 1))[0] + 1
    for k in starts:
        pick = rng.choice(int(widths[k - 1]), 64, replace=False)
        pick = pick[pick != 0]  # local 0 is already the structural predecessor
        s_src.append(lptr[k - 1] + pick)
        s_dst.append(np.full(pick.shape[0], lptr[k], np.int64))
    src = np.concatenate(s_src)
    dst = np.concatenate(s_dst)
    # power-law total out-degree
    outdeg = np.bincount(src, minlength=n)
    want = _powerlaw_degrees(rng, n)
    extra = np.maximum(0, want - outdeg)
    lend = lptr[lvl + 1]
    room = n - lend
    extra[room <= 0] = 0
    u = np.repeat(v, extra)
    span = np.minimum(20_000, room[u])
    t = lend[u] + np.floor(rng.random(u.shape[0]) * span).astype(np.int64)
    src = np.concatenate([src, u])
    dst = np.concatenate([dst, t])
    # long skip edges up to ~4M, keeping every out-degree <= 64
    outdeg = np.bincount(src, minlength=n)
    n_skip = max(0, 4_000_000 - src.shape[0])
    cand = rng.integers(0, n, int(n_skip * 1.3))
    cand = cand[room[cand] > 0]
    order = np.argsort(cand, kind="stable")
    cs = cand[order]
    first = np.searchsorted(cs, cs, side="left")
    rank = np.empty_like(cand)
    rank[order] = np.arange(cs.shape[0]) - first
    ok = outdeg[cand] + rank < 64
    cand = cand[ok][:n_skip]
    span = np.minimum(200_000, room[cand])
    t = lend[cand] + np.floor(rng.random(cand.shape[0]) * span).astype(np.int64)
    src = np.concatenate([src, cand])
    dst = np.concatenate([dst, t])
    ne = src.shape[0]
    nbytes = _log_uniform(rng, KIB, 16 * MIB, ne)
    comp = _log_uniform(rng, 1, 10_000, n)
    mem = _log_uniform(rng, 4 * KIB, 64 * MIB, n)
    label = rng.integers(0, K, n).astype(np.int32)
    return _finish("wrn_1m", rng, n, src, dst, comp, nbytes, mem, label, K,
                   {"levels_expected": int(n_lvls), "wide_levels": n_wide,
                    "wide_width": wide_w, "chain_levels": int(chain_lens.sum())})


# --------------------------------------------------------------------------
# Config 4: refinement loop, successive placements of the config-2 graph.
# --------------------------------------------------------------------------

def config4_moves(graph: SynthGraph, n_place: int = 1000, frac: float = 0.01,
                  seed: int = SEED_BASE + 4) -> MoveSchedule:
    """Placement p moves a uniform sample of round(frac * V) distinct ops of
    placement p-1 (placement -1 is the graph's own) to a uniform *different*
    label; step p draws from PCG64(seed + p), so placements depend on the seed
    alone, never on any evaluation result."""
    n, K = graph.n_nodes, graph.n_labels
    m = int(round(frac * n))
    cur = graph.placement.copy()
    nodes, labels = [], []
    for p in range(n_place):
        r = _rng(seed + p)
        sel = r.choice(n, m, replace=False).astype(np.int64)
        new = ((cur[sel] + r.integers(1, K, m)) % K).astype(np.int32)
        cur[sel] = new
        nodes.append(sel.astype(np.int32))
        labels.append(new)
    ptr = np.arange(n_place + 1, dtype=np.int64) * m
    node = np.concatenate(nodes) if nodes else np.zeros(0, np.int32)
    label = np.concatenate(labels) if labels else np.zeros(0, np.int32)
    return MoveSchedule(graph.placement.copy(), ptr, node, label, K)


def materialize_placements(sched: MoveSchedule, first: int = 0, count: int | None = None):
    """Placements first..first+count-1 as an int32 [count][V] array."""
    n_place = sched.n_place
    count = n_place - first if count is None else count
    cur = sched.base.copy()
    out = np.empty((count, cur.shape[0]), np.int32)
    for p in range(first + count):
        a, b = sched.ptr[p], sched.ptr[p + 1]
        cur[sched.node[a:b]] = sched.label[a:b]
        if p >= first:
            out[p - first] = cur
    return out


def node_kinds(g: SynthGraph, seed: int = SEED_BASE + 100, p_res: float = 0.10,
               p_ref: float = 0.08):
    """Memory kinds of the nodes (Sec. 3.2.1): the graph's own when its
    generator records them, else a seeded draw -- a fraction p_res residual,
    p_ref reference nodes each mutating a uniform residual node, the rest
    normal. Returns (node_type int32[V], ref_target int32[V])."""
    if "node_type" in g.meta:
        return g.meta["node_type"], g.meta["ref_target"]
    rng = _rng(seed)
    n = g.n_nodes
    u = rng.random(n)
    node_type = np.where(u < p_res, 1, np.where(u < p_res + p_ref, 2, 0)).astype(np.int32)
    res = np.nonzero(node_type == 1)[0]
    ref_target = np.full(n, -1, np.int32)
    refs = np.nonzero(node_type == 2)[0]
    if res.size:
        ref_target[refs] = res[rng.integers(0, res.size, refs.size)]
    else:
        node_type[refs] = 0
    return node_type, ref_target


def make_config(i: int, seed: int | None = None) -> SynthGraph:
    """Configs 0-3 (config 4 is config 2 plus ``config4_moves``)."""
    fns = [config0, config1, config2, config3]
    if not 0 <= i < len(fns):
        raise ValueError(f"no graph config {i}")
    return fns[i](SEED_BASE + i if seed is None else seed)


# --------------------------------------------------------------------------
# Small random DAGs for exhaustive checks.
# --------------------------------------------------------------------------

def random_dag(rng: np.random.Generator, n: int, p_edge: float = 0.3,
               max_weight: int = 3, n_labels: int = 3, p_multi: float = 0.1,
               shuffle: bool = True) -> SynthGraph:
    """Random DAG on n nodes: a random topological order, each forward pair
    joined with probability p_edge, some edges doubled (multi-edges). Small
    integer weights in [0, max_weight] force ties."""
    topo = rng.permutation(n) if shuffle else np.arange(n)
    src, dst = [], []
    for i in range(n):
        for j in range(i + 1, n):
            if rng.random() < p_edge:
                src.append(int(topo[i])); dst.append(int(topo[j]))
                if rng.random() < p_multi:
                    src.append(int(topo[i])); dst.append(int(topo[j]))
    ne = len(src)
    comp = rng.integers(0, max_weight + 1, n).astype(np.int64)
    cost = rng.integers(0, max_weight + 1, ne).astype(np.int64)
    mem = rng.integers(0, 100, n).astype(np.int64)
    label = rng.integers(0, max(1, n_labels), n).astype(np.int32)
    return SynthGraph("random_dag", n, np.asarray(src, np.int32), np.asarray(dst, np.int32),
                      comp, cost, mem, label, max(1, n_labels),
                      np.full(max(1, n_labels), 150, np.int64), {})


def long_edge_dag(rng: np.random.Generator, levels: int = 80, width: int = 40,
                  n_sources: int = 600, n_long: int = 3, min_long_span: int = 20,
                  mid_levels=None, n_labels: int = 4) -> SynthGraph:
    """A layered DAG rich in long edges: a first level of ``n_sources`` nodes,
    then ``levels`` levels of ``width`` nodes. Every node past the first level
    has one in-edge from the level before it (which fixes its level) and
    ``n_long`` in-edges from random nodes at least ``min_long_span`` levels
    back; a level in ``mid_levels`` (level -> count) instead gives each node
    that many in-edges of span 5 to 11. Small weights force ties."""
    if mid_levels is None:
        mid_levels = {30: 2, 31: 2, 45: 1, 60: 1}
    ids = [np.arange(n_sources)]
    nxt = n_sources
    for _ in range(levels):
        ids.append(np.arange(nxt, nxt + width))
        nxt += width
    n = nxt
    src, dst = [], []
    for lv in range(1, levels + 1):
        for v in ids[lv]:
            src.append(int(rng.choice(ids[lv - 1]))); dst.append(int(v))
            if lv in mid_levels:
                for _ in range(mid_levels[lv]):
                    span = int(rng.integers(5, 12))
                    if lv - span >= 0:
                        src.append(int(rng.choice(ids[lv - span]))); dst.append(int(v))
            elif lv - min_long_span >= 0:
                pool = np.concatenate(ids[:lv - min_long_span + 1])
                for u in rng.choice(pool, n_long, replace=False):
                    src.append(int(u)); dst.append(int(v))
    perm = rng.permutation(n)            # ids in no particular order
    src = perm[np.asarray(src, np.int64)].astype(np.int32)
    dst = perm[np.asarray(dst, np.int64)].astype(np.int32)
    ne = src.shape[0]
    comp = rng.integers(1, 10, n).astype(np.int64)
    cost = rng.integers(0, 10, ne).astype(np.int64)
    mem = rng.integers(0, 100, n).astype(np.int64)
    label = rng.integers(0, n_labels, n).astype(np.int32)
    return SynthGraph("long_edge_dag", n, src, dst, comp, cost, mem, label, n_labels,
                      np.full(n_labels, 5_000, np.int64), {})


def chain_graph(rng: np.random.Generator, n: int, n_labels: int = 2) -> SynthGraph:
    """The path 0 -> 1 -> ... -> n-1 with random weights and labels."""
    src = np.arange(max(n - 1, 0), dtype=np.int32)
    dst = src + 1
    comp = rng.integers(0, 1000, n).astype(np.int64)
    cost = rng.integers(0, 1000, max(n - 1, 0)).astype(np.int64)
    mem = rng.integers(0, 1000, n).astype(np.int64)
    label = rng.integers(0, n_labels, n).astype(np.int32)
    return SynthGraph("chain", n, src, dst, comp, cost, mem, label, n_labels,
                      np.full(n_labels, 10_000, np.int64), {})


def layered_dag(rng: np.random.Generator, widths, fan_in, max_span: int = 4,
                max_weight: int = 50, n_labels: int = 4) -> SynthGraph:
    """DAG built level by level: level k has widths[k] nodes; each node of a
    level k >= 1 draws 1..fan_in[k] distinct predecessors, the first from
    level k - 1 (so its level is exactly k) and the others from levels
    k - 1 - U{0..max_span-1} (clamped at 0). Shapes the test cases need --
    levels of exactly 64 / 65 nodes, wide levels read back at short spans,
    levels with hundreds of edges on few nodes -- are set by the schedule.
    Ids are permuted and edges shuffled."""
    widths = [int(w) for w in widths]
    lptr = np.concatenate([[0], np.cumsum(widths)]).astype(np.int64)
    n = int(lptr[-1])
    src, dst = [], []
    for k in range(1, len(widths)):
        for v in range(int(lptr[k]), int(lptr[k + 1])):
            want = int(rng.integers(1, int(fan_in[k]) + 1))
            preds = {int(rng.integers(lptr[k - 1], lptr[k]))}
            tries = 0
            while len(preds) < want and tries < 4 * want:
                kk = max(0, k - 1 - int(rng.integers(0, max_span)))
                preds.add(int(rng.integers(lptr[kk], lptr[kk + 1])))
                tries += 1
            for u in preds:
                src.append(u)
                dst.append(v)
    perm = rng.permutation(n).astype(np.int64)
    src = perm[np.asarray(src, np.int64)].astype(np.int32)
    dst = perm[np.asarray(dst, np.int64)].astype(np.int32)
    order = rng.permutation(src.shape[0])
    src, dst = src[order], dst[order]
    ne = src.shape[0]
    comp = rng.integers(0, max_weight + 1, n).astype(np.int64)
    cost = rng.integers(0, max_weight + 1, ne).astype(np.int64)
    mem = rng.integers(0, 1000, n).astype(np.int64)
    label = rng.integers(0, n_labels, n).astype(np.int32)
    return SynthGraph("layered", n, src, dst, comp, cost, mem, label, n_labels,
                      np.full(n_labels, 50_000, np.int64), {"levels": len(widths)})


def path_clusters(rng, g: SynthGraph, max_extra: int = 4, p_odd: float = 0.5):
    """Cluster ids for the mapping stage's inputs: the nodes are covered by
    random paths of the DAG (from a random unassigned node, up to `max_extra`
    steps to random unassigned successors), one cluster per path; with
    probability p_odd two unrelated nodes are then put together (usually not a
    path); 0-2 further ids stay empty. Returns (cluster int64[V], n_clusters)."""
    n = g.n_nodes
    succ = [[] for _ in range(n)]
    for a, b in zip(g.src.tolist(), g.dst.tolist()):
        succ[a].append(b)
    cl = np.full(n, -1, np.int64)
    C = 0
    for v in rng.permutation(n).tolist():
        if cl[v] >= 0:
            continue
        cl[v] = C
        u = v
        for _ in range(int(rng.integers(0, max_extra + 1))):
            free = [b for b in succ[u] if cl[b] < 0]
            if not free:
                break
            u = free[int(rng.integers(0, len(free)))]
            cl[u] = C
        C += 1
    if n >= 4 and rng.random() < p_odd:
        a, b = rng.choice(n, 2, replace=False)
        cl[b] = cl[a]
    C += int(rng.integers(0, 3))
    return cl, C
