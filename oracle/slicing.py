"""Oracle for the primary clusters of graph slicing (ParDNN, Alg. 1, Sec. 3.1.1).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/``, the smoke check
and the CPU-baseline leg of ``bench.py`` may use it. It composes the
sequential oracle's own routines (``tb_levels``, ``critical_path``) on the
subgraph that remains after each round; no code is shared with the HIP path.

Alg. 1 takes K heaviest paths one after another: the weighted levels of the
remaining graph are recomputed, its heaviest path -- with fresh levels, a
critical path -- becomes primary cluster j, and the path's nodes and their
edges leave the graph. Readings: before any placement every edge carries its
communication cost (every node its own label); the heaviest path is the
canonical critical path (smallest-id start among the critical nodes without a
remaining predecessor, then the smallest-id tight successor); a round on an
empty graph yields an empty path and makespan 0.
"""
from __future__ import annotations

import numpy as np

from . import critical_path, tb_levels


def slice_primaries(n_nodes, src, dst, comp, edge_cost, K):
    """(primary int32[V], paths list of int32 arrays, makespan int64[K])."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    comp = np.asarray(comp, np.int64)
    edge_cost = np.asarray(edge_cost, np.int64)
    alive = np.ones(n_nodes, bool)
    primary = np.full(n_nodes, -1, np.int32)
    paths, makespans = [], []
    for j in range(K):
        ids = np.nonzero(alive)[0]            # ascending: ids keep their order
        if ids.size == 0:
            paths.append(np.zeros(0, np.int32))
            makespans.append(0)
            continue
        remap = np.full(n_nodes, -1, np.int64)
        remap[ids] = np.arange(ids.size)
        keep = alive[src] & alive[dst]
        s, d = remap[src[keep]], remap[dst[keep]]
        c, w = edge_cost[keep], comp[ids]
        label = np.arange(ids.size, dtype=np.int32)   # every edge pays its cost
        tl, bl, m = tb_levels(ids.size, s, d, w, c, label)
        _, path = critical_path(ids.size, s, d, w, c, label, tl, bl, m)
        p = ids[path].astype(np.int32)
        primary[p] = j
        alive[p] = False
        paths.append(p)
        makespans.append(int(m))
    return primary, paths, np.array(makespans, np.int64)


def slice_all(n_nodes, src, dst, comp, edge_cost, K):
    """Alg. 1 in full: the K primary clusters (fresh weighted levels before
    each), then the secondary clusters peeled with the weighted levels of the
    graph that remains after the K-th primary, never recomputed (Sec. 3.1.1:
    past K paths the levels are no longer refreshed, so a path found is heavy
    by those priorities but need not be critical).

    The secondary walk (find_heaviest_path on stale priorities): it starts at
    the remaining node without a remaining predecessor of largest priority
    w = tl + bl, steps to the remaining successor of largest w, and stops at a
    node with no remaining successor (a single node when the start has none);
    ties in w go to the smaller node id. The path's nodes and edges then leave
    the graph and the next walk starts.

    Returns (cluster int32[V]: j for the node's cluster, primaries 0..K-1 and
    secondaries K, K+1, ... in the order found; paths: one int32 array of
    original ids per cluster, in the same order)."""
    import heapq

    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    comp = np.asarray(comp, np.int64)
    edge_cost = np.asarray(edge_cost, np.int64)
    primary, paths, _ = slice_primaries(n_nodes, src, dst, comp, edge_cost, K)
    cluster = primary.copy()
    paths = list(paths)
    ids = np.nonzero(primary < 0)[0]        # ascending: ids keep their order
    R = int(ids.size)
    if R == 0:
        return cluster, paths
    remap = np.full(n_nodes, -1, np.int64)
    remap[ids] = np.arange(R)
    keep = (primary[src] < 0) & (primary[dst] < 0)
    s, d = remap[src[keep]], remap[dst[keep]]
    # the weighted levels of the remaining graph, every edge paying
    tl, bl, _ = tb_levels(R, s, d, comp[ids], edge_cost[keep], np.arange(R, dtype=np.int32))
    w = (tl + bl).tolist()
    succ = [[] for _ in range(R)]
    indeg = [0] * R
    for a, b in zip(s.tolist(), d.tolist()):
        succ[a].append(b)
        indeg[b] += 1
    removed = [False] * R
    sources = [(-w[v], v) for v in range(R) if indeg[v] == 0]
    heapq.heapify(sources)
    j = K
    while sources:
        _, start = heapq.heappop(sources)
        path = [start]
        removed[start] = True
        cur = start
        while True:
            best = -1
            for t in succ[cur]:
                if not removed[t] and (best < 0 or (w[t], -t) > (w[best], -best)):
                    best = t
            if best < 0:
                break
            path.append(best)
            removed[best] = True
            cur = best
        for u in path:                       # the path's edges leave the graph
            for t in succ[u]:
                indeg[t] -= 1
                if indeg[t] == 0 and not removed[t]:
                    heapq.heappush(sources, (-w[t], t))
        orig = ids[np.array(path, np.int64)].astype(np.int32)
        cluster[orig] = j
        paths.append(orig)
        j += 1
    return cluster, paths
