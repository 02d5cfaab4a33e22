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
