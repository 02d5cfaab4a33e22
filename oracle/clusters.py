"""Oracle for cluster criticality in the mapping stage (ParDNN, Sec. 3.1.2).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/``, the smoke check
and the CPU-baseline leg of ``bench.py`` may use it. It calls the sequential
oracle's ``tb_levels`` and ``levelize``; no code is shared with the HIP path.

Once slicing has produced linear clusters (paths), the paper maps them to
partitions in order of criticality: the length of the longest source-to-sink
path that runs along the whole cluster, where communication between two nodes
of the same cluster costs nothing. With the cluster ids as labels, the
weighted levels give every part of such a path: the longest way into the
cluster's first node is tl(first), the cluster itself costs the sum of its
computation weights (its internal edges are free), and the longest way out
after its last node is bl(last) - comp(last). So

    criticality(c) = tl(first) + sum of comp over c + bl(last) - comp(last).

Readings: the nodes of a cluster, taken in (hop level, id) order, must form a
path (an edge from each to the next); a cluster that does not -- or has no
node -- has no such path and gets -1, sorting after every linear one; clusters
of equal criticality keep ascending id order.
"""
from __future__ import annotations

import numpy as np

from . import levelize, tb_levels


def cluster_criticality(n_nodes, src, dst, comp, edge_cost, cluster, n_clusters):
    """(criticality int64[n_clusters], order int32[n_clusters]). Raises
    ValueError on a cluster id outside [0, n_clusters)."""
    cluster = np.asarray(cluster, np.int64)
    comp = np.asarray(comp, np.int64)
    C = int(n_clusters)
    if C < 1 and n_nodes > 0:
        raise ValueError("n_clusters must be >= 1")
    if n_nodes and ((cluster < 0).any() or (cluster >= C).any()):
        raise ValueError("cluster id outside [0, n_clusters)")
    crit = [-1] * C
    if n_nodes:
        tl, bl, _ = tb_levels(n_nodes, src, dst, comp, edge_cost, cluster.astype(np.int32))
        level = levelize(n_nodes, src, dst)[0]
        edges = set(zip(np.asarray(src).tolist(), np.asarray(dst).tolist()))
        members = [[] for _ in range(C)]
        for v in range(n_nodes):
            members[int(cluster[v])].append(v)
        for c in range(C):
            nodes = sorted(members[c], key=lambda v: (int(level[v]), v))
            if not nodes:
                continue
            if any((nodes[i], nodes[i + 1]) not in edges for i in range(len(nodes) - 1)):
                continue   # not a path: nothing runs along the whole cluster
            first, last = nodes[0], nodes[-1]
            crit[c] = (int(tl[first]) + sum(int(comp[v]) for v in nodes)
                       + int(bl[last]) - int(comp[last]))
    order = sorted(range(C), key=lambda c: (-crit[c], c))
    return np.array(crit, np.int64), np.array(order, np.int32)
