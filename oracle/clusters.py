"""Oracle for cluster criticality in the mapping stage (ParDNN, Sec. 3.1.2).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/``, the smoke check
and the CPU-baseline leg of ``bench.py`` may use it. It calls the sequential
oracle's ``tb_levels``; no code is shared with the HIP path.

Once slicing has produced linear clusters, the paper maps them to partitions
in order of criticality: the length of the longest source-to-sink path that
passes through a cluster, where communication between two nodes of the same
cluster costs nothing. Treating the cluster ids as labels, the weighted level
w(n) = tl(n) + bl(n) of a node is the longest path through n under exactly
that cost rule, so the criticality of cluster c is the largest w(n) over its
nodes.

Readings: a cluster without nodes gets criticality -1 and sorts after every
non-empty one; clusters of equal criticality keep ascending id order.
"""
from __future__ import annotations

import numpy as np

from . import tb_levels


def cluster_criticality(n_nodes, src, dst, comp, edge_cost, cluster, n_clusters):
    """(criticality int64[n_clusters], order int32[n_clusters]). Raises
    ValueError on a cluster id outside [0, n_clusters)."""
    cluster = np.asarray(cluster, np.int64)
    C = int(n_clusters)
    if C < 1 and n_nodes > 0:
        raise ValueError("n_clusters must be >= 1")
    if n_nodes and ((cluster < 0).any() or (cluster >= C).any()):
        raise ValueError("cluster id outside [0, n_clusters)")
    crit = [-1] * C
    if n_nodes:
        tl, bl, _ = tb_levels(n_nodes, src, dst, comp, edge_cost, cluster.astype(np.int32))
        for v in range(n_nodes):
            w = int(tl[v]) + int(bl[v])
            c = int(cluster[v])
            if w > crit[c]:
                crit[c] = w
    order = sorted(range(C), key=lambda c: (-crit[c], c))
    return np.array(crit, np.int64), np.array(order, np.int32)
