"""Oracle for the terms of level-aware load balancing (ParDNN, Eq. 2, Sec. 3.1.2).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/``, the smoke check
and the CPU-baseline leg of ``bench.py`` may use it. Plain numpy and Python
loops over the definitions; it calls the sequential oracle's ``levelize`` for
hop levels and shares no code with the HIP path.

In the mapping stage each secondary cluster sc goes to the partition that
minimises Eq. 2: the computation already placed on that partition whose top
level falls inside span(sc), plus the communication sc would then exchange
with the other partitions. Table 2 defines span(sc) in time: from the
expected finish of the last parent of the cluster's first node to the
expected start of the first child of its last node.

Readings (the paper leaves these open):

* The span is measured in time on the top levels ``tl`` the caller passes;
  the paper's "levels" in its Fenwick-tree remark are read as these top
  levels, so that Eq. 2, Table 2 and that remark agree.
* A finish time is tl + comp; without parents the span starts at 0, without
  children it ends at the makespan max(tl + comp). The bounds are inclusive.
* The first and last node of a cluster are its smallest and largest
  (hop level, id); for a path these are its two ends.
* Edges inside one cluster carry no communication; every other edge between
  the cluster and a node on partition k counts toward comm[k], parallel edges
  each once.
* Ties of Eq. 2 go to the partition with the most communication (the
  paper's rule), then to the smallest partition index. A cluster without
  nodes gets span [0, -1], zero rows and choice -1.
"""
from __future__ import annotations

import numpy as np

from . import levelize


def span_work(n_nodes, src, dst, comp, edge_cost, label, K, cluster, n_clusters, tl,
              clusters=None):
    """dict of span_lo, span_hi [C], work, comm [C][K], choice [C]; with
    ``clusters`` (ids) only those rows, in that order. ValueError on bad ids."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    comp = np.asarray(comp, np.int64)
    edge_cost = np.asarray(edge_cost, np.int64)
    label = np.asarray(label, np.int64)
    cluster = np.asarray(cluster, np.int64)
    tl = np.asarray(tl, np.int64)
    C = int(n_clusters)
    if K < 1 or C < 0:
        raise ValueError("K must be >= 1 and n_clusters >= 0")
    if n_nodes and ((label < -1).any() or (label >= K).any()):
        raise ValueError("label outside [-1, K)")
    if n_nodes and ((cluster < -1).any() or (cluster >= C).any()):
        raise ValueError("cluster outside [-1, n_clusters)")
    rows = list(range(C)) if clusters is None else [int(c) for c in clusters]

    level = levelize(n_nodes, src, dst)[0] if n_nodes else np.zeros(0, np.int32)
    preds = [[] for _ in range(n_nodes)]
    succs = [[] for _ in range(n_nodes)]
    for a, b in zip(src.tolist(), dst.tolist()):
        preds[b].append(a)
        succs[a].append(b)
    makespan = int((tl + comp).max()) if n_nodes else 0

    members = {c: [] for c in rows}
    for v in range(n_nodes):
        c = int(cluster[v])
        if c in members:
            members[c].append(v)

    R = len(rows)
    lo = np.zeros(R, np.int64)
    hi = np.full(R, -1, np.int64)
    work = np.zeros((R, K), np.int64)
    comm = np.zeros((R, K), np.int64)
    choice = np.full(R, -1, np.int32)
    for r, c in enumerate(rows):
        nodes = members[c]
        if not nodes:
            continue
        first = min(nodes, key=lambda v: (int(level[v]), v))
        last = max(nodes, key=lambda v: (int(level[v]), v))
        lo[r] = max([int(tl[p] + comp[p]) for p in preds[first]], default=0)
        hi[r] = min([int(tl[ch]) for ch in succs[last]], default=makespan)
        inside = (tl >= lo[r]) & (tl <= hi[r])
        for k in range(K):
            work[r, k] = int(comp[inside & (label == k)].sum())
        # edges between the cluster and mapped nodes outside it
        in_c = cluster == c
        out_e = in_c[src] & ~in_c[dst] & (label[dst] >= 0)    # cluster -> mapped node
        in_e = in_c[dst] & ~in_c[src] & (label[src] >= 0)     # mapped node -> cluster
        np.add.at(comm[r], label[dst[out_e]], edge_cost[out_e])
        np.add.at(comm[r], label[src[in_e]], edge_cost[in_e])
        total = int(comm[r].sum())
        cost = [int(work[r, k]) + total - int(comm[r, k]) for k in range(K)]
        choice[r] = min(range(K), key=lambda k: (cost[k], -int(comm[r, k]), k))
    return {"span_lo": lo, "span_hi": hi, "work": work, "comm": comm, "choice": choice}
