"""Exhaustive path enumeration on tiny DAGs (independent check of the oracle).

Nothing here runs a topological order or a dynamic programme: every quantity
is read off the full list of directed paths, straight from the definitions of
the paper's Table 2 (a path's length is the sum of comp over its nodes plus
the comm of its edges; comm is zero inside a label).
"""
from __future__ import annotations


def enumerate_paths(n, src, dst):
    """Every directed path as (nodes, edges); single nodes included."""
    out = [[] for _ in range(n)]
    for e in range(len(src)):
        out[int(src[e])].append(e)
    paths = []

    def walk(v, nodes, edges):
        paths.append((tuple(nodes), tuple(edges)))
        for e in out[v]:
            s = int(dst[e])
            nodes.append(s)
            edges.append(e)
            walk(s, nodes, edges)
            nodes.pop()
            edges.pop()

    for v in range(n):
        walk(v, [v], [])
    return paths


def brute_force(n, src, dst, comp, cost, label):
    """tl, bl, M, crit and the canonical path by enumerating all paths."""
    indeg = [0] * n
    outdeg = [0] * n
    for e in range(len(src)):
        indeg[int(dst[e])] += 1
        outdeg[int(src[e])] += 1

    def comm(e):
        return 0 if label[int(src[e])] == label[int(dst[e])] else int(cost[e])

    paths = enumerate_paths(n, src, dst)
    tl = [0] * n
    bl = [0] * n
    best = 0
    full = []
    for nodes, edges in paths:
        length = sum(int(comp[v]) for v in nodes) + sum(comm(e) for e in edges)
        first, last = nodes[0], nodes[-1]
        if indeg[first] == 0:
            tl[last] = max(tl[last], length - int(comp[last]))
        if outdeg[last] == 0:
            bl[first] = max(bl[first], length)
        if indeg[first] == 0 and outdeg[last] == 0:
            full.append((length, nodes))
            best = max(best, length)
    crit = [0] * n
    canon = None
    for length, nodes in full:
        if length == best:
            for v in nodes:
                crit[v] = 1
            if canon is None or nodes < canon:
                canon = nodes
    return tl, bl, best, crit, list(canon) if canon is not None else []


def hop_levels(n, src, dst):
    """Longest hop count from any source, over all paths."""
    level = [0] * n
    indeg = [0] * n
    for e in range(len(src)):
        indeg[int(dst[e])] += 1
    for nodes, _ in enumerate_paths(n, src, dst):
        if indeg[nodes[0]] == 0:
            level[nodes[-1]] = max(level[nodes[-1]], len(nodes) - 1)
    return level
