"""Sequential CPU oracle for placement-aware critical-path evaluation.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT. Only ``tests/``, the smoke check
in ``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import this
package. The HIP library never loads it and shares no code with it.

The arithmetic lives in ``pardnn_oracle.c`` (plain C, one thread); this module
only marshals numpy arrays through ctypes. Each wrapper names the definition it
follows in the paper (ParDNN, arXiv 2008.08636):

* ``levelize``      -- hop levels by Kahn's algorithm (Sec. 3.1.1: weighted
                        levels by a topological-order pass in O(V + E);
                        levels index the per-level work tables of Sec. 3.1.2).
* ``tb_levels``     -- tl, bl and the makespan (Table 2: tl, bl, w_lvl, CP).
* ``critical_path`` -- critical nodes and the canonical critical path
                        (Table 2: CP; Alg. 1 find_heaviest_path on fresh
                        weighted levels).
* ``label_memory``  -- per-label memory sums and overflow (Sec. 3.2, Memory
                        Heuristic II totals; Sec. 4, capacity).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")
SRC_PATH = os.path.join(HERE, "pardnn_oracle.c")

OK, E_INVAL, E_CYCLE, E_OVERFLOW, E_NOMEM = 0, -1, -2, -3, -4


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"oracle {what} failed with status {status}")
        self.status = status


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (single-threaded, -O3)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O3", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared",
             "-o", tmp, SRC_PATH])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def bind(path: str):
    """Load an oracle shared library from ``path`` and declare its signatures."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.orc_validate.argtypes = [i32, i64, P, P, P, P, P]
    lib.orc_levelize.argtypes = [i32, i64, P, P, P, P, P, P]
    lib.orc_tb_levels.argtypes = [i32, i64, P, P, P, P, P, P, P, P]
    lib.orc_critical_path.argtypes = [i32, i64, P, P, P, P, P, P, P, i64, P, P, P]
    lib.orc_label_memory.argtypes = [i32, P, P, i32, P, P, P]
    for f in (lib.orc_validate, lib.orc_levelize, lib.orc_tb_levels,
              lib.orc_critical_path, lib.orc_label_memory):
        f.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=True)
        _lib = bind(LIB_PATH)
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def validate(n_nodes, src, dst, comp, edge_cost, mem) -> int:
    """Status of the input checks: ids in range, weights >= 0, no overflow."""
    src, dst, comp, edge_cost, mem = _i32(src), _i32(dst), _i64(comp), _i64(edge_cost), _i64(mem)
    return _load().orc_validate(n_nodes, len(src), _ptr(src), _ptr(dst), _ptr(comp),
                                _ptr(edge_cost), _ptr(mem))


def levelize(n_nodes, src, dst):
    """Hop levels, (level, id) order and level offsets; raises on a cycle."""
    src, dst = _i32(src), _i32(dst)
    level = np.empty(n_nodes, np.int32)
    order = np.empty(n_nodes, np.int32)
    level_ptr = np.empty(n_nodes + 1, np.int32)
    nl = np.zeros(1, np.int32)
    st = _load().orc_levelize(n_nodes, len(src), _ptr(src), _ptr(dst), _ptr(level),
                              _ptr(order), _ptr(level_ptr), _ptr(nl))
    if st != OK:
        raise OracleError(st, "levelize")
    n = int(nl[0])
    return level, order, level_ptr[: n + 1].copy(), n


def tb_levels(n_nodes, src, dst, comp, edge_cost, label):
    """(tl, bl, makespan) of Table 2 under the placement ``label``."""
    src, dst, comp, edge_cost, label = _i32(src), _i32(dst), _i64(comp), _i64(edge_cost), _i32(label)
    tl = np.empty(n_nodes, np.int64)
    bl = np.empty(n_nodes, np.int64)
    m = np.zeros(1, np.int64)
    st = _load().orc_tb_levels(n_nodes, len(src), _ptr(src), _ptr(dst), _ptr(comp),
                               _ptr(edge_cost), _ptr(label), _ptr(tl), _ptr(bl), _ptr(m))
    if st != OK:
        raise OracleError(st, "tb_levels")
    return tl, bl, int(m[0])


def critical_path(n_nodes, src, dst, comp, edge_cost, label, tl, bl, makespan):
    """(is_critical uint8[V], canonical path int32[len]) for given tl/bl/M."""
    src, dst, comp, edge_cost, label = _i32(src), _i32(dst), _i64(comp), _i64(edge_cost), _i32(label)
    tl, bl = _i64(tl), _i64(bl)
    crit = np.empty(n_nodes, np.uint8)
    path = np.empty(max(n_nodes, 1), np.int32)
    plen = np.zeros(1, np.int32)
    st = _load().orc_critical_path(n_nodes, len(src), _ptr(src), _ptr(dst), _ptr(comp),
                                   _ptr(edge_cost), _ptr(label), _ptr(tl), _ptr(bl),
                                   int(makespan), _ptr(crit), _ptr(path), _ptr(plen))
    if st != OK:
        raise OracleError(st, "critical_path")
    return crit, path[: int(plen[0])].copy()


def label_memory(n_nodes, mem, label, n_labels, capacity=None):
    """(label_mem int64[K], overflow int64[K]) for labels in [0, K)."""
    mem, label = _i64(mem), _i32(label)
    cap = None if capacity is None else _i64(capacity)
    sums = np.empty(max(n_labels, 1), np.int64)
    over = np.empty(max(n_labels, 1), np.int64)
    st = _load().orc_label_memory(n_nodes, _ptr(mem), _ptr(label), n_labels, _ptr(cap),
                                  _ptr(sums), _ptr(over))
    if st != OK:
        raise OracleError(st, "label_memory")
    return sums[:n_labels].copy(), over[:n_labels].copy()


def evaluate(n_nodes, src, dst, comp, edge_cost, mem, label, n_labels, capacity=None):
    """One full placement evaluation: every output of the hot path."""
    tl, bl, m = tb_levels(n_nodes, src, dst, comp, edge_cost, label)
    crit, path = critical_path(n_nodes, src, dst, comp, edge_cost, label, tl, bl, m)
    sums, over = label_memory(n_nodes, mem, label, n_labels, capacity)
    return {"tl": tl, "bl": bl, "makespan": m, "is_critical": crit, "path": path,
            "label_mem": sums, "overflow": over}
