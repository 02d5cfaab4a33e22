"""MI355X (gfx950) placement-aware critical-path evaluator: Python binding.

The evaluation of ParDNN's partitioner hot path (arXiv 2008.08636: weighted
levels tl/bl, makespan, critical path, per-label memory) runs entirely in the
HIP kernels of ``libpardnn.so``, behind the C ABI of ``include/pardnn.h``.
This module only marshals arguments: torch tensors provide device memory and
the current HIP stream, and each function below forwards to the C entry point
of the same name. There is no fallback: without the built library every call
raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "PardnnError", "load_library", "Graph",
    "pardnn_graph_create", "pardnn_graph_destroy", "pardnn_set_stream", "pardnn_get_info",
    "pardnn_levelize", "pardnn_tb_levels", "pardnn_critical_path", "pardnn_label_memory",
    "pardnn_apply_moves", "pardnn_build_placements", "pardnn_evaluate_batch",
    "pardnn_evaluate_batch_fixed",
    "pardnn_evaluate_moves",
    "pardnn_tb_levels_batch", "pardnn_memory_balance", "pardnn_slice_primaries",
    "pardnn_slice_graph",
    "pardnn_cluster_criticality", "pardnn_span_work", "pardnn_set_timing",
    "pardnn_get_timing", "pardnn_set_deferred_errors", "pardnn_take_errors",
    "pardnn_status_string", "pardnn_last_error",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpardnn.so")

OK, E_INVAL, E_CYCLE, E_OVERFLOW, E_NOMEM, E_DEVICE = 0, -1, -2, -3, -4, -5


class PardnnError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        super().__init__(f"{func} failed: status {status} ({detail})")
        self.status = status


class _Info(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int64),
                ("n_levels", ctypes.c_int32), ("max_width", ctypes.c_int32),
                ("device", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libpardnn.so and declare the C signatures (raises if not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2008_08636_amd.build`")
    lib = ctypes.CDLL(path)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "pardnn_graph_create": [i32, i64, P, P, P, P, P, P, ctypes.POINTER(P)],
        "pardnn_graph_destroy": [P],
        "pardnn_set_stream": [P, P],
        "pardnn_get_info": [P, ctypes.POINTER(_Info)],
        "pardnn_levelize": [P, P, P, P, ctypes.POINTER(i32)],
        "pardnn_tb_levels": [P, P, P, P, P],
        "pardnn_critical_path": [P, P, P, P, P, P, P, P],
        "pardnn_label_memory": [P, P, i32, P, P, P],
        "pardnn_apply_moves": [P, P, i32, P, P],
        "pardnn_build_placements": [P, P, i32, P, i64, P, P, P],
        "pardnn_evaluate_batch": [P, i32, P, i32, P, P, P, P, P, P, i32, P, P, P],
        "pardnn_evaluate_batch_fixed": [P, i32, P, i32, P, P, P, P, P, P, i32, P, P, P],
        "pardnn_evaluate_moves": [P, P, i32, P, i64, P, P, i32, P, P, P, P, P, P, i32, P, P, P],
        "pardnn_tb_levels_batch": [P, i32, P, P, P, P],
        "pardnn_memory_balance": [P, i32, P, P, P, i32, P, P, P, P],
        "pardnn_slice_primaries": [P, i32, P, P, i32, P, P],
        "pardnn_slice_graph": [P, i32, P, P, P, P, P],
        "pardnn_cluster_criticality": [P, P, i32, P, P],
        "pardnn_span_work": [P, P, i32, P, i32, P, P, P, P, P, P],
        "pardnn_set_timing": [P, ctypes.c_int],
        "pardnn_get_timing": [P, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_float)],
        "pardnn_set_deferred_errors": [P, ctypes.c_int],
        "pardnn_take_errors": [P],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.pardnn_status_string.argtypes = [ctypes.c_int]
    lib.pardnn_status_string.restype = ctypes.c_char_p
    lib.pardnn_last_error.argtypes = []
    lib.pardnn_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def pardnn_status_string(status: int) -> str:
    return load_library().pardnn_status_string(status).decode()


def pardnn_last_error() -> str:
    return load_library().pardnn_last_error().decode()


def _check(status: int, func: str):
    if status != OK:
        raise PardnnError(status, func, pardnn_last_error() or pardnn_status_string(status))


def _ptr(t, dtype=None, numel=None, name="tensor"):
    """Device pointer of a contiguous CUDA/HIP tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must live on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} must hold at least {numel} elements, has {t.numel()}")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() > 0 else None


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


# ---------------------------------------------------------------- C entry points --

def pardnn_graph_create(n_nodes, src, dst, comp, edge_cost, mem, stream=None):
    n_edges = src.numel()
    h = ctypes.c_void_p()
    st = load_library().pardnn_graph_create(
        n_nodes, n_edges, _ptr(src, torch.int32, n_edges, "src"),
        _ptr(dst, torch.int32, n_edges, "dst"), _ptr(comp, torch.int64, n_nodes, "comp"),
        _ptr(edge_cost, torch.int64, n_edges, "edge_cost"), _ptr(mem, torch.int64, n_nodes, "mem"),
        _stream(stream), ctypes.byref(h))
    _check(st, "pardnn_graph_create")
    return h


def pardnn_graph_destroy(h):
    _check(load_library().pardnn_graph_destroy(h), "pardnn_graph_destroy")


def pardnn_set_stream(h, stream=None):
    _check(load_library().pardnn_set_stream(h, _stream(stream)), "pardnn_set_stream")


def pardnn_get_info(h) -> dict:
    info = _Info()
    _check(load_library().pardnn_get_info(h, ctypes.byref(info)), "pardnn_get_info")
    return {f: getattr(info, f) for f, _ in _Info._fields_}


def pardnn_levelize(h, level=None, order=None, level_ptr=None) -> int:
    n = ctypes.c_int32(-1)
    _check(load_library().pardnn_levelize(h, _ptr(level, torch.int32, name="level"),
                                          _ptr(order, torch.int32, name="order"),
                                          _ptr(level_ptr, torch.int32, name="level_ptr"),
                                          ctypes.byref(n)), "pardnn_levelize")
    return n.value


def _n_nodes(h) -> int:
    return pardnn_get_info(h)["n_nodes"]


def pardnn_tb_levels(h, placement, tl, bl, makespan):
    V = _n_nodes(h)
    _check(load_library().pardnn_tb_levels(h, _ptr(placement, torch.int32, V, "placement"),
                                           _ptr(tl, torch.int64, V, "tl"),
                                           _ptr(bl, torch.int64, V, "bl"),
                                           _ptr(makespan, torch.int64, 1, "makespan")),
           "pardnn_tb_levels")


def pardnn_critical_path(h, placement, tl, bl, makespan, is_critical, path, path_len):
    V = _n_nodes(h)
    _check(load_library().pardnn_critical_path(
        h, _ptr(placement, torch.int32, V, "placement"), _ptr(tl, torch.int64, V, "tl"),
        _ptr(bl, torch.int64, V, "bl"), _ptr(makespan, torch.int64, 1, "makespan"),
        _ptr(is_critical, torch.uint8, V, "is_critical"), _ptr(path, torch.int32, V, "path"),
        _ptr(path_len, torch.int32, 1, "path_len")), "pardnn_critical_path")


def pardnn_label_memory(h, placement, n_labels, capacity, label_mem, overflow=None):
    _check(load_library().pardnn_label_memory(
        h, _ptr(placement, torch.int32, _n_nodes(h), "placement"), n_labels,
        _ptr(capacity, torch.int64, n_labels, "capacity"),
        _ptr(label_mem, torch.int64, n_labels, "label_mem"),
        _ptr(overflow, torch.int64, n_labels, "overflow")), "pardnn_label_memory")


def pardnn_apply_moves(h, placement, node, label):
    n = node.numel()
    _check(load_library().pardnn_apply_moves(
        h, _ptr(placement, torch.int32, name="placement"), n, _ptr(node, torch.int32, n, "node"),
        _ptr(label, torch.int32, n, "label")), "pardnn_apply_moves")


def _n_moves(node, label, n_moves):
    """The number of moves: the length of node (and label) unless given."""
    if n_moves is None:
        n_moves = 0 if node is None else node.numel()
    for t, name in ((node, "node"), (label, "label")):
        if n_moves > 0 and (t is None or t.numel() < n_moves):
            raise ValueError(f"{name} must hold at least n_moves = {n_moves} elements")
    return n_moves


def pardnn_build_placements(h, base, n_place, step_ptr, node, label, placements, n_moves=None):
    n_moves = _n_moves(node, label, n_moves)
    _check(load_library().pardnn_build_placements(
        h, _ptr(base, torch.int32, name="base"), n_place,
        _ptr(step_ptr, torch.int64, n_place + 1, "step_ptr"), n_moves,
        _ptr(node, torch.int32, name="node"), _ptr(label, torch.int32, name="label"),
        _ptr(placements, torch.int32, name="placements")),
        "pardnn_build_placements")


def pardnn_evaluate_batch(h, n_place, placements, n_labels, capacity, tl, bl, makespan,
                          is_critical=None, path=None, path_stride=0, path_len=None,
                          label_mem=None, overflow=None):
    _check(load_library().pardnn_evaluate_batch(
        h, n_place, _ptr(placements, torch.int32, name="placements"), n_labels,
        _ptr(capacity, torch.int64, name="capacity"), _ptr(tl, torch.int64, name="tl"),
        _ptr(bl, torch.int64, name="bl"), _ptr(makespan, torch.int64, n_place, "makespan"),
        _ptr(is_critical, torch.uint8, name="is_critical"), _ptr(path, torch.int32, name="path"),
        path_stride, _ptr(path_len, torch.int32, name="path_len"),
        _ptr(label_mem, torch.int64, name="label_mem"), _ptr(overflow, torch.int64, name="overflow")),
        "pardnn_evaluate_batch")


def pardnn_evaluate_batch_fixed(h, n_place, placements, n_labels, capacity, tl, bl, makespan,
                                is_critical=None, path=None, path_stride=0, path_len=None,
                                label_mem=None, overflow=None):
    _check(load_library().pardnn_evaluate_batch_fixed(
        h, n_place, _ptr(placements, torch.int32, name="placements"), n_labels,
        _ptr(capacity, torch.int64, name="capacity"), _ptr(tl, torch.int64, name="tl"),
        _ptr(bl, torch.int64, name="bl"), _ptr(makespan, torch.int64, n_place, "makespan"),
        _ptr(is_critical, torch.uint8, name="is_critical"), _ptr(path, torch.int32, name="path"),
        path_stride, _ptr(path_len, torch.int32, name="path_len"),
        _ptr(label_mem, torch.int64, name="label_mem"), _ptr(overflow, torch.int64, name="overflow")),
        "pardnn_evaluate_batch_fixed")


def pardnn_evaluate_moves(h, base, n_place, step_ptr, node, label, n_labels, capacity, tl, bl,
                          makespan, is_critical=None, path=None, path_stride=0, path_len=None,
                          label_mem=None, overflow=None, n_moves=None):
    n_moves = _n_moves(node, label, n_moves)
    _check(load_library().pardnn_evaluate_moves(
        h, _ptr(base, torch.int32, name="base"), n_place,
        _ptr(step_ptr, torch.int64, n_place + 1, "step_ptr"), n_moves,
        _ptr(node, torch.int32, name="node"),
        _ptr(label, torch.int32, name="label"), n_labels,
        _ptr(capacity, torch.int64, name="capacity"), _ptr(tl, torch.int64, name="tl"),
        _ptr(bl, torch.int64, name="bl"), _ptr(makespan, torch.int64, n_place, "makespan"),
        _ptr(is_critical, torch.uint8, name="is_critical"), _ptr(path, torch.int32, name="path"),
        path_stride, _ptr(path_len, torch.int32, name="path_len"),
        _ptr(label_mem, torch.int64, name="label_mem"), _ptr(overflow, torch.int64, name="overflow")),
        "pardnn_evaluate_moves")


def pardnn_tb_levels_batch(h, n_place, placements, tl, bl, makespan):
    _check(load_library().pardnn_tb_levels_batch(
        h, n_place, _ptr(placements, torch.int32, name="placements"),
        _ptr(tl, torch.int64, name="tl"), _ptr(bl, torch.int64, name="bl"),
        _ptr(makespan, torch.int64, n_place, "makespan")), "pardnn_tb_levels_batch")


def pardnn_memory_balance(h, n_place, placements, node_type, ref_target, n_labels, res_mem,
                          nor_mem, balanced, ref_misplaced):
    V, PK = _n_nodes(h), max(n_place, 0) * max(n_labels, 0)
    _check(load_library().pardnn_memory_balance(
        h, n_place, _ptr(placements, torch.int32, V * max(n_place, 0), "placements"),
        _ptr(node_type, torch.int32, V, "node_type"), _ptr(ref_target, torch.int32, V, "ref_target"),
        n_labels, _ptr(res_mem, torch.int64, PK, "res_mem"), _ptr(nor_mem, torch.int64, PK, "nor_mem"),
        _ptr(balanced, torch.uint8, PK, "balanced"),
        _ptr(ref_misplaced, torch.int64, max(n_place, 0), "ref_misplaced")), "pardnn_memory_balance")


def pardnn_slice_primaries(h, K, primary, paths, path_stride, path_len, makespan):
    Kn = max(K, 0)
    _check(load_library().pardnn_slice_primaries(
        h, K, _ptr(primary, torch.int32, _n_nodes(h), "primary"),
        _ptr(paths, torch.int32, Kn * max(path_stride, 0), "paths"), path_stride,
        _ptr(path_len, torch.int32, Kn, "path_len"), _ptr(makespan, torch.int64, Kn, "makespan")),
        "pardnn_slice_primaries")


def pardnn_slice_graph(h, K, cluster, cluster_off, cluster_nodes, n_clusters, makespan=None):
    n = _n_nodes(h)
    _check(load_library().pardnn_slice_graph(
        h, K, _ptr(cluster, torch.int32, n, "cluster"),
        _ptr(cluster_off, torch.int32, n + K + 1, "cluster_off"),
        _ptr(cluster_nodes, torch.int32, n, "cluster_nodes"),
        _ptr(n_clusters, torch.int32, 1, "n_clusters"),
        _ptr(makespan, torch.int64, K, "makespan")), "pardnn_slice_graph")


def pardnn_cluster_criticality(h, cluster, n_clusters, criticality, order):
    C = max(n_clusters, 0)
    _check(load_library().pardnn_cluster_criticality(
        h, _ptr(cluster, torch.int32, _n_nodes(h), "cluster"), n_clusters,
        _ptr(criticality, torch.int64, C, "criticality"), _ptr(order, torch.int32, C, "order")),
        "pardnn_cluster_criticality")


def pardnn_span_work(h, label, K, cluster, n_clusters, tl, span_lo, span_hi, work, comm, choice):
    V, C = _n_nodes(h), max(n_clusters, 0)
    CK = C * max(K, 0)
    _check(load_library().pardnn_span_work(
        h, _ptr(label, torch.int32, V, "label"), K, _ptr(cluster, torch.int32, V, "cluster"),
        n_clusters, _ptr(tl, torch.int64, V, "tl"), _ptr(span_lo, torch.int64, C, "span_lo"),
        _ptr(span_hi, torch.int64, C, "span_hi"), _ptr(work, torch.int64, CK, "work"),
        _ptr(comm, torch.int64, CK, "comm"), _ptr(choice, torch.int32, C, "choice")),
        "pardnn_span_work")


def pardnn_set_timing(h, enable: bool = True):
    _check(load_library().pardnn_set_timing(h, 1 if enable else 0), "pardnn_set_timing")


def pardnn_set_deferred_errors(h, enable: bool = True):
    _check(load_library().pardnn_set_deferred_errors(h, 1 if enable else 0),
           "pardnn_set_deferred_errors")


def pardnn_take_errors(h):
    _check(load_library().pardnn_take_errors(h), "pardnn_take_errors")


def pardnn_get_timing(h):
    """(kernel name, elapsed ms) of the last timed launch on the handle."""
    name = ctypes.c_char_p()
    ms = ctypes.c_float()
    _check(load_library().pardnn_get_timing(h, ctypes.byref(name), ctypes.byref(ms)),
           "pardnn_get_timing")
    return name.value.decode(), float(ms.value)


# ---------------------------------------------------------------- convenience --

class Graph:
    """One handle of the C library plus output allocation on the torch device."""

    def __init__(self, n_nodes, src, dst, comp, edge_cost, mem, device="cuda", stream=None):
        dev = torch.device(device)
        self.device = dev
        self.n_nodes = int(n_nodes)

        def on(x, dt):
            return torch.as_tensor(x, dtype=dt).to(dev).contiguous()

        self.n_edges = int(len(src))
        self._h = pardnn_graph_create(self.n_nodes, on(src, torch.int32), on(dst, torch.int32),
                                      on(comp, torch.int64), on(edge_cost, torch.int64),
                                      on(mem, torch.int64), stream)

    def close(self):
        if getattr(self, "_h", None) is not None:
            pardnn_graph_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def info(self) -> dict:
        return pardnn_get_info(self._h)

    def levelize(self):
        V = self.n_nodes
        level = torch.empty(V, dtype=torch.int32, device=self.device)
        order = torch.empty(V, dtype=torch.int32, device=self.device)
        level_ptr = torch.empty(V + 1, dtype=torch.int32, device=self.device)
        n = pardnn_levelize(self._h, level, order, level_ptr)
        return level, order, level_ptr[: n + 1], n

    def tb_levels(self, placement):
        V = self.n_nodes
        tl = torch.empty(V, dtype=torch.int64, device=self.device)
        bl = torch.empty(V, dtype=torch.int64, device=self.device)
        m = torch.empty(1, dtype=torch.int64, device=self.device)
        pardnn_tb_levels(self._h, placement, tl, bl, m)
        return tl, bl, m

    def critical_path(self, placement, tl, bl, makespan):
        V = self.n_nodes
        crit = torch.empty(V, dtype=torch.uint8, device=self.device)
        path = torch.empty(max(V, 1), dtype=torch.int32, device=self.device)
        plen = torch.empty(1, dtype=torch.int32, device=self.device)
        pardnn_critical_path(self._h, placement, tl, bl, makespan, crit, path, plen)
        return crit, path, plen

    def label_memory(self, placement, n_labels, capacity=None):
        sums = torch.empty(n_labels, dtype=torch.int64, device=self.device)
        over = torch.empty(n_labels, dtype=torch.int64, device=self.device)
        pardnn_label_memory(self._h, placement, n_labels, capacity, sums, over)
        return sums, over

    def apply_moves(self, placement, node, label):
        pardnn_apply_moves(self._h, placement, node, label)

    def build_placements(self, base, step_ptr, node, label):
        n_place = step_ptr.numel() - 1
        out = torch.empty((self.n_nodes, n_place), dtype=torch.int32, device=self.device)
        pardnn_build_placements(self._h, base, n_place, step_ptr, node, label, out)
        return out

    def _outputs(self, P, n_labels, crit, path, labels, values=True):
        V, dev = self.n_nodes, self.device
        L = self.info()["n_levels"]
        if L < 0:
            L = pardnn_levelize(self._h)
        out = {"makespan": torch.empty(P, dtype=torch.int64, device=dev)}
        if values:
            out["tl"] = torch.empty((V, P), dtype=torch.int64, device=dev)
            out["bl"] = torch.empty((V, P), dtype=torch.int64, device=dev)
        if crit:
            out["is_critical"] = torch.empty((V, P), dtype=torch.uint8, device=dev)
        if path:
            out["path"] = torch.empty((P, max(L, 1)), dtype=torch.int32, device=dev)
            out["path_len"] = torch.empty(P, dtype=torch.int32, device=dev)
        if labels and n_labels > 0:
            out["label_mem"] = torch.empty((P, n_labels), dtype=torch.int64, device=dev)
            out["overflow"] = torch.empty((P, n_labels), dtype=torch.int64, device=dev)
        return out, max(L, 1)

    def evaluate_moves(self, base, step_ptr, node, label, n_labels=0, capacity=None, crit=True,
                       path=True, labels=True, values=True):
        """All outputs for the successive placements base + moves (see
        pardnn_evaluate_moves); arrays are placement-minor [V][P]. values=False
        leaves out the per-node tl / bl; labels=False the label sums (n_labels
        is then a hint of the label range)."""
        P = step_ptr.numel() - 1
        out, stride = self._outputs(P, n_labels, crit, path, labels, values)
        pardnn_evaluate_moves(self._h, base, P, step_ptr, node, label,
                              n_labels, capacity, out.get("tl"), out.get("bl"),
                              out["makespan"], out.get("is_critical"), out.get("path"), stride,
                              out.get("path_len"), out.get("label_mem"), out.get("overflow"))
        return out

    def memory_balance(self, placements, node_type, ref_target, n_labels):
        """Memory Heuristic II per placement (see pardnn_memory_balance);
        placements [V] or [V][P] (placement-minor)."""
        P = 1 if placements.dim() == 1 else placements.shape[1]
        dev = self.device
        out = {
            "res_mem": torch.empty((P, n_labels), dtype=torch.int64, device=dev),
            "nor_mem": torch.empty((P, n_labels), dtype=torch.int64, device=dev),
            "balanced": torch.empty((P, n_labels), dtype=torch.uint8, device=dev),
            "ref_misplaced": torch.empty(P, dtype=torch.int64, device=dev),
        }
        pardnn_memory_balance(self._h, P, placements, node_type, ref_target, n_labels,
                              out["res_mem"], out["nor_mem"], out["balanced"],
                              out["ref_misplaced"])
        return out

    def cluster_criticality(self, cluster, n_clusters):
        """Criticality per cluster and the cluster order (see
        pardnn_cluster_criticality)."""
        crit = torch.empty(n_clusters, dtype=torch.int64, device=self.device)
        order = torch.empty(n_clusters, dtype=torch.int32, device=self.device)
        pardnn_cluster_criticality(self._h, cluster, n_clusters, crit, order)
        return crit, order

    def span_work(self, label, K, cluster, n_clusters, tl):
        """Eq. 2 terms and choices for every cluster (see pardnn_span_work)."""
        C = n_clusters
        i64 = dict(dtype=torch.int64, device=self.device)
        out = {"span_lo": torch.empty(C, **i64), "span_hi": torch.empty(C, **i64),
               "work": torch.empty((C, K), **i64), "comm": torch.empty((C, K), **i64),
               "choice": torch.empty(C, dtype=torch.int32, device=self.device)}
        pardnn_span_work(self._h, label, K, cluster, C, tl, out["span_lo"], out["span_hi"],
                         out["work"], out["comm"], out["choice"])
        return out

    def slice_primaries(self, K):
        """The K primary clusters of graph slicing (see pardnn_slice_primaries)."""
        L = self.info()["n_levels"]
        if L < 0:
            L = pardnn_levelize(self._h)
        dev, stride = self.device, max(L, 1)
        out = {
            "primary": torch.empty(self.n_nodes, dtype=torch.int32, device=dev),
            "paths": torch.empty((K, stride), dtype=torch.int32, device=dev),
            "path_len": torch.empty(K, dtype=torch.int32, device=dev),
            "makespan": torch.empty(K, dtype=torch.int64, device=dev),
        }
        pardnn_slice_primaries(self._h, K, out["primary"], out["paths"], stride,
                               out["path_len"], out["makespan"])
        return out

    def slice_graph(self, K):
        """Graph slicing in full: primaries and secondaries (see
        pardnn_slice_graph). Returns cluster [V], the clusters as a list of
        node-id tensors in path order, and the primaries' makespans."""
        V, dev = self.n_nodes, self.device
        cluster = torch.empty(V, dtype=torch.int32, device=dev)
        off = torch.empty(V + K + 1, dtype=torch.int32, device=dev)
        nodes = torch.empty(max(V, 1), dtype=torch.int32, device=dev)
        n = torch.empty(1, dtype=torch.int32, device=dev)
        ms = torch.empty(max(K, 1), dtype=torch.int64, device=dev)
        pardnn_slice_graph(self._h, K, cluster, off, nodes, n, ms if K > 0 else None)
        nc = int(n.item())
        offs = off[: nc + 1].cpu().tolist()
        return {"cluster": cluster, "cluster_off": off[: nc + 1], "cluster_nodes": nodes[:V],
                "paths": [nodes[offs[c]:offs[c + 1]] for c in range(nc)], "makespan": ms[:K]}

    def evaluate_batch(self, placements, n_labels=0, capacity=None, crit=True, path=True,
                       labels=True):
        """All outputs for placements [V][P] (placement-minor)."""
        V, P = self.n_nodes, placements.shape[1]
        dev = self.device
        L = self.info()["n_levels"]
        if L < 0:
            L = pardnn_levelize(self._h)
        out = {
            "tl": torch.empty((V, P), dtype=torch.int64, device=dev),
            "bl": torch.empty((V, P), dtype=torch.int64, device=dev),
            "makespan": torch.empty(P, dtype=torch.int64, device=dev),
        }
        if crit:
            out["is_critical"] = torch.empty((V, P), dtype=torch.uint8, device=dev)
        stride = max(L, 1)
        if path:
            out["path"] = torch.empty((P, stride), dtype=torch.int32, device=dev)
            out["path_len"] = torch.empty(P, dtype=torch.int32, device=dev)
        if labels and n_labels > 0:
            out["label_mem"] = torch.empty((P, n_labels), dtype=torch.int64, device=dev)
            out["overflow"] = torch.empty((P, n_labels), dtype=torch.int64, device=dev)
        pardnn_evaluate_batch(self._h, P, placements, n_labels, capacity,
                              out["tl"], out["bl"], out["makespan"], out.get("is_critical"),
                              out.get("path"), stride, out.get("path_len"),
                              out.get("label_mem"), out.get("overflow"))
        return out
