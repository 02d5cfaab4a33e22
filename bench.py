#!/usr/bin/env python3
"""Benchmark of the placement-aware critical-path evaluator on one MI355X.

Default workload (one "step" = one pass of the whole hot path over one batch):
the refinement loop of 1,000 successive placements of the transformer-shaped
training DAG (48 blocks, ~307k ops, ~867k edges, 16 labels), each placement
moving 1 % of the ops. A step applies the per-step moves and evaluates every
placement in full -- t-levels, b-levels, makespan, critical nodes, canonical
critical path, per-label memory and overflow -- in one call
(pardnn_evaluate_moves). Graph structure (create + levelize) is built once
before the timed region and reported apart.

Printed: ONE JSON line with GTEPS (2E relaxations per placement per t+b sweep)
as `value`, placement evaluations/s, the roofline of the dominant kernel
(HIP events around it, on the library's stream), and the CPU oracle timed on a
bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GTEPS (edges relaxed/sec, t+b sweep) and placement evaluations/sec, 1 MI355X"
HBM_PEAK_GBS = 8000.0


def algorithmic_bytes_batch(V: int, E: int, P: int) -> int:
    """Bytes a full evaluation of P placements moves at minimum: per placement
    24 B per edge (neighbour label 4 + value 8, for the t and the b sweep) and
    53 B per node (t sweep: label 4, tl 8, tl + comp 8; b sweep: label 4, bl 8;
    critical flags: tl 8, bl 8, flag 1; label sums: label 4); per batch the
    shared structure, 24 B per edge (neighbour id 4 + cost 8, twice) and 32 B
    per node (offsets 4 + comp 8, twice; mem 8)."""
    return P * (24 * E + 53 * V) + 24 * E + 32 * V


def algorithmic_bytes_sweep(V: int, E: int, P: int) -> int:
    """The share of the same accounting that the sweep kernel moves (t and b
    sweeps plus the label sums; the critical flags are written afterwards): per
    placement 24 B per edge and 36 B per node, plus the shared structure."""
    return P * (24 * E + 36 * V) + 24 * E + 32 * V


def algorithmic_bytes_single(V: int, E: int) -> int:
    """One full evaluation of one placement: 48 B per edge, 85 B per node."""
    return 48 * E + 85 * V


def algorithmic_bytes_tb_single(V: int, E: int) -> int:
    """One t+b sweep of one placement without the critical path: 48 B per edge
    (per direction: neighbour id 4, cost 8, neighbour label 4, value 8) and
    64 B per node (labels 4 + 4, offsets 4 + 4, comp 8 + 8, tl written 8,
    tl + comp 8, bl 8, bl written 8)."""
    return 48 * E + 64 * V


def algorithmic_bytes_secondary(V: int, E: int) -> int:
    """The secondary walk of graph slicing over the graph left after the
    primaries (bounded here by the whole graph): per node its priority (8 B)
    read and its cluster id and list entry written (4 + 4 B); per edge the
    successor id read (4 B) and the successor's removed flag tested (4 B)."""
    return 16 * V + 8 * E


def algorithmic_bytes_mem_balance(V: int, P: int, K: int, n_ref: int) -> int:
    """The sums kernel of Memory Heuristic II on P placements: the [V][P]
    placement matrix (4 B per entry), the target label of each reference node
    (4 B per placement), per node mem 8, kind 4, target 4; per placement and
    label two sums written (16 B) and 8 B of misplaced count."""
    return 4 * V * P + 4 * n_ref * P + 16 * V + 16 * P * K + 8 * P


def algorithmic_bytes_span_work(V: int, E: int, C: int, K: int) -> int:
    """Eq. 2 terms for C clusters and K partitions: per node label 4, cluster 4,
    level 4, tl 8, comp 8; per edge src 4, dst 4, cost 8; per cluster the span
    (16 B) and choice (4 B) written; per (cluster, partition) work and comm
    (16 B) written."""
    return 28 * V + 16 * E + 20 * C + 16 * C * K


def source_digest(*names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2008_08636_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload_key: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
        e = d[kernel][workload_key]
        if e.get("source_digest") != source_digest(*e["sources"]):
            return None
        return int(e["hbm_bytes_per_launch"])
    except Exception:
        return None


def host_cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def start_cpu_baseline(mode: str, budget_s: float, config: int = 2, n_place: int = 1000):
    """Start the oracle's timing (oracle/timing.py) as a child process pinned to
    one core, before this process touches the GPU, and take that core out of
    this process's own affinity so that the two do not share it. Returns the
    child (or None when there is no core to spare)."""
    import subprocess

    cores = sorted(os.sched_getaffinity(0))
    if budget_s <= 0 or len(cores) < 2:
        return None
    core = cores[-1]
    os.sched_setaffinity(0, set(cores[:-1]))
    cmd = [sys.executable, "-m", "oracle.timing", "--mode", mode, "--config", str(config),
           "--configs", "0,1,2", "--n-place", str(n_place), "--budget", str(budget_s),
           "--core", str(core)]
    return subprocess.Popen(cmd, cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                            text=True)


def finish_cpu_baseline(child, timeout_s: float):
    """The child's JSON result, or None if it failed."""
    if child is None:
        return None
    try:
        out, err = child.communicate(timeout=timeout_s)
    except Exception:
        child.kill()
        child.communicate()
        print("[bench] CPU baseline timed out", file=sys.stderr, flush=True)
        return None
    if child.returncode != 0:
        print(f"[bench] CPU baseline failed: {err[-500:]}", file=sys.stderr, flush=True)
        return None
    return json.loads(out.strip().splitlines()[-1])


def cpu_baseline_line(r, E: int, what: str):
    """cpu_baseline object of the refinement line from the child's result."""
    if r is None:
        return None
    med = r["median_s"]
    return {
        "value": round(2 * E / med / 1e9, 6),
        "unit": "GTEPS",
        "cores": len(r["pinned_cores"]),
        "kind": "oracle",
        "sample": f"{what}: {r['what']}, each evaluated in full (levels, tl, bl, makespan, "
                  f"critical path, label memory) by the oracle built with {r['build']}, one "
                  f"thread pinned to core {r['pinned_cores']}; median {med * 1e3:.1f} ms per "
                  f"evaluation ({1 / med:.2f} evaluations/s) over {r['reps']} timed runs after "
                  f"a warm-up; host: {r['nproc']} logical CPUs, '{r['cpu_model']}'",
        "median_ms": round(med * 1e3, 3),
        "reps": r["reps"],
        "nproc": r["nproc"],
        "cpu_model": r["cpu_model"],
    }


ROWS = ("refinement", "single", "memory_balance", "cluster_criticality", "slicing", "slice_graph",
        "span_work")


def time_calls(P, G, fn, steps: int, warmup: int):
    """Wall time per call (ms) and the mean HIP-event time of the call's timed
    kernel (ms) over `steps` calls after `warmup` untimed ones."""
    import numpy as np
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ks = []
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
        ks.append(P.pardnn_get_timing(G.handle)[1])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    return wall, float(np.mean(ks)), P.pardnn_get_timing(G.handle)[0]


def hbm_roofline(kernel: str, kernel_ms: float, alg_bytes: int, note: str = ""):
    achieved = alg_bytes / (kernel_ms / 1e3) / 1e9
    r = {"bound": "hbm", "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS, "unit": "GB/s",
         "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": None, "kernel": kernel,
         "kernel_ms": round(kernel_ms, 4), "algorithmic_bytes_per_launch": alg_bytes}
    if note:
        r["note"] = note
    return r


def bench_single(args, child) -> int:
    """One full evaluation of one placement (t/b levels, critical path, label
    memory: pardnn_tb_levels + pardnn_critical_path + pardnn_label_memory) on
    each of the four single-graph workloads; one JSON line, `value` on the
    transformer graph."""
    import numpy as np
    import torch

    import paper_2008_08636_amd as P
    import workloads as W

    P.load_library()
    names = {0: "tiny layered DAG", 1: "stacked-LSTM training DAG",
             2: "transformer training DAG", 3: "Wide-ResNet-shaped DAG"}
    per, cpu = {}, {}
    for i in (0, 1, 2, 3):
        g = W.make_config(i)
        V, E, K = g.n_nodes, g.n_edges, g.n_labels
        G = P.Graph(V, g.src, g.dst, g.comp, g.edge_cost, g.mem)
        P.pardnn_set_timing(G.handle, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        L = P.pardnn_levelize(G.handle)
        torch.cuda.synchronize()
        levelize_ms = (time.perf_counter() - t0) * 1e3
        kahn_ms = P.pardnn_get_timing(G.handle)[1]
        lab = torch.as_tensor(g.placement, dtype=torch.int32).cuda()
        cap = torch.as_tensor(g.capacity, dtype=torch.int64).cuda()
        tl = torch.empty(V, dtype=torch.int64, device="cuda")
        bl = torch.empty(V, dtype=torch.int64, device="cuda")
        m = torch.empty(1, dtype=torch.int64, device="cuda")
        crit = torch.empty(V, dtype=torch.uint8, device="cuda")
        path = torch.empty(max(V, 1), dtype=torch.int32, device="cuda")
        plen = torch.empty(1, dtype=torch.int32, device="cuda")
        sums = torch.empty(K, dtype=torch.int64, device="cuda")
        over = torch.empty(K, dtype=torch.int64, device="cuda")

        def fn():
            P.pardnn_tb_levels(G.handle, lab, tl, bl, m)
            P.pardnn_critical_path(G.handle, lab, tl, bl, m, crit, path, plen)
            P.pardnn_label_memory(G.handle, lab, K, cap, sums, over)

        steps = args.steps if i != 3 else max(2, args.steps // 4)
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ks = []
        t0 = time.perf_counter()
        for _ in range(steps):
            P.pardnn_tb_levels(G.handle, lab, tl, bl, m)
            ks.append(P.pardnn_get_timing(G.handle)[1])
            P.pardnn_critical_path(G.handle, lab, tl, bl, m, crit, path, plen)
            P.pardnn_label_memory(G.handle, lab, K, cap, sums, over)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / steps
        sweep_ms = float(np.mean(ks))
        per[f"config{i}"] = {"workload": names[i], "V": V, "E": E, "levels": L,
                             "levelize_ms": round(levelize_ms, 3), "k_kahn_ms": round(kahn_ms, 3),
                             "ms": round(wall, 4), "sweep_ms": round(sweep_ms, 4),
                             "us_per_level": round(sweep_ms * 1e3 / max(L, 1), 4),
                             "gteps": round(2 * E / (wall / 1e3) / 1e9, 4)}
        print(f"[bench] single config{i}: {wall:.3f} ms per evaluation, sweep {sweep_ms:.3f} ms",
              file=sys.stderr, flush=True)
        if i == 2:
            main = per["config2"]
            roof = hbm_roofline(P.pardnn_get_timing(G.handle)[0], sweep_ms,
                                algorithmic_bytes_tb_single(V, E),
                                "one placement walks the level chain one level at a time: "
                                "latency-bound")
        G.close()
    r = finish_cpu_baseline(child, 4 * args.cpu_budget + 120)
    if r is not None:
        for k, x in r["per_config"].items():
            cpu[k] = {"ms": round(x["median_s"] * 1e3, 3), "reps": x["reps"]}
    line = {
        "metric": "single-placement full evaluations/sec (t/b levels, critical path, label "
                  "memory), 1 MI355X",
        "value": round(1e3 / main["ms"], 3), "unit": "evaluations/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": main["ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": "one placement of the transformer training DAG, evaluated in "
                               "full; the other graphs alongside", "per_graph": per},
        "roofline": roof,
        "cpu_baseline": ({"value": round(1e3 / cpu["config2"]["ms"], 3), "unit": "evaluations/s",
                          "cores": len(r["pinned_cores"]), "kind": "oracle",
                          "sample": f"whole evaluations of each graph's own placement by the "
                                    f"oracle built with {r['build']}, one thread pinned to core "
                                    f"{r['pinned_cores']}, median over the timed runs after a "
                                    f"warm-up: " +
                                    ", ".join(f"{k} {v['ms']} ms x {v['reps']}"
                                              for k, v in cpu.items()) +
                                    f"; host: {r['nproc']} logical CPUs, '{r['cpu_model']}'"}
                         if cpu and "config2" in cpu else None),
    }
    print(json.dumps(line), flush=True)
    return 0


def bench_row(args, row: str) -> int:
    """One JSON line for a row after the core path, on the transformer graph."""
    import numpy as np
    import torch

    import paper_2008_08636_amd as P
    import workloads as W

    P.load_library()
    dev = lambda x, dt: torch.as_tensor(np.ascontiguousarray(x), dtype=dt).cuda()
    g = W.make_config(2)
    V, E, K = g.n_nodes, g.n_edges, g.n_labels
    G = P.Graph(V, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    L = P.pardnn_levelize(G.handle)
    P.pardnn_set_timing(G.handle, True)
    graph_desc = f"transformer-shaped training DAG, 48 blocks, V={V}, E={E}, {L} levels"
    print(f"[bench] row {row}: {graph_desc}", file=sys.stderr, flush=True)
    budget = args.cpu_budget
    cpu = None
    sweep_note = ("a single-placement sweep walks the level chain one level at a time, so "
                  "its bound is per-level latency, not bandwidth")

    if row == "memory_balance":
        sched = W.config4_moves(g, n_place=args.n_place)
        Pn = sched.n_place
        pl = G.build_placements(dev(sched.base, torch.int32), dev(sched.ptr, torch.int64),
                                dev(sched.node, torch.int32), dev(sched.label, torch.int32))
        kind_h, tgt_h = W.node_kinds(g)
        kind, tgt = dev(kind_h, torch.int32), dev(tgt_h, torch.int32)
        i64 = dict(dtype=torch.int64, device="cuda")
        res, nor = torch.empty((Pn, K), **i64), torch.empty((Pn, K), **i64)
        bal = torch.empty((Pn, K), dtype=torch.uint8, device="cuda")
        mis = torch.empty(Pn, **i64)
        fn = lambda: P.pardnn_memory_balance(G.handle, Pn, pl, kind, tgt, K, res, nor, bal, mis)
        wall, k_ms, kname = time_calls(P, G, fn, args.steps, args.warmup)
        n_ref = int(((kind_h == 2) & (tgt_h >= 0)).sum())
        roof = hbm_roofline(kname, k_ms, algorithmic_bytes_mem_balance(V, Pn, K, n_ref))
        roof["traffic"] = load_traffic("k_mem_balance_sums", f"heuristic2_transformer_V{V}_P{Pn}")
        value, unit = Pn / (wall / 1e3), "placements/s"
        metric = "Memory Heuristic II evaluations/sec (Eq. 6 per partition), 1 MI355X"
        workload = (f"Eq. 6 balance of {Pn} placements of the refinement loop (1% of ops moved "
                    f"per placement) on the {graph_desc}, {K} partitions, node kinds from the "
                    f"graph (variables residual, their optimiser updates reference nodes)")
        if budget > 0:
            print("[bench] timing the oracle ...", file=sys.stderr, flush=True)
            from oracle.memory_balance import memory_balance
            n, dt = 0, 0.0
            while n < Pn and dt < budget:
                pls = W.materialize_placements(sched, n, min(64, Pn - n))
                t0 = time.perf_counter()
                for q in range(pls.shape[0]):
                    memory_balance(V, g.mem, kind_h, tgt_h, pls[q], K)
                dt += time.perf_counter() - t0
                n += pls.shape[0]
            cpu = {"value": round(n / dt, 3), "unit": unit, "cores": 1, "kind": "oracle",
                   "sample": f"first {n} placements of the same loop, {dt:.1f} s on one core "
                             f"of '{host_cpu_model()}'"}
    elif row in ("cluster_criticality", "span_work"):
        n_pri = 16
        primary = G.slice_primaries(n_pri)["primary"]
        prim_h = primary.cpu().numpy()
        free = np.nonzero(prim_h < 0)[0]
        if row == "cluster_criticality":
            cl_h = np.where(prim_h >= 0, prim_h, n_pri + np.cumsum(prim_h < 0) - 1)
            C = n_pri + free.size
            cl = dev(cl_h, torch.int32)
            crit = torch.empty(C, dtype=torch.int64, device="cuda")
            order = torch.empty(C, dtype=torch.int32, device="cuda")
            fn = lambda: P.pardnn_cluster_criticality(G.handle, cl, C, crit, order)
            wall, k_ms, kname = time_calls(P, G, fn, args.steps, args.warmup)
            roof = hbm_roofline(kname, k_ms, algorithmic_bytes_tb_single(V, E), sweep_note)
            value, unit = C / (wall / 1e3), "clusters/s"
            metric = "cluster criticality rankings/sec (clusters ranked), 1 MI355X"
            workload = (f"criticality and order of {C} clusters (the {n_pri} primaries of "
                        f"slicing, every other node on its own) on the {graph_desc}")
            if budget > 0:
                print("[bench] timing the oracle ...", file=sys.stderr, flush=True)
                from oracle.clusters import cluster_criticality
                t0, reps = time.perf_counter(), 0
                while reps < 1 or time.perf_counter() - t0 < budget:
                    cluster_criticality(V, g.src, g.dst, g.comp, g.edge_cost, cl_h, C)
                    reps += 1
                dt = time.perf_counter() - t0
                cpu = {"value": round(reps * C / dt, 1), "unit": unit, "cores": 1,
                       "kind": "oracle",
                       "sample": f"{reps} full calls ({C} clusters each), {dt:.1f} s on one "
                                 f"core of '{host_cpu_model()}'"}
        else:
            Kp = n_pri
            cl_h = np.full(V, -1, np.int64)
            cl_h[free] = np.arange(free.size)
            C = int(free.size)
            cl = dev(cl_h, torch.int32)
            lab = primary
            iota = torch.arange(V, dtype=torch.int32, device="cuda")
            tl = torch.empty(V, dtype=torch.int64, device="cuda")
            bl = torch.empty(V, dtype=torch.int64, device="cuda")
            m = torch.empty(1, dtype=torch.int64, device="cuda")
            P.pardnn_tb_levels(G.handle, iota, tl, bl, m)
            i64 = dict(dtype=torch.int64, device="cuda")
            lo, hi = torch.empty(C, **i64), torch.empty(C, **i64)
            work, comm = torch.empty((C, Kp), **i64), torch.empty((C, Kp), **i64)
            choice = torch.empty(C, dtype=torch.int32, device="cuda")
            fn = lambda: P.pardnn_span_work(G.handle, lab, Kp, cl, C, tl, lo, hi, work, comm,
                                            choice)
            wall, k_ms, kname = time_calls(P, G, fn, args.steps, args.warmup)
            roof = hbm_roofline(kname, k_ms, algorithmic_bytes_span_work(V, E, C, Kp),
                                "whole call: node pass, two radix sorts, a scan, spans, "
                                "communication table, queries, choice")
            value, unit = C / (wall / 1e3), "clusters/s"
            metric = "Eq. 2 span-work queries/sec (clusters answered), 1 MI355X"
            workload = (f"Eq. 2 terms and choice of {C} secondary clusters (every node "
                        f"outside the {Kp} slicing primaries on its own) against the {Kp} "
                        f"primaries as partitions, tl with every edge paying, on the "
                        f"{graph_desc}")
            if budget > 0:
                from oracle.span_work import span_work
                import oracle
                print("[bench] timing the oracle ...", file=sys.stderr, flush=True)
                tl_h = oracle.tb_levels(V, g.src, g.dst, g.comp, g.edge_cost, np.arange(V))[0]
                lab_h = prim_h
                span_work(V, g.src, g.dst, g.comp, g.edge_cost, lab_h, Kp, cl_h, C, tl_h,
                          clusters=[0])
                t0 = time.perf_counter()
                span_work(V, g.src, g.dst, g.comp, g.edge_cost, lab_h, Kp, cl_h, C, tl_h,
                          clusters=[])
                setup = time.perf_counter() - t0
                # the per-cluster cost from a sample large enough to stand
                # above the noise of the setup time; the sample size then
                # follows from the budget, capped so a wrong estimate cannot
                # run away
                probe = min(C, 64)
                t1 = time.perf_counter()
                span_work(V, g.src, g.dst, g.comp, g.edge_cost, lab_h, Kp, cl_h, C, tl_h,
                          clusters=np.linspace(0, C - 1, probe).astype(np.int64))
                per = max((time.perf_counter() - t1 - setup) / probe, 1e-4)
                n = max(8, min(C, 1024, int(max(budget - 2 * setup, 1) / per)))
                rows = np.linspace(0, C - 1, n).astype(np.int64)
                t0 = time.perf_counter()
                span_work(V, g.src, g.dst, g.comp, g.edge_cost, lab_h, Kp, cl_h, C, tl_h,
                          clusters=rows)
                dt = time.perf_counter() - t0
                cpu = {"value": round(n / dt, 2), "unit": unit, "cores": 1, "kind": "oracle",
                       "sample": f"{n} of the {C} clusters, evenly spaced, {dt:.1f} s on one "
                                 f"core of '{host_cpu_model()}'"}
    elif row == "slicing":
        Ks = 16
        stride = max(L, 1)
        primary = torch.empty(V, dtype=torch.int32, device="cuda")
        paths = torch.empty((Ks, stride), dtype=torch.int32, device="cuda")
        plen = torch.empty(Ks, dtype=torch.int32, device="cuda")
        ms = torch.empty(Ks, dtype=torch.int64, device="cuda")
        fn = lambda: P.pardnn_slice_primaries(G.handle, Ks, primary, paths, stride, plen, ms)
        wall, k_ms, kname = time_calls(P, G, fn, args.steps, args.warmup)
        roof = hbm_roofline(kname, k_ms, algorithmic_bytes_tb_single(V, E),
                            sweep_note + "; the timed launch is the last round's sweep")
        value, unit = Ks / (wall / 1e3), "rounds/s"
        metric = "graph slicing rounds/sec (Alg. 1 primaries), 1 MI355X"
        workload = f"{Ks} slicing rounds (Alg. 1 primaries) on the {graph_desc}"
        if budget > 0:
            print("[bench] timing the oracle ...", file=sys.stderr, flush=True)
            from oracle.slicing import slice_primaries
            t0, reps = time.perf_counter(), 0
            while reps < 1 or time.perf_counter() - t0 < budget:
                slice_primaries(V, g.src, g.dst, g.comp, g.edge_cost, Ks)
                reps += 1
            dt = time.perf_counter() - t0
            cpu = {"value": round(reps * Ks / dt, 3), "unit": unit, "cores": 1,
                   "kind": "oracle",
                   "sample": f"{reps} runs of the same {Ks} rounds, {dt:.1f} s on one core of "
                             f"'{host_cpu_model()}'"}
    elif row == "slice_graph":
        Ks = 16
        i32 = dict(dtype=torch.int32, device="cuda")
        cluster = torch.empty(V, **i32)
        off = torch.empty(V + Ks + 1, **i32)
        nodes = torch.empty(V, **i32)
        n_cl = torch.empty(1, **i32)
        ms = torch.empty(Ks, dtype=torch.int64, device="cuda")
        fn = lambda: P.pardnn_slice_graph(G.handle, Ks, cluster, off, nodes, n_cl, ms)
        wall, k_ms, kname = time_calls(P, G, fn, args.steps, args.warmup)
        n_clusters = int(n_cl.item())
        roof = hbm_roofline(kname, k_ms, algorithmic_bytes_secondary(V, E),
                            "the timed launches are the secondary clusters (priority sort, "
                            "then one wave following one dependent step per node); their "
                            "bound is latency")
        value, unit = 1e3 / wall, "slicings/s"
        metric = "graph slicings/sec (Alg. 1 in full: K primaries, then the secondary clusters), 1 MI355X"
        workload = (f"graph slicing with {Ks} primaries and the secondary walk on stale "
                    f"priorities ({n_clusters} clusters in all) on the {graph_desc}")
        if budget > 0:
            print("[bench] timing the oracle ...", file=sys.stderr, flush=True)
            from oracle.slicing import slice_all
            t0, reps = time.perf_counter(), 0
            while reps < 1 or time.perf_counter() - t0 < budget:
                slice_all(V, g.src, g.dst, g.comp, g.edge_cost, Ks)
                reps += 1
            dt = time.perf_counter() - t0
            cpu = {"value": round(reps / dt, 4), "unit": unit, "cores": 1, "kind": "oracle",
                   "sample": f"{reps} full slicings, {dt:.1f} s on one core of "
                             f"'{host_cpu_model()}'"}
    else:
        raise ValueError(row)

    print(f"[bench] {row}: {wall:.3f} ms/call, {value:.1f} {unit}", file=sys.stderr, flush=True)
    line = {
        "metric": metric, "value": round(value, 3), "unit": unit, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(wall, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int64",
        "data": "synthetic", "config": {"workload": workload, "V": V, "E": E, "levels": L},
        "roofline": roof, "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    G.close()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--n-place", type=int, default=1000)
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline (0: skip)")
    ap.add_argument("--no-single", action="store_true",
                    help="skip the single-placement latency report")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy three times (scale reference for the "
                         "FETCH_SIZE / WRITE_SIZE counters) and exit")
    ap.add_argument("--row", choices=ROWS, default="refinement",
                    help="refinement (default): the evaluator's refinement loop; the others "
                         "measure the rows after it on the same graph")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the evaluator has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        return 2
    # the CPU baseline runs beside the GPU work, on a core of its own, and is
    # started before anything touches the GPU
    child = None
    if args.row in ("refinement", "single") and not args.copy_calibration:
        child = start_cpu_baseline(args.row, args.cpu_budget, 2, args.n_place)

    import numpy as np
    import torch

    import paper_2008_08636_amd as P
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.copy_calibration:
        a = torch.ones(1 << 28, dtype=torch.int32, device="cuda")  # 1 GiB
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print("copied 1 GiB three times", file=sys.stderr, flush=True)
        return 0
    if args.row == "single":
        return bench_single(args, child)
    if args.row != "refinement":
        return bench_row(args, args.row)
    P.load_library()
    dev = lambda x, dt: torch.as_tensor(np.ascontiguousarray(x), dtype=dt).cuda()

    g = W.make_config(2)
    sched = W.config4_moves(g, n_place=args.n_place)
    V, E, K = g.n_nodes, g.n_edges, g.n_labels
    print(f"[bench] graph V={V} E={E}; {sched.n_place} placements, "
          f"{int(sched.ptr[1])} moves each", file=sys.stderr, flush=True)

    # the first launches load the library's code objects: warm the runtime on
    # a small graph so that structure_ms measures the structure build alone
    g0 = W.make_config(0)
    G0 = P.Graph(g0.n_nodes, g0.src, g0.dst, g0.comp, g0.edge_cost, g0.mem)
    P.pardnn_levelize(G0.handle)
    G0.close()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    G = P.Graph(V, g.src, g.dst, g.comp, g.edge_cost, g.mem)
    L = P.pardnn_levelize(G.handle)
    torch.cuda.synchronize()
    structure_ms = (time.perf_counter() - t0) * 1e3

    base = dev(sched.base, torch.int32)
    ptr = dev(sched.ptr, torch.int64)
    node = dev(sched.node, torch.int32)
    lab = dev(sched.label, torch.int32)
    cap = dev(g.capacity, torch.int64)
    Pn = sched.n_place
    out = {
        "tl": torch.empty((V, Pn), dtype=torch.int64, device="cuda"),
        "bl": torch.empty((V, Pn), dtype=torch.int64, device="cuda"),
        "makespan": torch.empty(Pn, dtype=torch.int64, device="cuda"),
        "crit": torch.empty((V, Pn), dtype=torch.uint8, device="cuda"),
        "path": torch.empty((Pn, L), dtype=torch.int32, device="cuda"),
        "path_len": torch.empty(Pn, dtype=torch.int32, device="cuda"),
        "label_mem": torch.empty((Pn, K), dtype=torch.int64, device="cuda"),
        "overflow": torch.empty((Pn, K), dtype=torch.int64, device="cuda"),
    }
    P.pardnn_set_timing(G.handle, True)
    # argument errors found on the device are taken after the timed steps
    # instead of after each call, so that the steps run back to back
    P.pardnn_set_deferred_errors(G.handle, True)

    def step():
        P.pardnn_evaluate_moves(G.handle, base, Pn, ptr, node, lab, K, cap, out["tl"], out["bl"],
                                out["makespan"], out["crit"], out["path"], L,
                                out["path_len"], out["label_mem"], out["overflow"])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    kernel_ms = []
    kernel_name = ""
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
        kernel_name, ms = P.pardnn_get_timing(G.handle)
        kernel_ms.append(ms)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = dt * 1e3 / args.steps
    evals_per_s = Pn / (ms_per_step / 1e3)
    gteps = Pn * 2 * E / (ms_per_step / 1e3) / 1e9
    print(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step, {evals_per_s:.0f} eval/s, "
          f"{gteps:.2f} GTEPS", file=sys.stderr, flush=True)

    # the same loop keeping only the per-placement results (makespan, path,
    # label sums, overflows): tl / bl and the critical flags are still
    # computed but not written out -- reported beside the full evaluation
    lean_ms = None
    if args.steps > 0:
        def lean():
            P.pardnn_evaluate_moves(G.handle, base, Pn, ptr, node, lab, K, cap, None, None,
                                    out["makespan"], None, out["path"], L, out["path_len"],
                                    out["label_mem"], out["overflow"])
        lean()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            lean()
        torch.cuda.synchronize()
        lean_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        print(f"[bench] per-placement results only: {lean_ms:.3f} ms/step", file=sys.stderr,
              flush=True)
    # the same loop without label sums: the labels are then unchecked, and
    # whether they fit the packed sweep (below the hint K) is decided on the
    # device
    nolab_ms = None
    if args.steps > 0:
        def nolab():
            P.pardnn_evaluate_moves(G.handle, base, Pn, ptr, node, lab, K, None, out["tl"],
                                    out["bl"], out["makespan"], out["crit"], out["path"], L,
                                    out["path_len"], None, None)
        nolab()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            nolab()
        torch.cuda.synchronize()
        nolab_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        print(f"[bench] without label sums: {nolab_ms:.3f} ms/step", file=sys.stderr, flush=True)
    P.pardnn_take_errors(G.handle)   # raises if any step found an argument error
    P.pardnn_set_deferred_errors(G.handle, False)

    k_ms = float(np.mean(kernel_ms))
    alg = algorithmic_bytes_sweep(V, E, Pn)
    achieved = alg / (k_ms / 1e3) / 1e9
    step_alg = algorithmic_bytes_batch(V, E, Pn)
    workload_key = f"c4_transformer_V{V}_E{E}_P{Pn}"
    traffic = load_traffic(kernel_name, workload_key)
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": kernel_name, "kernel_ms": round(k_ms, 4),
                "algorithmic_bytes_per_launch": alg,
                "step": {"algorithmic_bytes": step_alg,
                         "achieved": round(step_alg / (ms_per_step / 1e3) / 1e9, 2),
                         "frac": round(step_alg / (ms_per_step / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}}

    single = None
    if not args.no_single:
        pl = dev(g.placement, torch.int32)
        tl = torch.empty(V, dtype=torch.int64, device="cuda")
        bl = torch.empty(V, dtype=torch.int64, device="cuda")
        m = torch.empty(1, dtype=torch.int64, device="cuda")
        ts = []
        for i in range(6):
            P.pardnn_tb_levels(G.handle, pl, tl, bl, m)
            if i >= 1:
                ts.append(P.pardnn_get_timing(G.handle)[1])
        torch.cuda.synchronize()
        tb_ms = float(np.median(ts))
        single = {"workload": "one placement of the same graph (pardnn_tb_levels)",
                  "kernel": P.pardnn_get_timing(G.handle)[0], "tb_levels_ms": round(tb_ms, 4),
                  "levels": L,
                  "tau_us_per_level": round(tb_ms * 1e3 / max(L, 1), 4),
                  "gteps": round(2 * E / (tb_ms / 1e3) / 1e9, 4)}
        print(f"[bench] single placement t+b: {tb_ms:.3f} ms over {L} levels", file=sys.stderr,
              flush=True)

    cpu = None
    if child is not None:
        print("[bench] waiting for the CPU oracle timing ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline_line(finish_cpu_baseline(child, 4 * args.cpu_budget + 120), E,
                                "the same refinement loop")

    line = {
        "metric": METRIC,
        "value": round(gteps, 4),
        "unit": "GTEPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": (f"refinement loop: {Pn} successive placements (1% of ops moved per "
                         f"placement) of the transformer-shaped training DAG, 48 blocks, "
                         f"V={V}, E={E}, {L} levels, {K} labels; full evaluation of each"),
            "V": V, "E": E, "levels": L, "n_place": Pn, "labels": K,
            "moves_per_placement": int(sched.ptr[1]),
        },
        "evals_per_s": round(evals_per_s, 1),
        "results_only": (None if lean_ms is None else
                         {"ms_per_step": round(lean_ms, 4),
                          "evals_per_s": round(Pn / (lean_ms / 1e3), 1),
                          "note": "same loop; tl, bl and critical flags computed but not "
                                  "written out (makespan, path, label sums, overflows kept)"}),
        "no_label_sums": (None if nolab_ms is None else
                          {"ms_per_step": round(nolab_ms, 4),
                           "evals_per_s": round(Pn / (nolab_ms / 1e3), 1),
                           "note": "same loop without label sums (every other output written); "
                                   "the labels, hinted to lie below K, are checked on the "
                                   "device, which picks the packed sweep"}),
        "structure_ms": round(structure_ms, 2),
        "roofline": roofline,
        "single": single,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    G.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
