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


def cpu_baseline(g, sched, budget_s: float):
    """The oracle as it stands, single-threaded, on the first placements of the
    same refinement loop (bounded by `budget_s` seconds of CPU work)."""
    import oracle
    import workloads as W

    oracle.build(force=False)
    first = W.materialize_placements(sched, 0, 1)[0]
    t0 = time.perf_counter()
    oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem, first, g.n_labels,
                    g.capacity)
    t1 = time.perf_counter() - t0
    n = max(1, min(sched.n_place, int(budget_s / max(t1, 1e-6))))
    pls = W.materialize_placements(sched, 0, n)
    t0 = time.perf_counter()
    for p in range(n):
        oracle.evaluate(g.n_nodes, g.src, g.dst, g.comp, g.edge_cost, g.mem, pls[p],
                        g.n_labels, g.capacity)
    dt = time.perf_counter() - t0
    return {
        "value": round(n * 2 * g.n_edges / dt / 1e9, 6),
        "unit": "GTEPS",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {n} of the {sched.n_place} placements of the same loop, each "
                  f"evaluated in full (tl, bl, makespan, critical path, label memory); "
                  f"{n / dt:.2f} evaluations/s over {dt:.1f} s on one core of "
                  f"'{host_cpu_model()}'",
    }


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
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the evaluator has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        return 2

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
    P.load_library()
    dev = lambda x, dt: torch.as_tensor(np.ascontiguousarray(x), dtype=dt).cuda()

    g = W.make_config(2)
    sched = W.config4_moves(g, n_place=args.n_place)
    V, E, K = g.n_nodes, g.n_edges, g.n_labels
    print(f"[bench] graph V={V} E={E}; {sched.n_place} placements, "
          f"{int(sched.ptr[1])} moves each", file=sys.stderr, flush=True)

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
    if args.cpu_budget > 0:
        print("[bench] timing the CPU oracle ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(g, sched, args.cpu_budget)

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
