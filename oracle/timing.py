"""Timing of the oracle for the CPU-baseline leg of ``bench.py``.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``bench.py``'s CPU-baseline
leg runs this module, as a child process started before the benchmark touches
the GPU. It times the oracle as it stands -- the same C source, built here
with ``gcc -O3 -march=native`` for the host it runs on -- single-threaded,
pinned to one core, on the same seeded workload the benchmark uses, and
prints one JSON line.

Modes:
  refinement  the first placements of the refinement loop on the transformer
              graph, each evaluated in full (levels, tl, bl, makespan,
              critical path, label memory); one timing per placement;
  single      one placement of each listed config, evaluated in full,
              repeatedly (the budget split evenly over the configs).
The reported time is the median over at least ``--min-reps`` timed
evaluations after one untimed warm-up, within ``--budget`` seconds.
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

NATIVE_LIB = os.path.join(HERE, "liboracle_native.so")


def build_native() -> str:
    """The oracle's C source compiled for this host's CPU (-march=native)."""
    tmp = NATIVE_LIB + f".tmp{os.getpid()}"
    subprocess.check_call(["gcc", "-O3", "-march=native", "-std=c99", "-fPIC", "-shared",
                           "-o", tmp, os.path.join(HERE, "pardnn_oracle.c")])
    os.replace(tmp, NATIVE_LIB)
    return NATIVE_LIB


def lscpu_model() -> str:
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--mode", choices=("refinement", "single"), default="refinement")
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--configs", default="0,1,2", help="single mode: configs to time")
    ap.add_argument("--n-place", type=int, default=1000)
    ap.add_argument("--budget", type=float, default=15.0)
    ap.add_argument("--min-reps", type=int, default=10)
    ap.add_argument("--core", type=int, default=-1, help="pin to this core (-1: leave)")
    args = ap.parse_args()
    if args.core >= 0:
        os.sched_setaffinity(0, {args.core})
    pinned = sorted(os.sched_getaffinity(0))

    import numpy as np

    import oracle
    import workloads as W

    oracle._lib = oracle.bind(build_native())
    host = {"pinned_cores": pinned, "nproc": os.cpu_count(), "cpu_model": lscpu_model(),
            "build": "gcc -O3 -march=native -std=c99"}

    def timed(g, labs):
        V = g.n_nodes

        def evaluate(lab):
            oracle.evaluate(V, g.src, g.dst, g.comp, g.edge_cost, g.mem, lab, g.n_labels,
                            g.capacity)

        times = []
        for lab in labs:
            t0 = time.perf_counter()
            evaluate(lab)
            times.append(time.perf_counter() - t0)
        return {"median_s": float(np.median(times)), "mean_s": float(np.mean(times)),
                "reps": len(times), "min_s": float(np.min(times)),
                "max_s": float(np.max(times)), "V": V, "E": g.n_edges}

    def one_time(g, lab):
        t = timed(g, [lab, lab])   # the first run is the warm-up
        return t["min_s"]

    if args.mode == "refinement":
        g = W.make_config(args.config)
        sched = W.config4_moves(g, n_place=args.n_place)
        first = W.materialize_placements(sched, 0, 1)[0]
        t1 = one_time(g, first)
        n = max(args.min_reps, min(sched.n_place, int(args.budget / max(t1, 1e-6))))
        n = min(n, sched.n_place)
        pls = W.materialize_placements(sched, 0, n)
        r = timed(g, [pls[p] for p in range(n)])
        r["what"] = f"first {n} of the {sched.n_place} placements of the refinement loop"
        r.update(host)
    else:
        configs = [int(c) for c in args.configs.split(",") if c.strip()]
        r = {"per_config": {}}
        for c in configs:
            g = W.make_config(c)
            t1 = one_time(g, g.placement)
            n = max(args.min_reps, int(args.budget / len(configs) / max(t1, 1e-6)))
            x = timed(g, [g.placement] * n)
            x["what"] = f"config {c}'s own placement, {n} times"
            r["per_config"][f"config{c}"] = x
        r.update(host)
    print(json.dumps(r), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
