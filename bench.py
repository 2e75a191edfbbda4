#!/usr/bin/env python3
"""Derived tuples/s to fixpoint on one MI355X.

Workload: transitive closure plus per-source reach count over an R-MAT graph
(2^14 nodes, 2^18 distinct edges, a=0.57 b=0.19 c=0.19 d=0.05, seed 5) -- the
largest of the engine's workloads.  One step is one complete
xl_fixpoint_run of the program (index build, seed, every semi-naive round,
the count stratum) with the input edges already resident in device memory;
derived relations are cleared before each step.

Prints one JSON line.  `roofline` covers the dominant kernel (for the
headline the resident frontier kernel: every round of the closure, delta
expand or in-edge pull + membership test + merge), timed live with HIP
events on the engine's stream; `cpu_baseline` times the CPU oracle on a
bounded sample of the same workload (the closure rows of a few sources).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published

DESCRIPTIONS = {
    "tc_uniform": "transitive closure, uniform random graph (1,000 nodes, 4,000 edges, seed 1)",
    "sssp": "multi-source shortest paths, min aggregate (100,000 nodes, 1,000,000 edges, 64 sources, seed 2)",
    "lse_dag": "probabilistic reachability, logsumexp aggregate (20 x 5,000 layered DAG, 8 out-edges, "
               "256 sources, seed 3)",
    "same_generation": "same generation over a 20,000-node forest (seed 4)",
    "tc_rmat_count": "R-MAT transitive closure + reach_count (2^14 nodes, 2^18 edges, seed 5)",
    "triangle": "three-way triangle join tri(X,Y,Z) :- r(X,Y), s(Y,Z), t(X,Z), three relations of 65,536 rows "
                "with a 161-value hot core and 8 hubs (seed 6)",
}


KERNELS = {
    "front": "frontier_resident_k (every round of a first key in one workgroup, its row in LDS: delta "
             "expand or in-edge pull + membership test + merge)",
    "emit": "stage_k / dense_min_tile_k (fused delta expand + probe + fold into the head)",
    "pull": "dense_pull_k (fold of each marked key's in-edges against the delta, keys ordered by target)",
    "wcoj": "wcoj_probe_k (count and materialize passes: each driver row's shorter Z list probed into the longer)",
    "gather": "gather_round_k (per head row X staged in LDS: the delta rows of X's A values pushed through e2, "
              "test-and-set in LDS, changed words written back)",
}

# Algorithmic bytes per unit of work (candidates, new tuples), counting only
# what the join/dedup/merge must move:
#   set heads: per candidate (a head tuple produced, or an edge examined) the
#     matched edge's endpoint (4 B) and one membership probe of the packed key
#     (8 B); per new tuple the key written to the full relation (8 B), the
#     delta row written (8 B) and read again by the next round (8 B);
#   value heads (min / logsumexp): per candidate the edge's endpoint and
#     weight (8 B) and a key + value probe (12 B); per new or improved key
#     24 B as above;
#   triangle join: per probe the probed Z value (4 B) and one membership
#     test in the other list (4 B); per output triple its three columns
#     written (12 B).
BYTES_PER_UNIT = {
    "tc_uniform": (12.0, 24.0),
    "tc_rmat_count": (12.0, 24.0),
    "same_generation": (12.0, 24.0),
    "sssp": (20.0, 24.0),
    "lse_dag": (20.0, 24.0),
    "triangle": (8.0, 12.0),
}


def _algorithmic_bytes(workload: str, candidates: float, new: float) -> float:
    per_cand, per_new = BYTES_PER_UNIT[workload]
    return per_cand * candidates + per_new * new


def dominant_kernel(stats: list, workload: str) -> dict:
    """The join kernel family with the largest event-timed share: frontier
    rounds (closure-shaped strata), the generic fused stage kernel, the
    segmented pull fold (sum / logsumexp over dense heads), the triangle
    join's probes, or gathered rounds (same generation's shape)."""
    ms = {k: sum(s[k + "_ms"] for s in stats) for k in KERNELS}
    k = max(ms, key=lambda f: ms[f])
    return {"family": k, "ms": ms[k],
            "launches": sum(s[k + "_launches"] for s in stats),
            "bytes": sum(_algorithmic_bytes(workload, s[k + "_candidates"], s[k + "_new"]) for s in stats)}


FRONTIER_SOURCES = ("frontier.hip", "device_util.h", "device_types.h")


def frontier_sources_sha256() -> str:
    """Hash of the sources the frontier kernel is compiled from."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2609_27203_amd", "csrc")
    for f in FRONTIER_SOURCES:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()


def recorded_traffic(workload: str):
    """HBM bytes per launch of the dominant kernel from the committed counter
    record, or None when the kernel's sources changed since it was measured."""
    root = os.path.dirname(os.path.abspath(__file__))
    rec = os.path.join(root, "profiles", "frontier_resident_rmat_traffic.json")
    if workload != "tc_rmat_count" or not os.path.exists(rec):
        return None
    r = json.load(open(rec))
    return r["hbm_bytes_per_launch"] if r.get("frontier_sources_sha256") == frontier_sources_sha256() else None


def copy_calibration():
    """A plain 1 GiB device copy, profiled to scale FETCH_SIZE / WRITE_SIZE to bytes."""
    import torch
    n = 1 << 30
    x = torch.ones(n, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(2):
        torch.add(x, 0, out=y)
    torch.cuda.synchronize()
    print(f"copied {n} bytes twice", flush=True)


def cpu_baseline(wl, n_sources: int, seed: int = 7) -> dict:
    from oracle import evaluate
    from paper_2609_27203_amd import workloads as W
    src = wl.edb["edge"][1][0]
    rng = np.random.default_rng(seed)
    pick = np.sort(rng.choice(np.unique(src), n_sources, replace=False)).astype(np.int32)
    idb = {"path": ("i32", "i32"), "reach_count": ("i32", "i32")}
    t0 = time.perf_counter()
    res = evaluate(W.TC_COUNT_RULES, wl.edb, idb, restrict={"path": (0, pick)})
    dt = time.perf_counter() - t0
    rows = sum(len(r[1][0]) for r in res.relations.values())
    return {"value": rows / dt, "unit": "derived tuples/s", "cores": 1, "kind": "oracle",
            "sample": f"naive evaluation restricted to the closure of {n_sources} sampled sources "
                      f"({rows} derived rows in {dt:.2f} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workspace-gb", type=float, default=24.0)
    ap.add_argument("--cpu-sources", type=int, default=160)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB copy (counter calibration for the traffic figure)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default="tc_rmat_count",
                    help="one of the engine's six workloads (the headline line uses tc_rmat_count)")
    ap.add_argument("--index-mode", type=int, default=0, help="0 auto, 1 hash tables only, 2 prefer dense")
    ap.add_argument("--option", action="append", default=[], metavar="KEY=VALUE",
                    help="extra engine option (xl_context_set_option), repeatable")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this engine "
              "(the multi-GPU partitioning is design only)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_27203_amd import workloads as W
    from paper_2609_27203_amd import xlh

    wl = W.full_workloads()[args.workload]()
    ctx = xlh.Context(device=0, workspace_bytes=int(args.workspace_gb * (1 << 30)))
    ctx.set_option("profile", 1)
    ctx.set_option("index_mode", args.index_mode)
    for kv in args.option:
        k, v = kv.split("=")
        ctx.set_option(k, int(v))
    for name, (types, cols) in wl.edb.items():
        ctx.relation(name, types).load(cols)
    for name, types in wl.idb.items():
        ctx.relation(name, types)
    prog = ctx.compile(wl.rules)

    def step():
        for name in wl.idb:
            ctx.relations[name].clear()
        return prog.run()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        stats.append(step())
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = 1e3 * dt / args.steps
    derived = stats[-1]["derived_tuples"]

    dk = dominant_kernel(stats, args.workload)
    achieved = dk["bytes"] / (dk["ms"] * 1e-3) / 1e9 if dk["ms"] > 0 else 0.0
    traffic = recorded_traffic(args.workload) if dk["family"] == "front" else None
    roofline = {
        "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": round(traffic) if traffic is not None else None,
        "kernel": KERNELS[dk["family"]],
        "launches_per_step": dk["launches"] / args.steps,
        "avg_launch_ms": dk["ms"] / max(dk["launches"], 1),
        "algorithmic_bytes_per_launch": dk["bytes"] / max(dk["launches"], 1),
    }
    line = {
        "metric": "derived tuples/sec to fixpoint (1 MI355X)",
        "value": derived / (ms_per_step * 1e-3),
        "unit": "derived tuples/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32", "data": "synthetic",
        "config": {"workload": DESCRIPTIONS[args.workload], "index_mode": args.index_mode,
                   "derived_tuples": derived, "iterations": stats[-1]["iterations"],
                   "candidates": stats[-1]["candidates_total"], "parallelism": "none (1 GPU)"},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline and args.workload == "tc_rmat_count":
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sources)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    main()
