#!/usr/bin/env python3
"""Derived tuples/s to fixpoint on one MI355X.

Headline workload: transitive closure plus per-source reach count over an
R-MAT graph (2^14 nodes, 2^18 distinct edges, a=0.57 b=0.19 c=0.19 d=0.05,
seed 5), the largest of the engine's workloads.  One step is one complete
xl_fixpoint_run of the program (index build, seed, every semi-naive round,
the count stratum) with the input edges already resident in device memory;
derived relations are cleared before each step.

Prints one JSON line:
* value: derived tuples/s of the headline over the K timed steps;
* roofline: the headline's dominant kernel (the resident frontier kernel:
  every round of the closure).  `frac` is measured HBM traffic (rocprofv3
  FETCH_SIZE + WRITE_SIZE per launch, scaled by what a plain copy reads;
  stored in profiles/hbm_traffic.json and used only while the library's
  sources hash to the recorded value) over the kernel's event-timed launch
  duration and the 8 TB/s peak.  `frac_algorithmic` prices the same launch
  in the method's own units: 12 B per join-output candidate (each derived
  (x, z) times the out-degree of z, whether the kernel pushes or pulls) and
  24 B per new tuple.  `achievable_peak` is a 4 GiB device-to-device copy's
  rate on this device.  `on_chip` prices the kernel's examined candidates
  against the rate of its per-candidate step alone (csrc/ceiling.hip);
* per_config: the five workloads (and the triangle join), each 3 warm-up and
  10 timed runs (median, min, max; without the engine's per-launch events),
  with the same two fractions for its dominant kernel (launch durations
  from three further runs with the events) and for the whole run;
* cpu_baseline: the CPU oracle's semi-naive mode on a bounded sample of each
  workload, run in parallel on the host's cores (one process per core, each
  evaluating its own share of the sampled first keys).
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import platform
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2609_27203_amd", "csrc")
TRAFFIC = os.path.join(ROOT, "profiles", "hbm_traffic.json")
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published

CONFIGS = ["tc_uniform", "sssp", "lse_dag", "same_generation", "tc_rmat_count", "triangle"]

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

# dominant kernel family of each workload and the kernel the counters cover
FAMILY = {"tc_uniform": "front", "tc_rmat_count": "front", "sssp": "emit", "lse_dag": "pull",
          "same_generation": "gather", "triangle": "wcoj"}
KERNEL = {
    "front": "frontier_resident_k",
    "emit": "dense_min_tile_k",
    "pull": "dense_pull_k",
    "gather": "gather_by_a_k",
    "wcoj": "wcoj_probe_k",
}
KERNEL_DOC = {
    "front": "frontier_resident_k (every round of a first key in one workgroup, its row in LDS: delta "
             "expand or in-edge pull + membership test + merge)",
    "emit": "dense_min_tile_k (one workgroup per source and tile of targets, the tile's values in LDS: "
            "delta rows expanded through the (tile, Z) index, min folded in LDS)",
    "pull": "dense_pull_k (fold of each marked key's in-edges against the delta, keys ordered by target)",
    "gather": "gather_by_a_k (one workgroup per delta row A: the union of e2's Y lists over A's B bits "
              "built once in LDS, its nonzero words ORed into the head rows of A's X values with device "
              "atomics whose old values give the next delta words)",
    "wcoj": "wcoj_probe_k (count and materialize passes: each driver row's shorter Z list probed into "
            "the longer)",
}


def sources_sha256() -> str:
    """Hash of every source the library is built from (kernels and host code)."""
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        h.update(f.encode())
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()


def recorded_traffic(workload: str):
    """Measured HBM bytes per run of the workload's dominant kernel from the
    committed counter record, or None when the library's sources changed
    since it was measured."""
    if not os.path.exists(TRAFFIC):
        return None
    rec = json.load(open(TRAFFIC))
    if rec.get("sources_sha256") != sources_sha256():
        return None
    return rec["workloads"].get(workload)


# ---------------------------------------------------------------------------
# Algorithmic units of the method (join-output candidates C, new tuples).
# Per candidate: the matched edge's endpoint (4 B) and one membership probe of
# the packed key (8 B) for set heads; endpoint and weight (8 B) and a key +
# value probe (12 B) for value heads.  Per new tuple: written to the full
# relation (8 B), to the delta (8 B) and read from it next round (8 B).
# ---------------------------------------------------------------------------
def algorithmic(name, wl, rels, stats):
    """(run_bytes, kernel_bytes, units) for one fixpoint run."""
    if name in ("tc_uniform", "tc_rmat_count"):
        src, _ = wl.edb["edge"][1]
        z = rels["path"][1]
        n = int(max(src.max(), z.max())) + 1
        outdeg = np.bincount(src, minlength=n).astype(np.int64)
        # every derived (x, z) enters one delta and is joined with all edges out of z
        C = int((np.bincount(z, minlength=n).astype(np.int64) * outdeg).sum())
        N = len(z)
        run = 12 * C + 24 * N + (8 * N if "reach_count" in rels else 0)
        kern = 12 * C + 24 * stats["front_new"]
        return run, kern, {"C": C, "N": N, "new_in_kernel": stats["front_new"]}
    if name == "sssp":
        C = stats["emit_candidates"]       # each delta row joined with every out-edge (push)
        dsum = int(sum(stats["delta_rows"]))
        N = len(rels["dist"][0])
        return 20 * C + 24 * dsum + 12 * N, 20 * C + 24 * (dsum - stats["delta_rows"][0]), \
            {"C": C, "N": N, "sum_delta": dsum}
    if name == "lse_dag":
        src, _, _ = wl.edb["edge"][1]
        z = rels["score"][1]
        n = int(max(src.max(), z.max())) + 1
        outdeg = np.bincount(src, minlength=n).astype(np.int64)
        seed = int(outdeg[wl.edb["source"][1][0]].sum())
        C_rounds = int(outdeg[z].sum())   # on the layered DAG every key is in exactly one delta
        N = len(z)
        return 20 * (C_rounds + seed) + 24 * N, 20 * C_rounds + 24 * (N - stats["delta_rows"][0]), \
            {"C": C_rounds + seed, "N": N}
    if name == "same_generation":
        N = len(rels["sg"][0])            # every sg tuple is derived exactly once: C = N
        return 36 * N, 36 * (N - stats["delta_rows"][0]), {"C": N, "N": N}
    if name == "triangle":
        P, N = stats["wcoj_candidates"], len(rels["tri"][0])   # probes; 8 B each + 12 B per triple
        return 8 * P + 12 * N, 8 * P + 12 * N, {"probes": P, "N": N}
    raise KeyError(name)


def make_context(wl, args, xlh):
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
    return ctx, ctx.compile(wl.rules)


def fractions(name, wl, ctx, stats_list, ms_run):
    """Roofline figures of the dominant kernel and of the whole run."""
    fam = FAMILY[name]
    rels = {n: ctx.relations[n].read() for n in wl.idb}
    last = stats_list[-1]
    run_b, kern_b, units = algorithmic(name, wl, rels, last)
    k = len(stats_list)
    kern_ms = sum(s[fam + "_ms"] for s in stats_list) / k
    launches = sum(s[fam + "_launches"] for s in stats_list) / k
    out = {
        "kernel": KERNEL_DOC[fam], "kernel_ms_per_run": kern_ms, "launches_per_run": launches,
        "avg_launch_ms": kern_ms / max(launches, 1),
        "algorithmic_bytes_per_launch": kern_b / max(launches, 1),
        "achieved_algorithmic": kern_b / (kern_ms * 1e-3) / 1e9 if kern_ms > 0 else None,
        "units": units, "algorithmic_bytes_per_run": run_b,
        "run_frac_algorithmic": run_b / (ms_run * 1e-3) / 1e9 / HBM_PEAK_GBS,
    }
    out["frac_algorithmic"] = out["achieved_algorithmic"] / HBM_PEAK_GBS if out["achieved_algorithmic"] else None
    rec = recorded_traffic(name)
    if rec is not None and kern_ms > 0:
        per_run = rec["hbm_bytes_per_run"]
        out["traffic"] = per_run / max(launches, 1)
        out["achieved"] = per_run / (kern_ms * 1e-3) / 1e9
        out["frac"] = out["achieved"] / HBM_PEAK_GBS
        out["limiter"] = rec.get("limiter")
    else:
        out["traffic"] = out["achieved"] = out["frac"] = None
        out["limiter"] = "no counter record for the current sources"
    return out


def per_config(args, W, xlh, torch):
    """Each workload: warm-up runs, then the timed runs without the engine's
    per-launch events (ms per run), then three runs with them (the dominant
    kernel's launch durations)."""
    res = {}
    for name in CONFIGS:
        wl = W.full_workloads()[name]()
        ctx, prog = make_context(wl, args, xlh)
        ev, wall, stats = [], [], []
        ctx.set_option("profile", 0)
        for i in range(args.config_warmup + args.config_runs):
            for n in wl.idb:
                ctx.relations[n].clear()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            s = prog.run()
            torch.cuda.synchronize()
            if i >= args.config_warmup:
                wall.append(1e3 * (time.perf_counter() - t0))
                ev.append(s["ms_total"])
        ctx.set_option("profile", 1)
        for _ in range(3):
            for n in wl.idb:
                ctx.relations[n].clear()
            stats.append(prog.run())
        med = statistics.median(ev)
        f = fractions(name, wl, ctx, stats, med)
        derived = stats[-1]["derived_tuples"]
        if f["units"].get("C"):
            f["join_output_candidates_per_s"] = f["units"]["C"] / (med * 1e-3)
        res[name] = {"workload": DESCRIPTIONS[name], "derived_tuples": derived,
                     "iterations": stats[-1]["iterations"],
                     "ms_per_run": {"median": med, "min": min(ev), "max": max(ev),
                                    "wall_median": statistics.median(wall)},
                     "tuples_per_s": derived / (med * 1e-3), **f}
        print(f"{name}: {med:.3f} ms/run, {derived} tuples", file=sys.stderr, flush=True)
        ctx.close()
        del ctx, prog
        torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------------------
# On-chip ceiling of the frontier kernel (libxlh_ceiling.so): the rate of its
# per-candidate step (a 4-byte load from an L2-resident index column, a bit
# test and, when clear, an atomic OR in a 2 KB LDS row) with every load
# independent and no barrier, at the frontier kernel's workgroup size and LDS
# footprint (18,944 bytes of static LDS plus three 2 KB rows for a 16,384-node
# head), over the headline graph's edge target column.
# ---------------------------------------------------------------------------
FRONTIER_LDS_BYTES = 18944 + 3 * 2048


def copy_bandwidth(torch, gib=4):
    """Achievable HBM bandwidth on this device: a plain device-to-device copy
    of `gib` GiB (read + write bytes over the best of three event-timed runs)."""
    n = gib << 30
    x = torch.empty(n, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    x.fill_(1)
    best = 0.0
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        y.copy_(x)
        e1.record()
        e1.synchronize()
        best = max(best, 2 * n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del x, y
    torch.cuda.empty_cache()
    return best


def candidate_ceiling(col, torch):
    import ctypes as C
    L = C.CDLL(os.path.join(ROOT, "paper_2609_27203_amd", "libxlh_ceiling.so"))
    L.xlh_candidate_ceiling.argtypes = [C.c_void_p, C.c_uint64, C.c_uint32, C.c_int, C.c_size_t, C.c_void_p,
                                        C.c_void_p, C.POINTER(C.c_ulonglong), C.POINTER(C.c_float)]
    n = 1 << (len(col).bit_length() - 1)  # the largest power of two the column holds
    dcol = torch.from_numpy(np.ascontiguousarray(col[:n]).view(np.int32)).cuda()
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream()
    rates = {}
    for name, consecutive in (("random", 0), ("consecutive", 1)):
        best = 0.0
        for _ in range(4):  # the first run warms the column into L2
            cands, ms = C.c_ulonglong(0), C.c_float(0.0)
            rc = L.xlh_candidate_ceiling(C.c_void_p(dcol.data_ptr()), n, 128, consecutive, FRONTIER_LDS_BYTES,
                                         C.c_void_p(out.data_ptr()), C.c_void_p(stream.cuda_stream),
                                         C.byref(cands), C.byref(ms))
            if rc != 0:
                raise RuntimeError(f"xlh_candidate_ceiling failed with HIP error {rc}")
            best = max(best, cands.value / (ms.value * 1e-3))
        rates[name] = best
    return rates


# ---------------------------------------------------------------------------
# CPU baseline: the oracle's semi-naive mode, unchanged, on a bounded sample
# of each workload.
# Each worker process evaluates its own share of the sampled first keys
# (sources, nodes or driver values); the wall time spans the first start to
# the last end of the workers' evaluations.
# ---------------------------------------------------------------------------
CPU_SAMPLE = {  # first keys per worker (about one to two seconds of one core each)
    "tc_uniform": None,        # all sources, split over the workers
    "tc_rmat_count": 32,
    "sssp": 1,
    "lse_dag": 4,
    "same_generation": 800,
    "triangle": 4000,
}
_WL_CACHE = {}


def _cpu_job(job):
    name, part, nparts, seed = job
    from oracle.seminaive import evaluate_semi_naive as evaluate
    from paper_2609_27203_amd import workloads as W
    if name not in _WL_CACHE:
        _WL_CACHE[name] = W.full_workloads()[name]()
    wl = _WL_CACHE[name]
    rng = np.random.default_rng(seed)
    edb, restrict, rules, idb = dict(wl.edb), None, wl.rules, wl.idb
    per = CPU_SAMPLE[name]
    if name in ("tc_uniform", "tc_rmat_count"):
        keys = np.unique(wl.edb["edge"][1][0])
        pick = keys if per is None else rng.choice(keys, per * nparts, replace=False)
        mine = np.sort(pick)[part::nparts].astype(np.int32)
        restrict = {"path": (0, mine)}
    elif name in ("sssp", "lse_dag"):
        keys = wl.edb["source"][1][0]
        mine = np.sort(rng.choice(keys, min(len(keys), per * nparts), replace=False))[part::nparts]
        edb["source"] = (("i32",), [mine.astype(np.int32)])
    elif name == "same_generation":
        child, par = wl.edb["parent"][1]
        parent_of = dict(zip(child.tolist(), par.tolist()))
        start = np.sort(rng.choice(child, min(len(child), per * nparts), replace=False))[part::nparts]
        closed = set()
        for x in start.tolist():      # the sampled nodes and their ancestors (closed under the rules)
            while x in parent_of and x not in closed:
                closed.add(x)
                x = parent_of[x]
        mine = np.array(sorted(closed), np.int32)
        restrict = {"sg": (0, mine)}
    elif name == "triangle":
        types, (x, y) = wl.edb["r"]
        keys = np.unique(x)
        mine = np.sort(rng.choice(keys, min(len(keys), per * nparts), replace=False))[part::nparts]
        keep = np.isin(x, mine)
        edb["r"] = (types, [x[keep], y[keep]])
    t0 = time.time()
    res = evaluate(rules, edb, idb, restrict=restrict)
    t1 = time.time()
    return sum(len(r[1][0]) for r in res.relations.values()), len(mine), t0, t1


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baselines(names, workers):
    import multiprocessing as mp
    out = {}
    with mp.get_context("spawn").Pool(workers) as pool:
        for name in names:
            jobs = [(name, p, workers, 7) for p in range(workers)]
            parts = pool.map(_cpu_job, jobs, chunksize=1)
            rows = sum(p[0] for p in parts)
            keys = sum(p[1] for p in parts)
            wall = max(p[3] for p in parts) - min(p[2] for p in parts)
            out[name] = {"value": rows / wall, "unit": "derived tuples/s", "cores": workers, "kind": "oracle",
                         "sample": f"semi-naive evaluation (the oracle's Algorithm 1 mode, numpy) of {keys} "
                                   f"sampled first keys of the full workload, split over {workers} processes: "
                                   f"{rows} derived rows in {wall:.2f} s wall",
                         "host": f"{cpu_model()}; {len(os.sched_getaffinity(0))} cores visible"}
            print(f"cpu {name}: {rows / wall:.4g} tuples/s", file=sys.stderr, flush=True)
    return out


# ---------------------------------------------------------------------------
# Counter bookkeeping (rocprofv3 output -> profiles/hbm_traffic.json).
# ---------------------------------------------------------------------------
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


def _counter_rows(d, kernel=None):
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if kernel is None or kernel in r["Kernel_Name"]:
                rows.append(r)
    return rows


def _per_dispatch(rows, counter):
    """Counter value per dispatch (summed over the dimensions a row may be split into)."""
    acc = {}
    for r in rows:
        if r["Counter_Name"] == counter:
            acc[(r["Kernel_Name"], r["Dispatch_Id"])] = acc.get((r["Kernel_Name"], r["Dispatch_Id"]), 0.0) + \
                float(r["Counter_Value"])
    return acc


# Arguments of the profiled bench runs (the summaries quote the full commands).
TRACE_ARGS = "--steps 10 --warmup 3 --only-headline --no-cpu-baseline"
PMC_ARGS = "--steps 1 --warmup 0 --only-headline --no-cpu-baseline"
SQ_PASSES = ["SQ_WAVES SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_LDS SQ_INSTS_VALU "
             "SQ_INSTS_VMEM_RD SQ_INSTS_LDS GRBM_GUI_ACTIVE",
             "SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_SALU SQ_ACTIVE_INST_LDS TCC_HIT_sum TCC_MISS_sum"]


def profile_commands(d, name):
    """The rocprofv3 commands whose output summarize_counters / summarize_trace read."""
    kern = KERNEL[FAMILY[name]]
    cmds = [f"rocprofv3 --kernel-trace --stats -d {d}/{name}/trace -o run --output-format csv -- "
            f"python3 bench.py --workload {name} {TRACE_ARGS}"]
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        cmds.append(f"rocprofv3 --pmc {ctr} --kernel-include-regex {kern} -d {d}/{name}/{ctr} -o run "
                    f"--output-format csv -- python3 bench.py --workload {name} {PMC_ARGS}")
    for i, grp in enumerate(SQ_PASSES):
        cmds.append(f"rocprofv3 --pmc {grp} --kernel-include-regex {kern} -d {d}/{name}/sq/p{i + 1} -o run "
                    f"--output-format csv -- python3 bench.py --workload {name} {PMC_ARGS}")
    return cmds


def calibration_commands(d):
    return [f"rocprofv3 --pmc {ctr} -d {d}/calib/{ctr} -o run --output-format csv -- "
            f"python3 bench.py --copy-calibration" for ctr in ("FETCH_SIZE", "WRITE_SIZE")]


def summarize_trace(d):
    """Write profiles/<workload>_kernel_stats.md from <d>/<workload>/trace
    (rocprofv3 --kernel-trace --stats over 3 warm-up + 10 timed runs)."""
    runs = 13
    for name in CONFIGS:
        f = glob.glob(os.path.join(d, name, "trace", "**", "*kernel_stats.csv"), recursive=True)
        if not f:
            continue
        rows = list(csv.DictReader(open(f[0])))
        total = sum(float(r["TotalDurationNs"]) for r in rows)
        out = [f"# Kernel time of the {name} bench (rocprofv3 --kernel-trace --stats)", "",
               f"Workload: {DESCRIPTIONS[name]}.", "",
               "Command (repository root on the MI355X box, after `cd /tmp && export TMPDIR=/tmp`):", "",
               "    " + profile_commands(d, name)[0], "",
               f"The trace covers {runs} fixpoint runs (3 warm-up + 10 timed); 'ms per run' divides the "
               f"total by {runs}.  The totals also hold one-time work outside the runs (loading the inputs, "
               "and reading the result once after the timed runs: copies and the canonical sort of the "
               "read), so a kernel's per-call average is the figure to compare with the bench's "
               "event-timed launches.", "",
               "| kernel | calls | total ms | ms per run | avg ms | % |", "|---|---|---|---|---|---|"]
        for r in rows[:14]:
            tot = float(r["TotalDurationNs"]) * 1e-6
            out.append(f"| `{r['Name'][:80]}` | {r['Calls']} | {tot:.3f} | {tot / runs:.3f} | "
                       f"{float(r['AverageNs']) * 1e-6:.4f} | {float(r['Percentage']):.2f} |")
        out += ["", f"Sum over all kernels: {total * 1e-6:.2f} ms ({total * 1e-6 / runs:.3f} ms per run).", ""]
        path = os.path.join(ROOT, "profiles", f"{name}_kernel_stats.md")
        open(path, "w").write("\n".join(out))
        print(f"wrote {path}")


def summarize_counters(d):
    """Read <d>/calib/{FETCH_SIZE,WRITE_SIZE} and <d>/<workload>/{FETCH_SIZE,WRITE_SIZE,sq}
    (rocprofv3 --pmc output, one fixpoint run each) and write profiles/hbm_traffic.json."""
    scale = {}
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        vals = _per_dispatch(_counter_rows(os.path.join(d, "calib", ctr)), ctr)
        best = max(vals.values())          # the 1 GiB copy: largest dispatch
        scale[ctr] = best * 1024 / (1 << 30)
    # the hash of the sources the profiled runs used (written beside their output), else the tree's
    hfile = os.path.join(d, "sources_sha256.txt")
    sha = open(hfile).read().strip() if os.path.exists(hfile) else sources_sha256()
    rec = {"sources_sha256": sha, "copy_scale": scale, "workloads": {}}
    for name in CONFIGS:
        wd = os.path.join(d, name)
        if not os.path.isdir(wd):
            continue
        kern = KERNEL[FAMILY[name]]
        fetch = _per_dispatch(_counter_rows(os.path.join(wd, "FETCH_SIZE"), kern), "FETCH_SIZE")
        write = _per_dispatch(_counter_rows(os.path.join(wd, "WRITE_SIZE"), kern), "WRITE_SIZE")
        rd = sum(fetch.values()) * 1024 / scale["FETCH_SIZE"]
        wr = sum(write.values()) * 1024 / scale["WRITE_SIZE"]
        entry = {"kernel": kern, "dispatches_per_run": len(fetch), "hbm_read_bytes_per_run": rd,
                 "hbm_write_bytes_per_run": wr, "hbm_bytes_per_run": rd + wr}
        sq = _counter_rows(os.path.join(wd, "sq"), kern)
        if sq:
            tot = {}
            for r in sq:
                tot[r["Counter_Name"]] = tot.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            entry["sq"] = tot
            wc = tot.get("SQ_WAVE_CYCLES", 0.0)
            parts = []
            if wc:
                parts.append(f"waves wait {tot.get('SQ_WAIT_ANY', 0) / wc:.0%} of their cycles")
                if "SQ_WAIT_INST_LDS" in tot:
                    parts.append(f"{tot['SQ_WAIT_INST_LDS'] / wc:.0%} on LDS instructions")
            if tot.get("SQ_LDS_IDX_ACTIVE"):
                parts.append(f"LDS bank conflicts {tot.get('SQ_LDS_BANK_CONFLICT', 0) / tot['SQ_LDS_IDX_ACTIVE']:.0%}"
                             " of LDS index cycles")
            if tot.get("TCC_HIT_sum") is not None and tot.get("TCC_MISS_sum") is not None:
                h, m = tot["TCC_HIT_sum"], tot["TCC_MISS_sum"]
                parts.append(f"L2 hit rate {h / max(h + m, 1):.0%}")
            entry["limiter"] = "; ".join(parts) if parts else None
        rec["workloads"][name] = entry
    os.makedirs(os.path.dirname(TRAFFIC), exist_ok=True)
    json.dump(rec, open(TRAFFIC, "w"), indent=1, sort_keys=True)
    md = ["# HBM traffic and SQ counters of each workload's dominant kernel", "",
          "One fixpoint run per counter pass (rocprofv3 --pmc; repository root on the MI355X box, after "
          "`cd /tmp && export TMPDIR=/tmp`).  HBM bytes = FETCH_SIZE KiB * 1024 / "
          f"{scale['FETCH_SIZE']:.4f} + WRITE_SIZE KiB * 1024 / {scale['WRITE_SIZE']:.4f}: the factors a plain "
          "1 GiB device copy reads under the same counters.", "",
          f"Library sources sha256 at measurement: `{rec['sources_sha256']}` (bench.py uses the record only "
          "while the sources hash to it).", "", "Calibration commands:", ""]
    md += ["    " + c for c in calibration_commands(d)]
    md += ["", "| workload | kernel | dispatches per run | HBM read MB | HBM write MB | bound shown by the SQ/TCC counters |",
           "|---|---|---|---|---|---|"]
    for name, e in rec["workloads"].items():
        md.append(f"| {name} | `{e['kernel']}` | {e['dispatches_per_run']} | {e['hbm_read_bytes_per_run'] / 1e6:.1f} | "
                  f"{e['hbm_write_bytes_per_run'] / 1e6:.1f} | {e.get('limiter') or ''} |")
    md += ["", "Raw counter sums over one run (the dominant kernel's dispatches):", ""]
    for name, e in rec["workloads"].items():
        if "sq" in e:
            md.append(f"* {name}: " + ", ".join(f"{k} {v:.4g}" for k, v in sorted(e["sq"].items())))
    md += ["", "Commands per workload:", ""]
    for name in rec["workloads"]:
        md += ["    " + c for c in profile_commands(d, name)[1:]]
    open(os.path.join(ROOT, "profiles", "hbm_traffic.md"), "w").write("\n".join(md) + "\n")
    print(json.dumps(rec, indent=1, sort_keys=True))


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workspace-gb", type=float, default=24.0)
    ap.add_argument("--workload", default="tc_rmat_count",
                    help="headline workload, one of " + ", ".join(CONFIGS) + " (default tc_rmat_count)")
    ap.add_argument("--index-mode", type=int, default=0, help="0 auto, 1 hash tables only, 2 prefer dense")
    ap.add_argument("--option", action="append", default=[], metavar="KEY=VALUE",
                    help="extra engine option (xl_context_set_option), repeatable")
    ap.add_argument("--config-warmup", type=int, default=3)
    ap.add_argument("--config-runs", type=int, default=10)
    ap.add_argument("--only-headline", action="store_true", help="skip the per-config block")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-workers", type=int, default=0, help="0 = min(16, visible cores)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB copy (counter calibration for the traffic figure)")
    ap.add_argument("--summarize-counters", metavar="DIR",
                    help="write profiles/hbm_traffic.{json,md} from rocprofv3 --pmc output under DIR")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="write profiles/<workload>_kernel_stats.md from rocprofv3 --stats output under DIR")
    ap.add_argument("--print-profile-commands", metavar="DIR",
                    help="print the rocprofv3 commands that write the output the summaries read, and "
                         "record the library sources' hash in DIR/sources_sha256.txt")
    args = ap.parse_args()
    if args.print_profile_commands:
        os.makedirs(args.print_profile_commands, exist_ok=True)
        open(os.path.join(args.print_profile_commands, "sources_sha256.txt"), "w").write(sources_sha256() + "\n")
        for c in calibration_commands(args.print_profile_commands):
            print(c)
        for name in CONFIGS:
            for c in profile_commands(args.print_profile_commands, name):
                print(c)
        return
    if args.summarize_counters or args.summarize_trace:
        if args.summarize_counters:
            summarize_counters(args.summarize_counters)
        if args.summarize_trace:
            summarize_trace(args.summarize_trace)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the engine runs on one "
              "GPU only (the multi-GPU partitioning is a design, not code)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_27203_amd import workloads as W
    from paper_2609_27203_amd import xlh

    wl = W.full_workloads()[args.workload]()
    ctx, prog = make_context(wl, args, xlh)
    ceiling = candidate_ceiling(wl.edb["edge"][1][1], torch) if FAMILY[args.workload] == "front" else None

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
    f = fractions(args.workload, wl, ctx, stats, ms_per_step)
    ctx.close()
    del ctx, prog
    torch.cuda.empty_cache()

    achievable = copy_bandwidth(torch)
    roofline = {"bound": "hbm", "achieved": f["achieved"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": f["frac"], "traffic": f["traffic"],
                "achievable_peak": achievable,
                "frac_of_achievable": f["achieved"] / achievable if f["achieved"] else None,
                "achieved_algorithmic": f["achieved_algorithmic"], "frac_algorithmic": f["frac_algorithmic"],
                "algorithmic_bytes_per_launch": f["algorithmic_bytes_per_launch"],
                "kernel": f["kernel"], "launches_per_step": f["launches_per_run"],
                "avg_launch_ms": f["avg_launch_ms"], "limiter": f["limiter"]}
    if ceiling:
        front = sum(s["front_candidates"] for s in stats) / max(sum(s["front_ms"] for s in stats) * 1e-3, 1e-12)
        # the consecutive-address rate bounds the kernel; the random-address
        # rate (L2 line bandwidth: every 4-byte load its own 128-byte line)
        # is what it would reach with no locality at all
        roofline["on_chip"] = {
            "ceiling": "4-byte loads from an L2-resident index column, 64 consecutive per wavefront, each "
                       "followed by an LDS bit test-and-set; all loads independent, no barriers, the frontier "
                       "kernel's workgroup shape and LDS footprint",
            "unit": "candidates/s", "kernel": front, "peak": ceiling["consecutive"],
            "frac": front / ceiling["consecutive"],
            "random_address_rate": ceiling["random"], "kernel_over_random": front / ceiling["random"]}
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
                   "join_output_candidates": f["units"].get("C"), "parallelism": "none (1 GPU)"},
        "roofline": roofline,
    }
    if not args.only_headline:
        line["per_config"] = per_config(args, W, xlh, torch)
    if not args.no_cpu_baseline:
        workers = args.cpu_workers or min(16, len(os.sched_getaffinity(0)))
        names = [args.workload] if args.only_headline else CONFIGS
        cpu = cpu_baselines(names, workers)
        line["cpu_baseline"] = cpu[args.workload]
        if "per_config" in line:
            for name in names:
                line["per_config"][name]["cpu_baseline"] = cpu[name]
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    sys.path.insert(0, ROOT)
    main()
