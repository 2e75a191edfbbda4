"""Write SHA-256 digests of the oracle's full-size outputs to full_digests.json.

    python tests/golden/make_full_digests.py [--jobs N] [--only NAME ...]

Calls only the CPU oracle (oracle/) on the seeded full-size workloads
(paper_2609_27203_amd/workloads.py draws the inputs; it holds no evaluation
arithmetic).  Large fixpoints are computed in batches of first-key values
through the oracle's `restrict` argument; this is exact where the first head
column passes unchanged from the recursive atom into the head (path(X,.),
dist(S,.)), because then the rows of one first key never depend on another
key's rows.  Batches cover ascending, disjoint ranges of first keys, so their
canonical outputs concatenate into the canonical output of the whole
relation.

Digest of a relation: SHA-256 over its rows in ascending lexicographic order
(signed int32 keys), each row as its columns' 4-byte little-endian images
(int32 as is, float32 by its bits) one after another.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import evaluate  # noqa: E402
from paper_2609_27203_amd import workloads as W  # noqa: E402

OUT = os.path.join(HERE, "full_digests.json")


def row_bytes(cols) -> bytes:
    """Rows in the given order, each as its columns' 4-byte images."""
    return np.stack([np.ascontiguousarray(c).view(np.uint32) for c in cols], axis=1).astype("<u4").tobytes()


def _tc_uniform():
    wl = W.tc_uniform()
    res = evaluate(wl.rules, wl.edb, wl.idb)
    cols = res.relations["path"][1]
    return wl, {"path": [cols]}, {"path_sizes": res.sizes["path"]}


def _sssp_batch(sources):
    wl = W.sssp()
    sub = dict(wl.edb)
    sub["source"] = (("i32",), [np.asarray(sources, np.int32)])
    return evaluate(wl.rules, sub, wl.idb).relations["dist"][1]


def _rmat_batch(keys):
    wl = W.tc_rmat()
    res = evaluate(W.TC_COUNT_RULES, wl.edb, wl.idb, restrict={"path": (0, np.asarray(keys, np.int32))})
    return res.relations["path"][1], res.relations["reach_count"][1], res.sizes["path"]


def _sg():
    wl = W.same_generation()
    res = evaluate(wl.rules, wl.edb, wl.idb)
    return wl, {"sg": [res.relations["sg"][1]]}, {"sg_sizes": res.sizes["sg"]}


def _batched(fn, batches, jobs):
    with ProcessPoolExecutor(jobs) as ex:
        out = []
        for i, r in enumerate(ex.map(fn, batches)):
            out.append(r)
            print(f"  batch {i + 1}/{len(batches)} done", flush=True)
        return out


def compute(name, jobs):
    if name == "tc_uniform":
        return _tc_uniform()
    if name == "same_generation":
        return _sg()
    if name == "sssp":
        wl = W.sssp()
        src = np.sort(wl.edb["source"][1][0])
        parts = _batched(_sssp_batch, [src[i:i + 4] for i in range(0, len(src), 4)], jobs)
        return wl, {"dist": parts}, {}
    if name == "tc_rmat_count":
        wl = W.tc_rmat()
        keys = np.unique(wl.edb["edge"][1][0])   # a first key with no out-edge derives nothing
        parts = _batched(_rmat_batch, [keys[i:i + 128] for i in range(0, len(keys), 128)], jobs)
        # per-application sizes of the whole relation: the batches' sizes added
        # up, each batch holding its last size once its own fixpoint is reached
        n_it = max(len(p[2]) for p in parts)
        sizes = [sum(p[2][min(k, len(p[2]) - 1)] for p in parts) for k in range(n_it)]
        return wl, {"path": [p[0] for p in parts], "reach_count": [p[1] for p in parts]}, {"path_sizes": sizes}
    raise KeyError(name)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=4)
    ap.add_argument("--only", nargs="*", default=None)
    args = ap.parse_args()
    names = args.only or ["tc_uniform", "sssp", "same_generation", "tc_rmat_count"]
    record = json.load(open(OUT)) if os.path.exists(OUT) else {}
    for name in names:
        t0 = time.time()
        print(f"{name}: evaluating", flush=True)
        wl, rels, extra = compute(name, args.jobs)
        entry = {"inputs_sha256": wl.digest(), "relations": {}, **extra}
        for rel, parts in rels.items():
            h = hashlib.sha256()
            rows = 0
            for cols in parts:
                h.update(row_bytes(cols))
                rows += len(cols[0])
            entry["relations"][rel] = {"rows": rows, "sha256": h.hexdigest()}
        entry["oracle_seconds"] = round(time.time() - t0, 1)
        record[name] = entry
        print(f"{name}: {entry}", flush=True)
        json.dump(record, open(OUT, "w"), indent=1, sort_keys=True)


if __name__ == "__main__":
    main()
