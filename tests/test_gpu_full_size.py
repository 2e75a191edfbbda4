"""Full-size parity: every row of the five full-size workloads, in the
launch configuration the benchmark times (default options, index mode 0)
and with every derived relation in hash tables (index mode 1: the generic
keyed-table paths and their batched rounds).

Each result is decided twice, by independent routes:
* a certificate from a textbook routine computed here on the CPU
  (tests/certificates.py): breadth-first search from every node for the
  closures (rows, counts and per-pass delta sizes), the binary32 Bellman
  equations for shortest paths, the float64 forward pass for logsumexp, the
  closed form for same generation;
* the CPU oracle's own full-size output, as SHA-256 digests written by
  tests/golden/make_full_digests.py (which calls only the oracle), compared
  with the digest of the engine's rows -- bit for bit; logsumexp values are
  not bit-exact, so there the oracle evaluates 32 sampled sources here.
"""
import json
import os

import numpy as np
import pytest

import certificates as CERT
from helpers import LSE_TOL, assert_same_relation, engine_run, select_rows
from oracle import evaluate
from paper_2609_27203_amd import workloads as W

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]
DIGESTS = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "full_digests.json")))

_RUNS = {}
_CLOSURES = {}


def _full(name, workspace_gb, index_mode=0):
    """The engine's full-size result (one run per workload, index mode and
    session; a new run frees the previous one's rows)."""
    key = (name, index_mode)
    if key not in _RUNS:
        _RUNS.clear()
        wl = W.full_workloads()[name]()
        print(f"case: full {name} index_mode={index_mode} {wl.digest()[:12]}", flush=True)
        rels, stats, ctx = engine_run(wl, workspace_bytes=workspace_gb << 30, options={"index_mode": index_mode})
        ctx.close()
        _RUNS[key] = (wl, rels, stats)
    return _RUNS[key]


def _closure(name, n, src, dst):
    """Breadth-first-search closure matrix and level sizes (cached per workload)."""
    if name not in _CLOSURES:
        reached, levels = CERT.closure_bits(n, src, dst)
        _CLOSURES[name] = (CERT.reached_matrix(reached, n), levels)
    return _CLOSURES[name]


def _check_digest(name, wl, rels):
    rec = DIGESTS[name]
    assert rec["inputs_sha256"] == wl.digest(), f"{name}: inputs differ from the ones the digests were made for"
    for rel, exp in rec["relations"].items():
        assert len(rels[rel][0]) == exp["rows"], f"{rel}: {len(rels[rel][0])} rows, oracle {exp['rows']}"
        assert CERT.row_digest(rels[rel]) == exp["sha256"], f"{rel}: rows differ from the oracle's"


def _levels(sizes):
    return [sizes[0]] + [b - a for a, b in zip(sizes, sizes[1:])]


@pytest.mark.parametrize("index_mode", [0, 1])
def test_full_tc_uniform_every_row(index_mode):
    wl, rels, stats = _full("tc_uniform", 4, index_mode)
    src, dst = wl.edb["edge"][1]
    n = wl.params["n_nodes"]
    m, levels = _closure("tc_uniform", n, src, dst)
    CERT.check_closure_rows(m, *rels["path"])
    assert stats["delta_rows"] == levels and stats["iterations"] == len(levels) - 1
    _check_digest("tc_uniform", wl, rels)
    assert _levels(DIGESTS["tc_uniform"]["path_sizes"]) == levels


@pytest.mark.parametrize("index_mode", [0, 1])
def test_full_tc_rmat_count_every_row(index_mode):
    """The headline workload: all 128.9 M closure rows, all reach counts,
    the per-pass delta sizes and the derived-tuple count the benchmark
    reports."""
    wl, rels, stats = _full("tc_rmat_count", 32, index_mode)
    src, dst = wl.edb["edge"][1]
    n = 1 << wl.params["scale"]
    m, levels = _closure("tc_rmat_count", n, src, dst)
    CERT.check_closure_rows(m, *rels["path"])
    cnt = m.sum(axis=1)
    rc = rels["reach_count"]
    assert np.array_equal(rc[0], np.flatnonzero(cnt)) and np.array_equal(rc[1], cnt[cnt > 0])
    # the closure stratum's seed and passes, then the count stratum's rows
    assert stats["delta_rows"] == levels + [len(rc[0])] and stats["iterations"] == len(levels) - 1
    assert stats["derived_tuples"] == int(cnt.sum()) + int((cnt > 0).sum())
    _check_digest("tc_rmat_count", wl, rels)
    assert _levels(DIGESTS["tc_rmat_count"]["path_sizes"]) == levels


@pytest.mark.parametrize("index_mode", [0, 1])
def test_full_sssp_every_row(index_mode):
    """All 64 sources, bit for bit: the binary32 Bellman equations hold for
    every node, and the rows' digest is the oracle's."""
    wl, rels, _ = _full("sssp", 8, index_mode)
    src, dst, w = wl.edb["edge"][1]
    sources = np.sort(wl.edb["source"][1][0])
    CERT.bellman_check(wl.params["n_nodes"], src, dst, w, sources, *rels["dist"])
    _check_digest("sssp", wl, rels)


@pytest.mark.parametrize("index_mode", [0, 1])
def test_full_lse_every_row_forward_pass(index_mode):
    """All 256 sources: every row within 1e-5 * max(1, |ref|) of the float64
    forward pass, and exactly the (source, node) pairs joined by a path."""
    wl, rels, _ = _full("lse_dag", 8, index_mode)
    src, dst, w = wl.edb["edge"][1]
    L, K = wl.params["n_layers"], wl.params["width"]
    sources = np.sort(wl.edb["source"][1][0])
    total = CERT.forward_scores(L * K, src, dst, w, sources, L)
    worst = CERT.check_scores(total, sources, *rels["score"], tol=LSE_TOL)
    print(f"lse worst error / max(1, |ref|): {worst:.3g}", flush=True)


@pytest.mark.parametrize("part", [0, 1])
def test_full_lse_oracle_sampled_sources(part):
    """32 sources (two halves of 16) recomputed by the oracle, row by row."""
    wl, rels, _ = _full("lse_dag", 8)
    sources = wl.edb["source"][1][0]
    pick = np.sort(np.random.default_rng(3).choice(sources, 32, replace=False))[part::2]
    sub = dict(wl.edb)
    sub["source"] = (("i32",), [pick.astype(np.int32)])
    ref = evaluate(wl.rules, sub, wl.idb)
    assert_same_relation("score", wl.idb["score"], select_rows(rels["score"], 0, pick),
                         ref.relations["score"][1], " (oracle-sampled sources)", tol=(LSE_TOL, 1.0))


@pytest.mark.parametrize("index_mode", [0, 1])
def test_full_same_generation_every_row(index_mode):
    wl, rels, stats = _full("same_generation", 8, index_mode)
    x, y = rels["sg"]
    n = len(wl.params["depth"])
    keys = CERT.same_generation_keys(wl.edb["parent"][1][0], wl.params["depth"], wl.params["root"], n)
    assert np.array_equal(x.astype(np.int64) * n + y, keys)
    assert stats["derived_tuples"] == len(keys)
    _check_digest("same_generation", wl, rels)


def test_join_over_the_full_rmat_closure():
    """A later stratum joins the 128.9 M-row closure by its second column (an
    index built by sorting the whole relation, beyond 2^25 rows):
    into(Z) :- edge(_, Y), path(Z, Y) holds every node with a path row, since
    every path ends with an edge into its last node."""
    base = W.tc_rmat()
    rules = W.TC_RULES + "into(Z) :- edge(_,Y), path(Z,Y).\n"
    wl = W.Workload("rmat_later_join", rules, base.edb, {"path": ("i32", "i32"), "into": ("i32",)})
    print("case: full R-MAT closure joined by its second column", flush=True)
    rels, stats, ctx = engine_run(wl, workspace_bytes=32 << 30)
    ctx.close()
    src, dst = wl.edb["edge"][1]
    n = 1 << base.params["scale"]
    m = CERT.reached_matrix(CERT.closure_bits(n, src, dst)[0], n)
    CERT.check_closure_rows(m, *rels["path"])
    assert np.array_equal(rels["into"][0], np.flatnonzero(m.any(axis=1)).astype(np.int32))
