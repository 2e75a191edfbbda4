"""CPU checks of the full-size certificates (tests/certificates.py): on reduced
workloads each one accepts the oracle's result and rejects a corrupted copy,
and the closure certificate's levels equal the oracle's per-iteration
growth."""
import hashlib
import os
import sys

import numpy as np
import pytest

import certificates as CERT
from oracle import evaluate
from paper_2609_27203_amd import workloads as W

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))


def _levels(ref, name):
    sizes = ref.sizes[name]
    return [sizes[0]] + [b - a for a, b in zip(sizes, sizes[1:])]


@pytest.mark.parametrize("name", ["tc_uniform", "tc_rmat_count"])
def test_closure_bits_equal_the_oracle(name):
    wl = W.small_workloads()[name]()
    src, dst = wl.edb["edge"][1]
    n = int(max(src.max(), dst.max())) + 1
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    reached, levels = CERT.closure_bits(n, src, dst, block=128)
    assert levels == _levels(ref, "path")
    m = CERT.reached_matrix(reached, n)
    x, y = ref.relations["path"][1]
    CERT.check_closure_rows(m, x, y)
    if name == "tc_rmat_count":
        rc = ref.relations["reach_count"][1]
        cnt = m.sum(axis=1)
        assert np.array_equal(rc[0], np.flatnonzero(cnt)) and np.array_equal(rc[1], cnt[cnt > 0])
    for bad in ((x[1:], y[1:]), (np.append(x, x[-1]), np.append(y, y[-1])), (x[::-1], y[::-1])):
        with pytest.raises(AssertionError):
            CERT.check_closure_rows(m, *bad)
    missing = np.flatnonzero(~m.ravel())[0]        # a pair that is not in the closure
    xx = np.append(x, missing // n).astype(np.int32)
    yy = np.append(y, missing % n).astype(np.int32)
    order = np.lexsort((yy, xx))
    with pytest.raises(AssertionError):
        CERT.check_closure_rows(m, xx[order], yy[order])


def test_bellman_check_accepts_the_oracle_and_rejects_changes():
    wl = W.small_workloads()["sssp"]()
    src, dst, w = wl.edb["edge"][1]
    sources = wl.edb["source"][1][0]
    n = wl.params["n_nodes"]
    s, y, d = evaluate(wl.rules, wl.edb, wl.idb).relations["dist"][1]
    CERT.bellman_check(n, src, dst, w, sources, s, y, d)
    i = len(d) // 2
    up = d.copy()
    up[i] = np.nextafter(up[i], np.float32(np.inf))
    down = d.copy()
    down[i] = np.nextafter(down[i], np.float32(0))
    for cols in ((s, y, up), (s, y, down), (s[1:], y[1:], d[1:])):
        with pytest.raises(AssertionError):
            CERT.bellman_check(n, src, dst, w, sources, *cols)


def test_forward_scores_accept_the_oracle_and_reject_changes():
    wl = W.small_workloads()["lse_dag"]()
    L, K = wl.params["n_layers"], wl.params["width"]
    src, dst, w = wl.edb["edge"][1]
    sources = wl.edb["source"][1][0]
    s, y, p = evaluate(wl.rules, wl.edb, wl.idb).relations["score"][1]
    total = CERT.forward_scores(L * K, src, dst, w, sources, L)
    assert CERT.check_scores(total, sources, s, y, p) < 1e-6
    off = p.copy()
    off[7] += 1e-4 * max(1.0, abs(float(off[7])))
    for cols in ((s, y, off), (s[1:], y[1:], p[1:])):
        with pytest.raises(AssertionError):
            CERT.check_scores(total, sources, *cols)


def test_same_generation_keys_equal_the_oracle():
    wl = W.small_workloads()["same_generation"]()
    child = wl.edb["parent"][1][0]
    n = len(wl.params["depth"])
    x, y = evaluate(wl.rules, wl.edb, wl.idb).relations["sg"][1]
    keys = CERT.same_generation_keys(child, wl.params["depth"], wl.params["root"], n)
    assert np.array_equal(keys, x.astype(np.int64) * n + y)


def test_row_digest_is_the_digest_script_definition():
    import make_full_digests as M
    cols = [np.array([3, -1, 7], np.int32), np.array([0.5, -2.0, 1e30], np.float32)]
    assert CERT.row_digest(cols) == hashlib.sha256(M.row_bytes(cols)).hexdigest()
    # int32 images little-endian, one row after another
    assert M.row_bytes([np.array([1, 2], np.int32), np.array([3, 4], np.int32)]) == \
        bytes([1, 0, 0, 0, 3, 0, 0, 0, 2, 0, 0, 0, 4, 0, 0, 0])


def test_stored_full_size_digests_agree_with_the_certificates():
    """The oracle's full-size outputs (digests written by
    golden/make_full_digests.py) equal what breadth-first search and the
    same-generation closed form give for the same inputs."""
    import json
    rec = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "full_digests.json")))
    for name in ("tc_uniform", "tc_rmat_count"):
        wl = W.full_workloads()[name]()
        assert rec[name]["inputs_sha256"] == wl.digest()
        src, dst = wl.edb["edge"][1]
        n = int(max(src.max(), dst.max())) + 1
        reached, levels = CERT.closure_bits(n, src, dst)
        m = CERT.reached_matrix(reached, n)
        x, y = (a.astype(np.int32) for a in np.nonzero(m))
        assert rec[name]["relations"]["path"] == {"rows": len(x), "sha256": CERT.row_digest([x, y])}
        sizes = rec[name]["path_sizes"]
        assert [sizes[0]] + [b - a for a, b in zip(sizes, sizes[1:])] == levels
        if name == "tc_rmat_count":
            cnt = m.sum(axis=1)
            rc = [np.flatnonzero(cnt).astype(np.int32), cnt[cnt > 0].astype(np.int32)]
            assert rec[name]["relations"]["reach_count"] == {"rows": len(rc[0]), "sha256": CERT.row_digest(rc)}
        del m, reached, x, y
    wl = W.same_generation()
    assert rec["same_generation"]["inputs_sha256"] == wl.digest()
    n = len(wl.params["depth"])
    keys = CERT.same_generation_keys(wl.edb["parent"][1][0], wl.params["depth"], wl.params["root"], n)
    cols = [(keys // n).astype(np.int32), (keys % n).astype(np.int32)]
    assert rec["same_generation"]["relations"]["sg"] == {"rows": len(keys), "sha256": CERT.row_digest(cols)}
