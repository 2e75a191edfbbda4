"""Pins for the CPU oracle: it is checked against things other than itself.

Each test fixes the oracle's output with an independent source of truth: the
paper's worked listings, closed forms, textbook graph algorithms (BFS, Floyd-
Warshall, Dijkstra), brute-force path enumeration and structural invariants.
"""
import heapq
import math
import os

import numpy as np
import pytest
import scipy.sparse as sp
from scipy.sparse import csgraph

from oracle import ConvergenceFailure, evaluate
from paper_2609_27203_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TC = W.TC_RULES
I2 = ("i32", "i32")


def _golden(name):
    rows = [tuple(int(x) for x in ln.split()) for ln in open(os.path.join(GOLDEN, name))
            if ln.strip() and not ln.startswith("#")]
    return sorted(rows)


def _rows(res, name):
    _, cols = res.relations[name]
    return sorted(zip(*[c.tolist() for c in cols]))


def _edges(src, dst):
    return {"edge": (I2, [np.asarray(src, np.int32), np.asarray(dst, np.int32)])}


# ---------------------------------------------------------------- worked examples
def test_listing_minimal_reach():
    rules = "reach(X, Y) :- edge(X, Y).\nreach(X, Z) :- reach(X, Y), edge(Y, Z)."
    res = evaluate(rules, _edges([1, 2, 3], [2, 3, 4]), {"reach": I2})
    assert _rows(res, "reach") == _golden("listing_minimal_reach.txt")
    assert sorted(y for x, y in _rows(res, "reach") if x == 1) == [2, 3, 4]


def test_listing_agg_degree():
    res = evaluate("degree(X, count(Y)) :- edge(X, Y).",
                   _edges([1, 1, 1, 2], [2, 3, 4, 3]), {"degree": I2})
    assert _rows(res, "degree") == _golden("listing_agg_degree.txt")


# ---------------------------------------------------------------- transitive closure
@pytest.mark.parametrize("n", [1, 2, 5, 17, 64])
def test_tc_chain_closed_form(n):
    src = np.arange(n - 1)
    res = evaluate(TC, _edges(src, src + 1), {"path": I2})
    got = _rows(res, "path")
    assert len(got) == n * (n - 1) // 2
    assert got == [(i, j) for i in range(n) for j in range(i + 1, n)]


@pytest.mark.parametrize("n", [1, 3, 8, 23])
def test_tc_cycle_closed_form(n):
    src = np.arange(n)
    res = evaluate(TC, _edges(src, (src + 1) % n), {"path": I2})
    got = _rows(res, "path")
    if n == 1:   # a single self-loop
        assert got == [(0, 0)]
    else:
        assert len(got) == n * n
        assert got == [(i, j) for i in range(n) for j in range(n)]


def _warshall(n, edges):
    reach = np.zeros((n, n), bool)
    for u, v in edges:
        reach[u, v] = True
    for k in range(n):
        reach |= reach[:, k:k + 1] & reach[k:k + 1, :]
    return sorted((int(i), int(j)) for i, j in zip(*np.nonzero(reach)))


def test_tc_all_graphs_on_three_nodes():
    pairs = [(u, v) for u in range(3) for v in range(3)]
    for mask in range(1 << len(pairs)):
        edges = [p for b, p in enumerate(pairs) if mask >> b & 1]
        if not edges:
            continue
        res = evaluate(TC, _edges(*zip(*edges)), {"path": I2})
        assert _rows(res, "path") == _warshall(3, edges), edges


@pytest.mark.parametrize("seed", range(12))
def test_tc_random_vs_warshall(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 13))
    m = int(rng.integers(1, n * n))
    edges = sorted({(int(rng.integers(n)), int(rng.integers(n))) for _ in range(m)})
    res = evaluate(TC, _edges(*zip(*edges)), {"path": I2})
    assert _rows(res, "path") == _warshall(n, edges)


def _walk_distance(n, src, dst):
    """Length of the shortest walk of >= 1 edge between every pair (inf if none)."""
    g = sp.csr_matrix((np.ones(len(src)), (src, dst)), shape=(n, n))
    d = csgraph.shortest_path(g, unweighted=True)            # 0 on the diagonal
    walk = np.full((n, n), np.inf)
    for u, v in zip(src, dst):                                # first edge u->v, then v ~> y
        walk[u] = np.minimum(walk[u], 1 + d[v])
    return walk


def test_tc_uniform_small_vs_bfs_levels():
    wl = W.small_workloads()["tc_uniform"]()
    src, dst = wl.edb["edge"][1]
    n = wl.params["n_nodes"]
    res = evaluate(wl.rules, wl.edb, wl.idb)
    walk = _walk_distance(n, src, dst)
    expect = sorted((int(i), int(j)) for i, j in zip(*np.nonzero(np.isfinite(walk))))
    assert _rows(res, "path") == expect
    # naive iterate k holds exactly the pairs joined by a walk of at most k edges
    sizes = res.sizes["path"]
    for k, size in enumerate(sizes, start=1):
        assert size == int((walk <= k).sum())
    assert sizes[-1] == sizes[-2] and len(sizes) == int(walk[np.isfinite(walk)].max()) + 1


def test_reach_count_equals_closure_row_sums():
    wl = W.tc_rmat(scale=8, n_edges=1500, seed=21)
    src, dst = wl.edb["edge"][1]
    res = evaluate(wl.rules, wl.edb, wl.idb)
    walk = _walk_distance(1 << 8, src, dst)
    rows = np.isfinite(walk).sum(axis=1)
    expect = sorted((int(x), int(c)) for x, c in enumerate(rows) if c > 0)
    assert _rows(res, "reach_count") == expect
    assert res.iterations[("reach_count",)] == 2


def test_iteration_cap_raises():
    src = np.arange(6)
    with pytest.raises(ConvergenceFailure):
        evaluate(TC, _edges(src, src + 1), {"path": I2}, max_iterations=3)
    evaluate(TC, _edges(src, src + 1), {"path": I2}, max_iterations=7)


# ---------------------------------------------------------------- shortest paths (min)
SS = {"dist": ("i32", "i32", "f32")}


def _weighted(src, dst, w, sources):
    return {"edge": (("i32", "i32", "f32"), [np.asarray(src, np.int32), np.asarray(dst, np.int32),
                                             np.asarray(w, np.float32)]),
            "source": (("i32",), [np.asarray(sources, np.int32)])}


def test_min_chain_integer_weights():
    n = 40
    w = np.arange(1, n, dtype=np.float32)
    res = evaluate(W.SSSP_RULES, _weighted(np.arange(n - 1), np.arange(1, n), w, [0, 10]), SS)
    _, (s, y, d) = res.relations["dist"]
    for si, yi, di in zip(s, y, d):
        assert yi >= si
        assert di == np.float32(w[si:yi].sum())     # prefix sums, exact in f32


def test_min_diamond_takes_shorter_branch():
    res = evaluate(W.SSSP_RULES, _weighted([0, 0, 1, 2], [1, 2, 3, 3], [1, 5, 1, 1], [0]), SS)
    got = sorted(zip(*[c.tolist() for c in res.relations["dist"][1]]))
    assert got == [(0, 0, 0.0), (0, 1, 1.0), (0, 2, 5.0), (0, 3, 2.0)]


@pytest.mark.parametrize("seed", range(6))
def test_min_vs_floyd_warshall_integer_weights(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(3, 15))
    pairs = sorted({(int(rng.integers(n)), int(rng.integers(n))) for _ in range(3 * n)})
    pairs = [(u, v) for u, v in pairs if u != v]
    src, dst = map(np.asarray, zip(*pairs))
    w = rng.integers(1, 10, len(pairs)).astype(np.float32)
    sources = sorted(set(int(x) for x in rng.integers(0, n, 3)))
    res = evaluate(W.SSSP_RULES, _weighted(src, dst, w, sources), SS)
    g = sp.csr_matrix((w.astype(np.float64), (src, dst)), shape=(n, n))
    fw = csgraph.floyd_warshall(g)
    expect = sorted((s, y, float(fw[s, y])) for s in sources for y in range(n)
                    if np.isfinite(fw[s, y]))
    got = sorted((s, y, float(d)) for s, y, d in zip(*[c.tolist() for c in res.relations["dist"][1]]))
    assert got == expect


def _dijkstra_f32(n, src, dst, w, s):
    """Textbook Dijkstra whose relaxation is one binary32 addition."""
    adj = [[] for _ in range(n)]
    for u, v, x in zip(src.tolist(), dst.tolist(), w):
        adj[u].append((v, x))
    dist = {s: np.float32(0.0)}
    heap = [(0.0, s)]
    done = set()
    while heap:
        d, u = heapq.heappop(heap)
        if u in done:
            continue
        done.add(u)
        for v, x in adj[u]:
            nd = dist[u] + x                      # np.float32 + np.float32
            if v not in dist or nd < dist[v]:
                dist[v] = nd
                heapq.heappush(heap, (float(nd), v))
    return dist


def test_min_sssp_small_bit_exact_vs_f32_dijkstra():
    wl = W.small_workloads()["sssp"]()
    src, dst, w = wl.edb["edge"][1]
    res = evaluate(wl.rules, wl.edb, wl.idb)
    s_col, y_col, d_col = res.relations["dist"][1]
    n = wl.params["n_nodes"]
    for s in wl.edb["source"][1][0].tolist():
        ref = _dijkstra_f32(n, src, dst, w, s)
        sel = s_col == s
        got = dict(zip(y_col[sel].tolist(), d_col[sel]))
        assert set(got) == set(ref)
        for y, d in ref.items():
            assert got[y].view(np.int32) == np.float32(d).view(np.int32), (s, y)
    # the f64 textbook answer agrees within the hop-scaled rounding bound
    g = sp.csr_matrix((w.astype(np.float64), (src, dst)), shape=(n, n))
    sources = wl.edb["source"][1][0]
    d64 = csgraph.dijkstra(g, indices=sources)
    ref64 = d64[np.searchsorted(sources, s_col), y_col]
    assert np.all(np.abs(d_col - ref64) <= 64 * 2.0 ** -24 * ref64 + 1e-30)


# ---------------------------------------------------------------- logsumexp
LS = {"score": ("i32", "i32", "f32")}


def _paths_lse(n, src, dst, w, s):
    """log of the sum over all paths of >= 1 edge from s of exp(total weight), by enumeration."""
    adj = [[] for _ in range(n)]
    for u, v, x in zip(src, dst, w):
        adj[u].append((v, float(x)))
    acc = {}

    def walk(u, total):
        for v, x in adj[u]:
            acc.setdefault(v, []).append(total + x)
            walk(v, total + x)

    walk(s, 0.0)
    return {v: math.log(sum(math.exp(t) for t in ts)) for v, ts in acc.items()}


@pytest.mark.parametrize("seed", range(5))
def test_lse_small_dag_vs_path_enumeration(seed):
    wl = W.layered_dag(n_layers=5, width=4, out_degree=2, n_sources=2, seed=200 + seed)
    src, dst, w = [c.tolist() for c in wl.edb["edge"][1]]
    res = evaluate(wl.rules, wl.edb, wl.idb)
    s_col, y_col, p_col = [c.tolist() for c in res.relations["score"][1]]
    for s in wl.edb["source"][1][0].tolist():
        ref = _paths_lse(5 * 4, src, dst, w, s)
        got = {y: p for ss, y, p in zip(s_col, y_col, p_col) if ss == s}
        assert set(got) == set(ref)
        for y, p in ref.items():
            assert abs(got[y] - p) <= 1e-5 * max(1.0, abs(p))


@pytest.mark.parametrize("K,L,w", [(3, 5, -0.5), (4, 4, 0.25), (1, 7, -1.0)])
def test_lse_complete_layered_closed_form(K, L, w):
    src, dst = [], []
    for layer in range(L - 1):
        for a in range(K):
            for b in range(K):
                src.append(layer * K + a)
                dst.append((layer + 1) * K + b)
    inputs = _weighted(src, dst, np.full(len(src), w, np.float32), [0])
    res = evaluate(W.LSE_RULES, inputs, LS)
    for s, y, p in zip(*[c.tolist() for c in res.relations["score"][1]]):
        layer = y // K
        expect = (layer - 1) * math.log(K) + layer * w
        assert abs(p - expect) <= 1e-5 * max(1.0, abs(expect)), (y, p, expect)


def test_lse_single_path_is_weight_sum():
    w = np.array([-0.1, -2.5, -0.75, -0.3], np.float32)
    res = evaluate(W.LSE_RULES, _weighted([0, 1, 2, 3], [1, 2, 3, 4], w, [0]), LS)
    got = [p for _, _, p in zip(*[c.tolist() for c in res.relations["score"][1]])]
    assert np.allclose(got, np.cumsum(w.astype(np.float64)), rtol=0, atol=1e-6)


def test_lse_layered_forward_pass_small_workload():
    """Layer-by-layer forward pass in probability space (a textbook routine)."""
    wl = W.small_workloads()["lse_dag"]()
    L, K = wl.params["n_layers"], wl.params["width"]
    src, dst, w = wl.edb["edge"][1]
    res = evaluate(wl.rules, wl.edb, wl.idb)
    s_col, y_col, p_col = res.relations["score"][1]
    A = sp.csr_matrix((np.exp(w.astype(np.float64)), (src, dst)), shape=(L * K, L * K))
    for s in wl.edb["source"][1][0][:6].tolist():
        mass = np.zeros(L * K)
        mass[s] = 1.0
        total = np.zeros(L * K)
        for _ in range(L - 1):
            mass = A.T @ mass
            total += mass
        sel = s_col == s
        ref = np.log(total[y_col[sel]])
        assert np.count_nonzero(total) == sel.sum()
        assert np.all(np.abs(p_col[sel] - ref) <= 1e-5 * np.maximum(1.0, np.abs(ref)))


# ---------------------------------------------------------------- same generation
def test_sg_closed_form_small_forest():
    wl = W.small_workloads()["same_generation"]()
    depth, root = wl.params["depth"], wl.params["root"]
    res = evaluate(wl.rules, wl.edb, wl.idb)
    got = _rows(res, "sg")
    # nodes that have a parent (roots never appear in sg: both rules need parent(X,_))
    has_parent = np.zeros(len(depth), bool)
    has_parent[wl.edb["parent"][1][0]] = True
    groups = {}
    for v in np.flatnonzero(has_parent):
        groups.setdefault((int(root[v]), int(depth[v])), []).append(int(v))
    expect = sorted((x, y) for g in groups.values() for x in g for y in g if x != y)
    assert got == expect
    assert len(got) == sum(len(g) * (len(g) - 1) for g in groups.values())


# ---------------------------------------------------------------- stratified negation
NEG_LISTING = """
degree(X, count(Y)) :- edge(X, Y).
violation(X) :- edge(X, _), not degree(X, _).
sink(Y) :- edge(_, Y), not degree(Y, _).
"""


def test_listing_negation_constraint_and_sinks():
    res = evaluate(NEG_LISTING, _edges([1, 1, 1, 2], [2, 3, 4, 3]),
                   {"degree": I2, "violation": ("i32",), "sink": ("i32",)})
    assert _rows(res, "violation") == []
    assert _rows(res, "sink") == _golden("listing_negation_degree.txt")
    assert _rows(res, "degree") == _golden("listing_agg_degree.txt")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_negation_set_difference_brute_force(seed):
    """oneway = E minus the reversed E, and a constant in the negated literal,
    against Python set algebra over the edge tuples."""
    rng = np.random.default_rng(seed)
    n, m = 12, 40
    src, dst = rng.integers(0, n, m), rng.integers(0, n, m)
    rules = """
    oneway(X, Y) :- edge(X, Y), not edge(Y, X).
    notfrom0(X, Y) :- edge(X, Y), not edge(0, Y).
    noloop(X) :- edge(X, _), not edge(X, X).
    """
    res = evaluate(rules, _edges(src, dst), {"oneway": I2, "notfrom0": I2, "noloop": ("i32",)})
    E = set(zip(src.tolist(), dst.tolist()))
    assert _rows(res, "oneway") == sorted((x, y) for x, y in E if (y, x) not in E)
    assert _rows(res, "notfrom0") == sorted((x, y) for x, y in E if (0, y) not in E)
    assert _rows(res, "noloop") == sorted({(x,) for x, _ in E if (x, x) not in E})


@pytest.mark.parametrize("seed", [3, 4])
def test_negation_of_a_recursive_relation_vs_bfs(seed):
    """Pairs (listed as an input relation) that the closure does not contain,
    against breadth-first search from every node."""
    rng = np.random.default_rng(seed)
    n, m = 15, 22
    src, dst = rng.integers(0, n, m), rng.integers(0, n, m)
    px, py = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    edb = _edges(src, dst)
    edb["pair"] = (I2, [px.ravel().astype(np.int32), py.ravel().astype(np.int32)])
    rules = TC + "unreached(X, Y) :- pair(X, Y), not path(X, Y).\n"
    res = evaluate(rules, edb, {"path": I2, "unreached": I2})
    adj = {u: set() for u in range(n)}
    for u, v in zip(src.tolist(), dst.tolist()):
        adj[u].add(v)
    expect = []
    for x in range(n):
        seen, todo = set(), list(adj[x])
        while todo:
            v = todo.pop()
            if v not in seen:
                seen.add(v)
                todo.extend(adj[v])
        expect += [(x, y) for y in range(n) if y not in seen]
    assert _rows(res, "unreached") == sorted(expect)
    assert len(_rows(res, "unreached")) + len(_rows(res, "path")) == n * n


def test_negation_repeated_variable_and_unbound_rejection():
    res = evaluate("nosym(X) :- node(X), not edge(X, X).",
                   {**_edges([1, 2, 3], [1, 3, 3]), "node": (("i32",), [np.array([1, 2, 3, 4], np.int32)])},
                   {"nosym": ("i32",)})
    assert _rows(res, "nosym") == [(2,), (4,)]
    with pytest.raises(ValueError):   # Z occurs only under 'not'
        evaluate("bad(X) :- edge(X, _), not edge(X, Z).", _edges([1], [2]), {"bad": ("i32",)})


def test_negation_inside_recursion_is_rejected():
    with pytest.raises(ValueError):
        evaluate("p(X) :- edge(X, _), not q(X).\nq(X) :- edge(_, X), not p(X).",
                 _edges([1, 2], [2, 3]), {"p": ("i32",), "q": ("i32",)})
    with pytest.raises(ValueError):
        evaluate("p(X) :- edge(X, _), not p(X).", _edges([1], [2]), {"p": ("i32",)})


# ---------------------------------------------------------------- triangle join
TRI3 = ("i32", "i32", "i32")


def _tri_edb(r, s, t):
    def rel(p):
        p = np.asarray(p, np.int64).reshape(-1, 2)
        return (I2, [p[:, 0].astype(np.int32), p[:, 1].astype(np.int32)])
    return {"r": rel(r), "s": rel(s), "t": rel(t)}


@pytest.mark.parametrize("a,b,c", [(1, 1, 1), (2, 3, 4), (5, 1, 7), (6, 6, 6)])
def test_triangle_complete_tripartite_closed_form(a, b, c):
    """r = A x B, s = B x C, t = A x C with disjoint value ranges: every
    (x, y, z) in A x B x C is a triangle, a*b*c of them."""
    A, B, C = range(0, a), range(100, 100 + b), range(200, 200 + c)
    res = evaluate(W.TRIANGLE_RULES, _tri_edb([(x, y) for x in A for y in B], [(y, z) for y in B for z in C],
                                              [(x, z) for x in A for z in C]), {"tri": TRI3})
    assert _rows(res, "tri") == [(x, y, z) for x in A for y in B for z in C]


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_triangle_brute_force(seed):
    rng = np.random.default_rng(seed)
    r, s_, t = (rng.integers(0, 7, (25, 2)) for _ in range(3))
    res = evaluate(W.TRIANGLE_RULES, _tri_edb(r, s_, t), {"tri": TRI3})
    R, S, T = (set(map(tuple, m.tolist())) for m in (r, s_, t))
    expect = sorted({(x, y, z) for (x, y) in R for (y2, z) in S if y2 == y for (x2, z2) in T
                     if x2 == x and z2 == z})
    assert _rows(res, "tri") == expect
    assert len(expect) > 0


def test_triangle_small_workload_vs_set_intersection():
    """Per r row (x, y): the z values in s[y] intersected with t[x]."""
    wl = W.triangle(rows=4096, core=40, hubs=4, seed=16)
    res = evaluate(wl.rules, wl.edb, wl.idb)
    (r0, r1), (s0, s1), (t0, t1) = [wl.edb[k][1] for k in "rst"]
    S, T = {}, {}
    for y, z in zip(s0.tolist(), s1.tolist()):
        S.setdefault(y, set()).add(z)
    for x, z in zip(t0.tolist(), t1.tolist()):
        T.setdefault(x, set()).add(z)
    expect = sorted((x, y, z) for x, y in zip(r0.tolist(), r1.tolist())
                    for z in S.get(y, set()) & T.get(x, set()))
    assert _rows(res, "tri") == expect
    assert len(expect) == 64057


# ---------------------------------------------------------------- restriction helper
def test_restriction_matches_full_rows():
    wl = W.small_workloads()["tc_uniform"]()
    full = evaluate(wl.rules, wl.edb, wl.idb).relations["path"][1]
    pick = np.array([3, 17, 99], np.int32)
    part = evaluate(wl.rules, wl.edb, wl.idb, restrict={"path": (0, pick)}).relations["path"][1]
    sel = np.isin(full[0], pick)
    assert np.array_equal(part[0], full[0][sel]) and np.array_equal(part[1], full[1][sel])


# ---------------------------------------------------------------- planted mistakes
def test_planted_mistakes_are_caught(monkeypatch):
    """Plausible bugs in the oracle's arithmetic make a pin fail."""
    import oracle.datalog as D

    real_fold = D._fold

    def wrong_sign_lse(op, keys, vals, ty):
        if op == "logsumexp":   # drops the max shift's add-back
            k, out = real_fold(op, keys, vals, ty)
            m = real_fold("max", keys, vals, ty)[1]
            return k, (out - m).astype(np.float32)
        return real_fold(op, keys, vals, ty)

    monkeypatch.setattr(D, "_fold", wrong_sign_lse)
    with pytest.raises(AssertionError):
        test_lse_complete_layered_closed_form(3, 5, -0.5)
    monkeypatch.setattr(D, "_fold", real_fold)

    def max_for_min(op, keys, vals, ty):
        return real_fold("max" if op == "min" else op, keys, vals, ty)

    monkeypatch.setattr(D, "_fold", max_for_min)
    with pytest.raises(AssertionError):
        test_min_diamond_takes_shorter_branch()
    monkeypatch.setattr(D, "_fold", real_fold)

    real_body = D._eval_body

    def transposed_edges(rule, rels, var_types):   # join edge on its target column
        rels = dict(rels)
        if "edge" in rels:
            t, c = rels["edge"]
            rels["edge"] = (t, [c[1], c[0]] + list(c[2:]))
        return real_body(rule, rels, var_types)

    monkeypatch.setattr(D, "_eval_body", transposed_edges)
    with pytest.raises(AssertionError):
        test_tc_chain_closed_form(5)
    monkeypatch.setattr(D, "_eval_body", real_body)

    real_neg = D._negated_match

    def negation_ignores_second_column(pred, terms, rels, binding, var_types, n):
        terms = [t if j == 0 else ("anon",) for j, t in enumerate(terms)]
        return real_neg(pred, terms, rels, binding, var_types, n)

    monkeypatch.setattr(D, "_negated_match", negation_ignores_second_column)
    with pytest.raises(AssertionError):
        test_negation_set_difference_brute_force(0)
    monkeypatch.setattr(D, "_negated_match", real_neg)

    def transposed_t(rule, rels, var_types):   # joins t on its columns swapped
        rels = dict(rels)
        if "t" in rels:
            ty, c = rels["t"]
            rels["t"] = (ty, [c[1], c[0]])
        return real_body(rule, rels, var_types)

    monkeypatch.setattr(D, "_eval_body", transposed_t)
    with pytest.raises(AssertionError):
        test_triangle_brute_force(0)
    monkeypatch.setattr(D, "_eval_body", real_body)
