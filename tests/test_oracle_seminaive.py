"""The oracle's semi-naive mode (Algorithm 1, Sec. 4.1) against the naive
definition: the least fixpoint is the same relation, so sets and min/max
values agree bit for bit, integer path sums exactly, and logsumexp within
float rounding (its folds run in a different order).  The pass counts are
the engine's (seed = iteration 0, the final empty pass counts), pinned by
breadth-first levels on chains.  Where the naive fixpoint is not a semiring
path sum -- a constant added to a recursive sum's value -- the two differ on a
DAG whose paths to a node have different lengths, which is why the engine
refuses such rules."""
import numpy as np
import pytest

from oracle import evaluate
from oracle.seminaive import evaluate_semi_naive
from paper_2609_27203_amd import workloads as W


def _agree(wl_rules, edb, idb, lse_tol=1e-6):
    a = evaluate(wl_rules, edb, idb)
    b = evaluate_semi_naive(wl_rules, edb, idb)
    for rel, types in idb.items():
        ca, cb = a.relations[rel][1], b.relations[rel][1]
        assert len(ca[0]) == len(cb[0]), (rel, len(ca[0]), len(cb[0]))
        lse = f"{rel}(" in wl_rules and "logsumexp(" in wl_rules
        for t, x, y in zip(types, ca, cb):
            if t == "f32" and lse:
                err = np.abs(x.astype(np.float64) - y.astype(np.float64))
                assert np.all(err <= lse_tol * np.maximum(1.0, np.abs(x.astype(np.float64)))), rel
            elif t == "f32":
                assert np.array_equal(x.view(np.int32), y.view(np.int32)), rel
            else:
                assert np.array_equal(x, y), rel
    return a, b


@pytest.mark.parametrize("name", ["tc_uniform", "sssp", "lse_dag", "same_generation", "tc_rmat_count", "triangle"])
def test_small_workloads_agree_with_naive(name):
    wl = W.small_workloads()[name]()
    _agree(wl.rules, wl.edb, wl.idb)


def _random_dag(n, m, seed):
    rng = np.random.default_rng(seed)
    u = rng.integers(0, n, 4 * m)
    v = rng.integers(0, n, 4 * m)
    keep = u < v  # edges go from lower to higher ids: acyclic, paths of mixed lengths
    pairs = np.unique(np.stack([u[keep], v[keep]], 1), axis=0)[:m]
    w = (rng.random(len(pairs)) * -2.0 - 0.1).astype(np.float32)
    return pairs[:, 0].astype(np.int32), pairs[:, 1].astype(np.int32), w


@pytest.mark.parametrize("seed", range(4))
def test_random_graphs_agree_with_naive(seed):
    src, dst, w = _random_dag(40, 120, seed)
    rng = np.random.default_rng(100 + seed)
    # closure over a graph with cycles (back edges added)
    back = rng.integers(0, len(src), 10)
    cs, cd = np.concatenate([src, dst[back]]), np.concatenate([dst, src[back]])
    _agree(W.TC_RULES, {"edge": (("i32", "i32"), [cs, cd])}, {"path": ("i32", "i32")})
    # non-linear closure (two recursive atoms: two delta variants)
    _agree("path(X,Y) :- edge(X,Y).\npath(X,Y) :- path(X,Z), path(Z,Y).\n",
           {"edge": (("i32", "i32"), [cs, cd])}, {"path": ("i32", "i32")})
    sources = (("i32",), [np.array([0, 1, 2], np.int32)])
    wedge = (("i32", "i32", "f32"), [src, dst, w])
    _agree(W.SSSP_RULES, {"source": sources, "edge": (("i32", "i32", "f32"), [cs, cd, np.abs(
        np.concatenate([w, w[back]])) + np.float32(1.0)])}, {"dist": ("i32", "i32", "f32")})
    _agree(W.LSE_RULES, {"source": sources, "edge": wedge}, {"score": ("i32", "i32", "f32")})
    # path counts: a recursive sum that carries the recursive value unchanged
    _agree("""
npaths(S,Y,sum(C)) :- source(S), C is 1, edge(S,Y,_).
npaths(S,Y,sum(C)) :- npaths(S,Z,C1), edge(Z,Y,_), C is C1.
""", {"source": sources, "edge": wedge}, {"npaths": ("i32", "i32", "i32")})
    # mutual recursion (two heads in one stratum) and a later negated stratum
    _agree("""
odd(X,Y) :- edge(X,Y).
even(X,Y) :- odd(X,Z), edge(Z,Y).
odd(X,Y) :- even(X,Z), edge(Z,Y).
only_odd(X,Y) :- odd(X,Y), not even(X,Y).
""", {"edge": (("i32", "i32"), [cs, cd])},
           {"odd": ("i32", "i32"), "even": ("i32", "i32"), "only_odd": ("i32", "i32")})


def test_pass_counts_are_breadth_first_levels():
    """A chain of n nodes: n - 1 passes (the last one empty), and the
    closure grows by one level per pass."""
    n = 12
    src = np.arange(n - 1, dtype=np.int32)
    r = evaluate_semi_naive(W.TC_RULES, {"edge": (("i32", "i32"), [src, src + 1])}, {"path": ("i32", "i32")})
    assert r.iterations[("path",)] == n - 1
    total = np.cumsum(np.arange(n - 1, 0, -1))
    assert r.sizes["path"] == list(total) + [total[-1]]


def test_affine_recursive_sum_is_not_a_path_sum():
    """sum over C is C1 - K: on a DAG where a node is reached by paths of
    different lengths, the naive fixpoint adds each edge's K once, while
    passes add it once per pass in which the source's value changes.  On
    a layered DAG (every path to a node has the same length) the two agree."""
    rules = """
ws(S,Y,sum(C)) :- source(S), edge(S,Y,K), C is 0 - K.
ws(S,Y,sum(C)) :- ws(S,Z,C1), edge(Z,Y,K), C is C1 - K.
"""
    idb = {"ws": ("i32", "i32", "i32")}
    src = (("i32",), [np.array([0], np.int32)])
    # 0 -> 1 -> 2 and 0 -> 2: node 2 is reached in pass 0 and pass 1
    e = (("i32", "i32", "i32"), [np.array([0, 1, 0, 2], np.int32), np.array([1, 2, 2, 3], np.int32),
                                 np.array([1, 1, 1, 5], np.int32)])
    a = evaluate(rules, {"source": src, "edge": e}, idb).relations["ws"][1]
    b = evaluate_semi_naive(rules, {"source": src, "edge": e}, idb).relations["ws"][1]
    assert not np.array_equal(a[2], b[2])
    # naive: ws(1) = -1, ws(2) = (ws(1) - 1) + (0 - 1) = -3, ws(3) = ws(2) - 5 = -8
    assert a[2].tolist() == [-1, -3, -8]
    # layered (0 -> {1, 2} -> 3): every path to a node has one length
    e2 = (("i32", "i32", "i32"), [np.array([0, 0, 1, 2], np.int32), np.array([1, 2, 3, 3], np.int32),
                                  np.array([1, 2, 3, 4], np.int32)])
    _agree(rules, {"source": src, "edge": e2}, idb)
