"""Pins for the oracle's sum fold and its ``is`` arithmetic (subtraction
included), each against something other than the oracle itself.

* sum (paper Sec. 3 "Aggregations and constraints": sum is a head aggregate
  folded over a group's derivations): the number of paths from a source,
  which the path-counting program computes, has closed forms on a complete
  layered DAG (K^(L-1) at layer L) and on a grid (a binomial coefficient),
  and is counted by explicit path enumeration on small random DAGs; a
  weighted sum over derivations is checked against a one-pass dynamic
  program over the DAG in topological order with exact Python integers.
* ``is`` (paper Sec. 3 "Expressions, arithmetic, and user-defined
  functions"; Sec. 3.2: arithmetic keeps scalar types): a min over
  ``D is D1 - W`` on a chain gives negated prefix sums, on a random DAG the
  negated longest path (topological dynamic program); a max over
  ``D is D1 - W`` gives the negated shortest path (Dijkstra); hand-computed
  values for mixed signs, constants and one binary32 rounding per operation.
* Planted mistakes (a constant sum, a sum over distinct values, a sum that
  drops a derivation, '-' read as '+', f32 arithmetic rounded once at the
  end) must each make one of these pins fail.
"""
import heapq
import math

import numpy as np
import pytest

from oracle import evaluate

I2 = ("i32", "i32")
I3 = ("i32", "i32", "i32")

NPATHS = """
np(S,Y,sum(C)) :- source(S), edge(S,Y), C is 1.
np(S,Y,sum(C)) :- np(S,Z,C1), edge(Z,Y), C is C1.
"""

WSUM = """
ws(S,Y,sum(C)) :- source(S), edge(S,Y,W), C is W.
ws(S,Y,sum(C)) :- ws(S,Z,C1), edge(Z,Y,W), C is C1 {op} W.
"""

LOW = """
low(S,S,min(D)) :- source(S), D is 0.
low(S,Y,min(D)) :- low(S,Z,D1), edge(Z,Y,W), D is D1 - W.
"""

HIGH = """
high(S,S,max(D)) :- source(S), D is 0.
high(S,Y,max(D)) :- high(S,Z,D1), edge(Z,Y,W), D is D1 - W.
"""


def _rel(*cols, types=None):
    cols = [np.asarray(c) for c in cols]
    types = types or tuple("i32" for _ in cols)
    return (tuple(types), [np.asarray(c, np.float32 if t == "f32" else np.int32) for c, t in zip(cols, types)])


def _rows(res, name):
    _, cols = res.relations[name]
    return {tuple(r[:-1]): r[-1] for r in zip(*[c.tolist() for c in cols])}


def _random_dag(seed, n=14, p=0.3, wmax=9):
    """Edges u -> v with u < v (so ascending ids are a topological order)."""
    rng = np.random.default_rng(seed)
    src, dst = [], []
    for u in range(n):
        for v in range(u + 1, n):
            if rng.random() < p:
                src.append(u)
                dst.append(v)
    w = rng.integers(1, wmax + 1, len(src))
    return np.array(src), np.array(dst), w


# ---------------------------------------------------------------- sum: path counts
@pytest.mark.parametrize("K,L", [(3, 6), (2, 9), (5, 3), (1, 8)])
def test_sum_counts_paths_complete_layered_dag(K, L):
    """Layers 0..L-1 of K nodes, every node linked to every node of the next
    layer; a source in layer 0 reaches a node of layer l >= 1 by K^(l-1) paths."""
    src, dst = [], []
    for layer in range(L - 1):
        for a in range(K):
            for b in range(K):
                src.append(layer * K + a)
                dst.append((layer + 1) * K + b)
    res = evaluate(NPATHS, {"edge": _rel(src, dst), "source": _rel([0])}, {"np": I3})
    got = _rows(res, "np")
    assert len(got) == (L - 1) * K
    for (s, y), c in got.items():
        assert c == K ** (y // K - 1), (y, c)


@pytest.mark.parametrize("R,C", [(6, 6), (4, 9), (1, 5)])
def test_sum_counts_lattice_paths_binomial(R, C):
    """Grid (i, j) -> (i + 1, j), (i, j + 1): C(i + j, i) monotone paths from the corner."""
    node = lambda i, j: i * C + j  # noqa: E731
    src, dst = [], []
    for i in range(R):
        for j in range(C):
            if i + 1 < R:
                src.append(node(i, j))
                dst.append(node(i + 1, j))
            if j + 1 < C:
                src.append(node(i, j))
                dst.append(node(i, j + 1))
    res = evaluate(NPATHS, {"edge": _rel(src, dst), "source": _rel([0])}, {"np": I3})
    got = _rows(res, "np")
    expect = {(0, node(i, j)): math.comb(i + j, i) for i in range(R) for j in range(C) if i + j > 0}
    assert got == expect


def _count_paths(src, dst, s):
    """Paths of >= 1 edge from s to every node, by explicit enumeration."""
    adj = {}
    for u, v in zip(src.tolist(), dst.tolist()):
        adj.setdefault(u, []).append(v)
    count = {}

    def walk(u):
        for v in adj.get(u, []):
            count[v] = count.get(v, 0) + 1
            walk(v)

    walk(s)
    return count


@pytest.mark.parametrize("seed", range(6))
def test_sum_counts_paths_random_dag_enumeration(seed):
    src, dst, _ = _random_dag(seed)
    sources = [0, 1, 3]
    res = evaluate(NPATHS, {"edge": _rel(src, dst), "source": _rel(sources)}, {"np": I3})
    got = _rows(res, "np")
    expect = {(s, y): c for s in sources for y, c in _count_paths(src, dst, s).items()}
    assert got == expect
    assert max(expect.values()) > 2   # several paths meet somewhere


def _dag_fixpoint(src, dst, w, s, combine, fold):
    """One pass in topological (ascending id) order of the value equation a
    carried-value rule states on a DAG: a node's value is the fold of one
    contribution per derivation -- w(s, y) for a first edge out of s, and
    combine(value(z), w(z, y)) for every edge z -> y with z already valued."""
    val = {}
    n = int(max(src.max(), dst.max())) + 1
    base = {}
    for u, v, x in zip(src.tolist(), dst.tolist(), w.tolist()):
        if u == s:
            base.setdefault(v, []).append(x)
    into = {}
    for u, v, x in zip(src.tolist(), dst.tolist(), w.tolist()):
        into.setdefault(v, []).append((u, x))
    for y in range(n):
        parts = list(base.get(y, [])) + [combine(val[z], x) for z, x in into.get(y, []) if z in val]
        if parts:
            val[y] = fold(parts)
    return val


@pytest.mark.parametrize("op", ["+", "-"])
@pytest.mark.parametrize("seed", range(4))
def test_weighted_sum_over_derivations_vs_topological_pass(seed, op):
    src, dst, w = _random_dag(10 + seed, n=12)
    sources = [0, 2]
    edb = {"edge": _rel(src, dst, w), "source": _rel(sources)}
    res = evaluate(WSUM.format(op=op), edb, {"ws": I3})
    comb = (lambda a, b: a + b) if op == "+" else (lambda a, b: a - b)
    expect = {}
    for s in sources:
        for y, v in _dag_fixpoint(src, dst, w, s, comb, sum).items():
            expect[(s, y)] = v
    assert _rows(res, "ws") == expect


def test_weighted_sum_f32_integer_weights_vs_topological_pass():
    """The same with f32 weights: small integers, so every sum is exact."""
    src, dst, w = _random_dag(21, n=11, wmax=5)
    edb = {"edge": _rel(src, dst, w, types=("i32", "i32", "f32")), "source": _rel([0, 1])}
    res = evaluate(WSUM.format(op="-"), edb, {"ws": ("i32", "i32", "f32")})
    expect = {}
    for s in (0, 1):
        for y, v in _dag_fixpoint(src, dst, w, s, lambda a, b: a - b, sum).items():
            expect[(s, y)] = float(v)
    assert _rows(res, "ws") == expect


# ---------------------------------------------------------------- subtraction in 'is'
def test_subtraction_chain_gives_negated_prefix_sums():
    n = 30
    w = np.arange(1, n) * 3 % 11 + 1
    edb = {"edge": _rel(np.arange(n - 1), np.arange(1, n), w), "source": _rel([0, 7])}
    got = _rows(evaluate(LOW, edb, {"low": I3}), "low")
    expect = {(s, y): -int(w[s:y].sum()) for s in (0, 7) for y in range(s, n)}
    assert got == expect


def _longest(src, dst, w, s):
    """Longest path weight from s (0 for s itself) by a topological dynamic program."""
    best = {s: 0}
    for u, v, x in sorted(zip(src.tolist(), dst.tolist(), w.tolist())):
        if u in best:
            best[v] = max(best.get(v, -math.inf), best[u] + x)
    return best


def _shortest(src, dst, w, s):
    adj = {}
    for u, v, x in zip(src.tolist(), dst.tolist(), w.tolist()):
        adj.setdefault(u, []).append((v, x))
    dist, heap = {s: 0}, [(0, s)]
    while heap:
        d, u = heapq.heappop(heap)
        if d > dist[u]:
            continue
        for v, x in adj.get(u, []):
            if d + x < dist.get(v, math.inf):
                dist[v] = d + x
                heapq.heappush(heap, (d + x, v))
    return dist


@pytest.mark.parametrize("seed", range(5))
def test_subtraction_min_is_negated_longest_path(seed):
    src, dst, w = _random_dag(30 + seed)
    edb = {"edge": _rel(src, dst, w), "source": _rel([0, 1])}
    got = _rows(evaluate(LOW, edb, {"low": I3}), "low")
    expect = {(s, y): -d for s in (0, 1) for y, d in _longest(src, dst, w, s).items()}
    assert got == expect


@pytest.mark.parametrize("seed", range(3))
def test_subtraction_max_is_negated_shortest_path(seed):
    src, dst, w = _random_dag(40 + seed)
    edb = {"edge": _rel(src, dst, w), "source": _rel([0, 2])}
    got = _rows(evaluate(HIGH, edb, {"high": I3}), "high")
    expect = {(s, y): -d for s in (0, 2) for y, d in _shortest(src, dst, w, s).items()}
    assert got == expect


def test_mixed_signs_and_constants_hand_values():
    rows = [(10, 3, 1), (0, 5, 7), (-4, -4, 2), (100, 250, -50)]
    rules = "v(A,B,C,V) :- t(A,B,C), V is A - B + C - 2.\nw(A,V) :- t(A,_,_), V is 0 - A - 1."
    res = evaluate(rules, {"t": _rel(*zip(*rows))}, {"v": ("i32",) * 4, "w": I2})
    v = sorted(zip(*[c.tolist() for c in res.relations["v"][1]]))
    assert v == sorted([(10, 3, 1, 6), (0, 5, 7, 0), (-4, -4, 2, 0), (100, 250, -50, -202)])
    w = sorted(zip(*[c.tolist() for c in res.relations["w"][1]]))
    assert w == [(-4, 3), (0, -1), (10, -11), (100, -101)]


def test_f32_subtraction_rounds_after_every_operation():
    """binary32 values: 1.5 - 0.25 = 1.25 exactly; 1 - 2^-30 rounds to 1
    (less than half of the 2^-24 spacing below 1); 2^24 - (-1) - (-1): the
    first subtraction gives 2^24 + 1, which is a tie between 2^24 and
    2^24 + 2 and rounds to the even 2^24, and so does the second, so the
    result is 2^24, where one rounding of the exact 2^24 + 2 would give
    2^24 + 2."""
    a = np.array([1.5, 1.0, 2.0 ** 24], np.float32)
    b = np.array([0.25, 2.0 ** -30, -1.0], np.float32)
    c = np.array([0.0, 0.0, -1.0], np.float32)
    ty = ("f32", "f32", "f32")
    res = evaluate("d(A,V) :- t(A,B,C), V is A - B - C.", {"t": _rel(a, b, c, types=ty)},
                   {"d": ("f32", "f32")})
    got = dict(zip(*[c.tolist() for c in res.relations["d"][1]]))
    assert got == {1.5: 1.25, 1.0: 1.0, 2.0 ** 24: 2.0 ** 24}


# ---------------------------------------------------------------- planted mistakes
def test_planted_sum_and_subtraction_mistakes_are_caught(monkeypatch):
    import oracle.datalog as D

    real_fold = D._fold

    def planted(kind):
        def fold(op, keys, vals, ty):
            if op != "sum":
                return real_fold(op, keys, vals, ty)
            gkeys, out = real_fold(op, keys, vals, ty)
            if kind == "constant":
                return gkeys, np.full_like(out, 7)
            # recompute per group: distinct values only, or all but the first derivation
            order = np.lexsort([D._order(k) for k in keys][::-1])
            ks = [k[order] for k in keys]
            vs = vals[order]
            start = np.ones(len(vs), bool)
            start[1:] = False
            for k in ks:
                start[1:] |= k[1:] != k[:-1]
            bounds = list(np.flatnonzero(start)) + [len(vs)]
            res = []
            for lo, hi in zip(bounds[:-1], bounds[1:]):
                seg = vs[lo:hi]
                res.append(np.unique(seg).sum() if kind == "distinct" else seg[1:].sum() if hi - lo > 1 else seg[0])
            return gkeys, np.asarray(res, out.dtype)
        return fold

    for kind in ("constant", "distinct", "drop_first"):
        monkeypatch.setattr(D, "_fold", planted(kind))
        failed = 0
        for case in (lambda: test_sum_counts_paths_complete_layered_dag(3, 6),
                     lambda: test_sum_counts_lattice_paths_binomial(6, 6),
                     lambda: test_sum_counts_paths_random_dag_enumeration(0)):
            try:
                case()
            except AssertionError:
                failed += 1
        assert failed >= 2, kind
        monkeypatch.setattr(D, "_fold", real_fold)

    real_parse = D.parse

    def minus_as_plus(text):
        rules = real_parse(text)
        for r in rules:
            r.assigns = [(v, [(1, t) for _, t in parts]) for v, parts in r.assigns]
        return rules

    monkeypatch.setattr(D, "parse", minus_as_plus)
    for case in (test_subtraction_chain_gives_negated_prefix_sums, test_mixed_signs_and_constants_hand_values,
                 lambda: test_subtraction_min_is_negated_longest_path(0),
                 lambda: test_weighted_sum_over_derivations_vs_topological_pass(0, "-")):
        with pytest.raises(AssertionError):
            case()
    monkeypatch.setattr(D, "parse", real_parse)

    # f32 arithmetic kept in f64 and rounded once at the end of the expression
    real_body = D._eval_body
    orig_f32 = np.float32

    def once(rule, rels, var_types):
        saved = list(rule.assigns)
        try:
            b, n = real_body(D.Rule(rule.head, rule.head_terms, rule.agg, rule.atoms, [], rule.filters, rule.negs),
                             rels, var_types)
            for var, parts in saved:
                acc = np.zeros(n, np.float64)
                for sign, t in parts:
                    x = b[t[1]] if t[0] == "var" else t[1]
                    acc = acc + sign * np.asarray(x, np.float64)
                b[var] = acc.astype(orig_f32)
                var_types[var] = "f32"
            return b, n
        finally:
            rule.assigns = saved

    monkeypatch.setattr(D, "_eval_body", once)
    with pytest.raises(AssertionError):
        test_f32_subtraction_rounds_after_every_operation()
    monkeypatch.setattr(D, "_eval_body", real_body)
