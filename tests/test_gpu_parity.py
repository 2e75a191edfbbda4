"""GPU parity: the HIP engine (through the C ABI) against the CPU oracle.

Sets and counts must match bit for bit; min within 1e-6 relative (the f32
fixpoint is expected to be bit-exact); logsumexp within 1e-5 * max(1, |ref|).
"""
import os

import numpy as np
import pytest

from helpers import LSE_TOL, assert_same_relation, engine_run, value_tolerance
from oracle import evaluate
from paper_2609_27203_amd import workloads as W

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _compare(wl, rels, ref, where=""):
    for name, types in wl.idb.items():
        assert_same_relation(name, types, rels[name], ref.relations[name][1], where,
                             tol=value_tolerance(wl.rules, name))


def _golden(name):
    rows = [tuple(int(x) for x in ln.split()) for ln in open(os.path.join(GOLDEN, name))
            if ln.strip() and not ln.startswith("#")]
    return [np.array(c, np.int32) for c in zip(*sorted(rows))]


def _edges(src, dst):
    return {"edge": (("i32", "i32"), [np.asarray(src, np.int32), np.asarray(dst, np.int32)])}


# ------------------------------------------------------------- worked examples
def test_listing_minimal_reach():
    wl = W.Workload("listing", "reach(X, Y) :- edge(X, Y).\nreach(X, Z) :- reach(X, Y), edge(Y, Z).",
                    _edges([1, 2, 3], [2, 3, 4]), {"reach": ("i32", "i32")})
    print("case: listing minimal reach", flush=True)
    rels, stats, _ = engine_run(wl, workspace_bytes=256 << 20)
    exp = _golden("listing_minimal_reach.txt")
    assert all(np.array_equal(a, b) for a, b in zip(rels["reach"], exp))
    assert stats["delta_rows"] == [3, 2, 1, 0] and stats["iterations"] == 3


def test_listing_agg_degree():
    wl = W.Workload("agg", "degree(X, count(Y)) :- edge(X, Y).", _edges([1, 1, 1, 2], [2, 3, 4, 3]),
                    {"degree": ("i32", "i32")})
    print("case: listing degree count", flush=True)
    rels, _, _ = engine_run(wl, workspace_bytes=256 << 20)
    exp = _golden("listing_agg_degree.txt")
    assert all(np.array_equal(a, b) for a, b in zip(rels["degree"], exp))


# ------------------------------------------------------------- small workloads, every row
@pytest.mark.parametrize("index_mode", [0, 1])
@pytest.mark.parametrize("name", list(W.small_workloads()))
def test_small_workload_matches_oracle(name, index_mode):
    """index_mode 0 picks dense bitmaps for small set domains, 1 forces hash tables."""
    wl = W.small_workloads()[name]()
    print(f"case: small {name} index_mode={index_mode} {wl.digest()[:12]}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"index_mode": index_mode})
    _compare(wl, rels, ref)
    assert stats["derived_tuples"] == sum(len(r[1][0]) for r in ref.relations.values())


@pytest.mark.parametrize("index_mode", [0, 1])
@pytest.mark.parametrize("name", ["tc_uniform", "sssp", "same_generation", "tc_rmat_count"])
def test_small_workload_with_forced_table_growth(name, index_mode):
    """A tiny initial table / row list forces overflow, growth and re-run of
    rounds in index mode 1; in mode 0 every head here is a dense array or
    bitmap over its key domain, which never grows."""
    wl = W.small_workloads()[name]()
    print(f"case: growth {name} index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"hash_min_log2": 10, "index_mode": index_mode})
    _compare(wl, rels, ref)
    if index_mode == 0:
        assert stats["table_grows"] == 0
    else:
        assert stats["table_grows"] > 0


@pytest.mark.parametrize("resident", [0, 1])
@pytest.mark.parametrize("pull_ratio", [0, 1, 64, 1024])
@pytest.mark.parametrize("name", ["tc_uniform", "tc_rmat_count"])
def test_closure_push_and_pull_directions(name, pull_ratio, resident):
    """Frontier rounds give the same closure whether sources push, pull or mix,
    launched one round at a time or all rounds of a source in one launch; the
    per-pass delta sizes are the oracle's in both."""
    wl = W.small_workloads()[name]()
    print(f"case: direction {name} pull_ratio={pull_ratio} resident={resident}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"pull_ratio": pull_ratio, "frontier_resident": resident,
                                             "profile": 1})
    _compare(wl, rels, ref)
    levels = _delta_levels(ref, "path")
    counts = [len(ref.relations["reach_count"][1][0])] if "reach_count" in ref.relations else []
    assert stats["delta_rows"] == levels + counts   # the count stratum records the rows it produced
    passes = len(ref.sizes["path"]) - 1
    assert stats["iterations"] == passes
    assert stats["front_launches"] == (1 if resident else passes)
    assert stats["front_new"] == len(ref.relations["path"][1][0]) - stats["delta_rows"][0]


# ------------------------------------------------------------- stratified negation
NEG_RULES = W.TC_RULES + """
blocked(X) :- edge(X, X).
oneway(X, Y) :- edge(X, Y), not edge(Y, X).
notfrom0(X, Y) :- edge(X, Y), not edge(0, Y).
noloop(X) :- edge(X, _), not edge(X, X).
unreached(X, Y) :- pair(X, Y), not path(X, Y).
safe(X, Y) :- edge(X, Y), not blocked(Y).
safe(X, Y) :- safe(X, Z), edge(Z, Y), not blocked(Y), not blocked(Z).
sink(Y) :- edge(_, Y), not edge(Y, _).
"""
NEG_IDB = {"path": ("i32", "i32"), "blocked": ("i32",), "oneway": ("i32", "i32"),
           "notfrom0": ("i32", "i32"), "noloop": ("i32",), "unreached": ("i32", "i32"),
           "safe": ("i32", "i32"), "sink": ("i32",)}


def test_listing_negation_degree():
    """The paper's aggregation listing with its integrity constraint written as
    a rule (no violations) and the sinks it implies (golden file)."""
    wl = W.Workload("neg_listing", """
degree(X, count(Y)) :- edge(X, Y).
violation(X) :- edge(X, _), not degree(X, _).
sink(Y) :- edge(_, Y), not degree(Y, _).
""", _edges([1, 1, 1, 2], [2, 3, 4, 3]), {"degree": ("i32", "i32"), "violation": ("i32",), "sink": ("i32",)})
    print("case: negation listing", flush=True)
    rels, _, _ = engine_run(wl, workspace_bytes=256 << 20)
    assert len(rels["violation"][0]) == 0
    assert np.array_equal(rels["sink"][0], _golden("listing_negation_degree.txt")[0])


_NEG_REF = {}


def _negation_case(n, m, seed):
    """Random edges plus three self-loops (so 'blocked' is never empty) and
    all pairs over the first min(n, 60) nodes; the oracle's result is kept
    for the second index mode."""
    if (n, m, seed) not in _NEG_REF:
        rng = np.random.default_rng(seed)
        src = np.concatenate([rng.integers(0, n, m), [5, 17, 33]])
        dst = np.concatenate([rng.integers(0, n, m), [5, 17, 33]])
        keep = np.unique(src * n + dst)
        src, dst = (keep // n).astype(np.int32), (keep % n).astype(np.int32)
        edb = _edges(src, dst)
        k = min(n, 60)
        px, py = np.meshgrid(np.arange(k), np.arange(k), indexing="ij")
        edb["pair"] = (("i32", "i32"), [px.ravel().astype(np.int32), py.ravel().astype(np.int32)])
        wl = W.Workload("negation", NEG_RULES, edb, NEG_IDB)
        _NEG_REF[(n, m, seed)] = (wl, evaluate(wl.rules, wl.edb, wl.idb))
    return _NEG_REF[(n, m, seed)]


@pytest.mark.parametrize("index_mode", [0, 1])
@pytest.mark.parametrize("n,m,seed", [(40, 90, 0), (300, 1500, 1), (700, 1000, 2)])
def test_negation_matches_oracle(n, m, seed, index_mode):
    """Set difference against an EDB relation (with a constant, a repeated
    variable, '_' columns), against a closure from an earlier stratum, and
    inside a recursive rule, in both head representations."""
    print(f"case: negation n={n} m={m} seed={seed} index_mode={index_mode}", flush=True)
    wl, ref = _negation_case(n, m, seed)
    rels, _, _ = engine_run(wl, options={"index_mode": index_mode})
    _compare(wl, rels, ref)
    assert sum(len(r[1][0]) for r in ref.relations.values()) > 0


# ------------------------------------------------------------- triangle join
def _tri_case(rels3, rules, idb_name="tri"):
    """(rules, edb) -> Workload with the given binary relations."""
    edb = {n: (("i32", "i32"), [np.asarray(a, np.int32), np.asarray(b, np.int32)]) for n, (a, b) in rels3.items()}
    return W.Workload("tri_case", rules, edb, {idb_name: ("i32", "i32", "i32")})


@pytest.mark.parametrize("shorter", [0, 1])
@pytest.mark.parametrize("rules", [
    "tri(X,Y,Z) :- r(X,Y), s(Y,Z), t(X,Z).",
    "tri(Z,X,Y) :- s(Y,Z), r(X,Y), t(Z,X).",
    "tri(X,Y,Z) :- t(Z,X), s(Z,Y), r(Y,X).",
    "tri(X,Y,Z) :- r(X,Y), r(Y,Z), r(X,Z).",
])
def test_triangle_join_matches_oracle(rules, shorter):
    """Any atom order, column order and head order, one relation playing all
    three roles, probing the shorter list or always b's: every row against
    the oracle, in ascending head-column order."""
    wl0 = W.small_workloads()["triangle"]()
    wl = W.Workload("tri", rules, wl0.edb, wl0.idb)
    print(f"case: triangle rules={rules!r} shorter={shorter}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"wcoj_shorter": shorter, "profile": 1})
    _compare(wl, rels, ref)
    assert stats["wcoj_new"] == len(ref.relations["tri"][1][0])
    assert stats["wcoj_launches"] == 2


def test_triangle_join_edge_cases():
    """Empty relations, no triangles, a single triangle, negative values and
    lists of very different lengths."""
    cases = [
        {"r": ([], []), "s": ([1], [2]), "t": ([1], [2])},
        {"r": ([1], [2]), "s": ([2], [3]), "t": ([1], [4])},
        {"r": ([-5], [7]), "s": ([7], [-9]), "t": ([-5], [-9])},
        {"r": ([0] * 50, list(range(50))), "s": ([3] * 3000 + [4], list(range(-1500, 1500)) + [0]),
         "t": ([0] * 7, [-1500, -3, 0, 17, 1499, 1500, 99999])},
    ]
    for k, rels3 in enumerate(cases):
        wl = _tri_case(rels3, W.TRIANGLE_RULES)
        print(f"case: triangle edge case {k}", flush=True)
        ref = evaluate(wl.rules, wl.edb, wl.idb)
        for shorter in (0, 1):
            rels, _, _ = engine_run(wl, workspace_bytes=256 << 20, options={"wcoj_shorter": shorter})
            _compare(wl, rels, ref)


@pytest.mark.parametrize("rules", ["tri(Z,X,Y) :- s(Y,Z), r(X,Y), t(Z,X).",
                                   "tri(X,Y,Z) :- t(Z,X), s(Z,Y), r(Y,X)."])
def test_triangle_value_order_keys_of_exactly_32_bits(rules):
    """Indexes sorted by (key, value) whose key and value columns each span
    exactly 2^16 values: the composite sort keys take all 32 bits of the
    32-bit form (relations the rule reads in another column order than the
    one they are stored in are sorted, not read as they are)."""
    big = 65535
    rels3 = {"r": ([0, 5, big, 7, 1], [1, 2, 3, big, big]),
             "s": ([1, 2, 3, big, 0, 0], [0, big, 9, 7, big, 1]),
             "t": ([0, 5, big, 0, 7], [0, big, 9, big, 7])}
    wl = _tri_case(rels3, rules)
    print(f"case: triangle 32-bit order keys {rules!r}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    assert len(ref.relations["tri"][1][0]) > 0
    rels, _, _ = engine_run(wl, workspace_bytes=256 << 20)
    _compare(wl, rels, ref)


def test_triangle_full_size_sampled_and_sound():
    """The 3 x 65,536-row fixture: rows of 400 sampled driver rows against the
    oracle, every triple satisfying all three atoms, strictly ascending
    output, and the total equal to the definition counted row by row."""
    wl = W.full_workloads()["triangle"]()
    print("case: triangle full size", flush=True)
    rels, stats, _ = engine_run(wl, options={"profile": 1})
    x, y, z = (c.astype(np.int64) for c in rels["tri"])
    assert min(x.min(), y.min(), z.min()) >= 0 and max(x.max(), y.max(), z.max()) < 2**17
    key = (x << 34) | (y << 17) | z
    assert np.all(np.diff(key) > 0)
    for (a, b), name in [((x, y), "r"), ((y, z), "s"), ((x, z), "t")]:
        c0, c1 = (cc.astype(np.int64) for cc in wl.edb[name][1])
        assert np.isin(a * 2**32 + b, c0 * 2**32 + c1).all()
    (r0, r1), (s0, s1), (t0, t1) = [wl.edb[k][1] for k in "rst"]
    S, T = {}, {}
    for u, v in zip(s0.tolist(), s1.tolist()):
        S.setdefault(u, set()).add(v)
    for u, v in zip(t0.tolist(), t1.tolist()):
        T.setdefault(u, set()).add(v)
    total = sum(len(S.get(v, set()) & T.get(u, set())) for u, v in zip(r0.tolist(), r1.tolist()))
    assert len(x) == total and total > 4_000_000
    rng = np.random.default_rng(21)
    pick = rng.choice(len(r0), 400, replace=False)
    edb = dict(wl.edb)
    edb["r"] = (("i32", "i32"), [r0[pick], r1[pick]])
    ref = evaluate(wl.rules, edb, wl.idb).relations["tri"][1]
    sel = np.isin(x * 2**32 + y, r0[pick].astype(np.int64) * 2**32 + r1[pick])
    for got, exp in zip((x[sel], y[sel], z[sel]), ref):
        assert np.array_equal(got, exp.astype(np.int64))
    assert stats["wcoj_candidates"] < 5_000_000  # the probes stay near the output size


# ------------------------------------------------------------- index reuse across runs
@pytest.mark.parametrize("name", ["tc_rmat_count", "triangle", "sssp", "same_generation"])
def test_index_cache_across_runs(name):
    """With "index_cache_mb" the second run of a program over unchanged inputs
    builds no input index again and gives the same rows; reloading an input
    invalidates its cached indexes, and a tiny budget (LRU eviction between
    runs) changes nothing in the results."""
    from paper_2609_27203_amd import xlh
    wl = W.small_workloads()[name]()
    print(f"case: index cache {name}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    for budget in (256, 1):
        ctx = xlh.Context(device=0, workspace_bytes=1 << 30)
        ctx.set_option("index_cache_mb", budget)
        for n, (t, cols) in wl.edb.items():
            ctx.relation(n, t).load(cols)
        for n, t in wl.idb.items():
            ctx.relation(n, t)
        prog = ctx.compile(wl.rules)
        seen = []
        for run in range(3):
            for n in wl.idb:
                ctx.relations[n].clear()
            if run == 2:  # new rows for one input: its cached indexes are stale
                first = sorted(wl.edb)[0]
                ctx.relations[first].load(wl.edb[first][1])
            st = prog.run()
            rels = {n: ctx.relations[n].read() for n in wl.idb}
            _compare(wl, rels, ref, f" run {run} budget {budget}")
            seen.append((st["index_builds"], st["index_reuses"]))
        if name == "sssp":  # tiled min rounds read their own (Z, tile) layout, built per run
            continue
        assert seen[0][0] > 0 and seen[0][1] == 0
        if budget == 256:
            assert seen[1][1] > 0 and seen[1][0] < seen[0][0]
            assert seen[2][0] > 0


# ------------------------------------------------------------- product joins
@pytest.mark.parametrize("index_mode", [0, 1])
@pytest.mark.parametrize("product", [0, 1])
def test_product_joins_match_oracle(product, index_mode):
    """Rules whose two join steps are both keyed by the driver row (same
    generation's recursive rule, a filtered variant, a non-recursive pair
    rule) give the oracle's rows with and without the one-launch product."""
    base = W.small_workloads()["same_generation"]()
    rules = W.SG_RULES + """
cousins(X,Y) :- parent(X,A), sg(A,B), parent(Y,B), X < Y.
pairs(X,Y) :- parent(A,X), parent(B,Y), parent(A,B).
"""
    wl = W.Workload("sg_product", rules, base.edb,
                    {"sg": ("i32", "i32"), "cousins": ("i32", "i32"), "pairs": ("i32", "i32")})
    print(f"case: product joins product={product} index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, _, _ = engine_run(wl, options={"product_joins": product, "index_mode": index_mode})
    _compare(wl, rels, ref)


def test_product_join_row_over_the_limit_runs_unfused():
    """A driver row whose product of match lists reaches 2^24 is refused by
    the one-launch kernel; the rule then runs again with the steps apart and
    the result is still complete."""
    n = 4096
    edb = {"d": (("i32", "i32"), [np.array([0, 1], np.int32), np.array([0, 1], np.int32)]),
           "p": (("i32", "i32"), [np.arange(n, dtype=np.int32), np.zeros(n, np.int32)]),
           "q": (("i32", "i32"), [np.arange(n + 1, dtype=np.int32),
                                   np.concatenate([np.zeros(n), [1]]).astype(np.int32)])}
    wl = W.Workload("big_product", "h(X,Y) :- d(A,B), p(X,A), q(Y,B).", edb, {"h": ("i32", "i32")})
    print("case: product over the limit", flush=True)
    rels, _, _ = engine_run(wl, options={"product_joins": 1})
    x, y = rels["h"]
    # (a, b) = (0, 0): 4096 X times 4096 Y = 2^24 products in one row; (1, 1): no X
    assert len(x) == n * n
    key = x.astype(np.int64) * n + y
    assert np.array_equal(key, np.arange(n * n, dtype=np.int64))


COUNT_SHAPES_RULES = W.TC_RULES + """
out_count(X,count(Y)) :- path(X,Y).
in_count(Y,count(X)) :- path(X,Y).
far_count(X,count(Y)) :- path(X,Y), Y > X.
back(X,Z) :- edge(X,Y), path(Y,Z).
back_count(X,count(Z)) :- back(X,Z).
"""


@pytest.mark.parametrize("index_mode", [0, 1])
def test_counts_and_joins_over_a_finished_closure(index_mode):
    """Counts grouped by the closure's first column (read from its row offsets
    when the closure ran in frontier form), by its second column, with a
    filter, and a later join probing the closure by its first column."""
    base = W.small_workloads()["tc_rmat_count"]()
    idb = {"path": ("i32", "i32"), "out_count": ("i32", "i32"), "in_count": ("i32", "i32"),
           "far_count": ("i32", "i32"), "back": ("i32", "i32"), "back_count": ("i32", "i32")}
    wl = W.Workload("count_shapes", COUNT_SHAPES_RULES, base.edb, idb)
    print(f"case: count shapes index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"index_mode": index_mode})
    _compare(wl, rels, ref)
    assert stats["derived_tuples"] == sum(len(r[1][0]) for r in ref.relations.values())


PULL_RULES = {
    # integer sum over derivations: the number of paths from each source
    "npaths": ("""
npaths(S,Y,sum(C)) :- source(S), C is 1, edge(S,Y,_).
npaths(S,Y,sum(C)) :- npaths(S,Z,C1), edge(Z,Y,_), C is C1.
""", {"npaths": ("i32", "i32", "i32")}),
    # logsumexp with a comparison on the joined edge
    "score_filtered": ("""
score(S,Y,logsumexp(P)) :- source(S), edge(S,Y,P).
score(S,Y,logsumexp(P)) :- score(S,Z,P1), edge(Z,Y,W), W > -2.0, P is P1 + W.
""", {"score": ("i32", "i32", "f32")}),
}


@pytest.mark.parametrize("index_mode", [0, 1])
@pytest.mark.parametrize("name", list(PULL_RULES))
def test_sum_and_logsumexp_heads_dense_and_hashed(name, index_mode):
    """Carried-value sum/logsumexp rules: index mode 0 keeps the head in dense
    slots and folds each key's contributions by scanning its in-edges, mode 1
    sorts and folds candidates into a hash table; both match the oracle."""
    rules, idb = PULL_RULES[name]
    wl = W.Workload(name, rules, W.small_workloads()["lse_dag"]().edb, idb)
    print(f"case: pull heads {name} index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"index_mode": index_mode})
    _compare(wl, rels, ref)
    assert stats["derived_tuples"] == sum(len(r[1][0]) for r in ref.relations.values())


SUBTRACT_RULES = {
    # min over D1 - W: f32 weights are log-probabilities (<= 0), so every
    # step adds -W >= 0; tiled min rounds with the one-subtract form
    "min_f32": ("""
low(S,S,min(D)) :- source(S), D is 0.0.
low(S,Y,min(D)) :- low(S,Z,D1), edge(Z,Y,W), D is D1 - W.
""", {"low": ("i32", "i32", "f32")}),
    # max over D1 - K on integer weights: the negated shortest path
    "max_i32": ("""
high(S,S,max(D)) :- source(S), D is 0.
high(S,Y,max(D)) :- high(S,Z,D1), iedge(Z,Y,K), D is D1 - K.
""", {"high": ("i32", "i32", "i32")}),
    # a sum seeded through subtraction (a recursive sum carries its value
    # unchanged: a subtracted term would act once per pass, not once)
    "sum_i32": ("""
ws(S,Y,sum(C)) :- source(S), iedge(S,Y,K), C is 0 - K.
ws(S,Y,sum(C)) :- ws(S,Z,C1), iedge(Z,Y,_), C is C1.
""", {"ws": ("i32", "i32", "i32")}),
    # logsumexp of P1 - W (the dense pull's one-subtract form: a log-domain product)
    "lse_f32": ("""
score(S,Y,logsumexp(P)) :- source(S), edge(S,Y,P).
score(S,Y,logsumexp(P)) :- score(S,Z,P1), edge(Z,Y,W), P is P1 - W.
""", {"score": ("i32", "i32", "f32")}),
    # logsumexp of P1 - W - 1 (the general form)
    "lse_f32_terms": ("""
score(S,Y,logsumexp(P)) :- source(S), edge(S,Y,P).
score(S,Y,logsumexp(P)) :- score(S,Z,P1), edge(Z,Y,W), P is P1 - W - 1.0.
""", {"score": ("i32", "i32", "f32")}),
    # set heads through subtraction: an id shifted back one layer, its closure,
    # and three-term arithmetic with a comparison on the result
    "set_i32": ("""
hop(X,Y) :- edge(X,Z,_), Y is Z - 300.
back(X,Y) :- hop(X,Y).
back(X,Y) :- back(X,Z), hop(Z,Y).
mix(X,V) :- iedge(X,Y,K), V is Y - X - K + 7, V > 290.
""", {"hop": ("i32", "i32"), "back": ("i32", "i32"), "mix": ("i32", "i32")}),
}


@pytest.mark.parametrize("index_mode", [0, 1])
@pytest.mark.parametrize("name", list(SUBTRACT_RULES))
def test_subtraction_rules_match_oracle(name, index_mode):
    """Rules whose arithmetic subtracts, through every value-head form (tiled
    min rounds, the dense pull, hashed folds, the stage kernel's one-op and
    general forms); integer and min/max results bit for bit, logsumexp
    within its tolerance."""
    rules, idb = SUBTRACT_RULES[name]
    base = W.small_workloads()["lse_dag"]()
    src, dst, w = base.edb["edge"][1]
    edb = dict(base.edb)
    edb["iedge"] = (("i32", "i32", "i32"), [src, dst, ((src * 7 + dst * 3) % 9 + 1).astype(np.int32)])
    used = {k: v for k, v in edb.items() if k + "(" in rules}
    wl = W.Workload(f"subtract_{name}", rules, used, idb)
    print(f"case: subtraction {name} index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"index_mode": index_mode})
    for rel, types in wl.idb.items():
        tol = value_tolerance(wl.rules, rel)
        assert_same_relation(rel, types, rels[rel], ref.relations[rel][1],
                             tol=tol if tol[0] == LSE_TOL else (0.0, 0.0))
        assert len(rels[rel][0]) > 0, rel
    assert stats["derived_tuples"] == sum(len(r[1][0]) for r in ref.relations.values())


@pytest.mark.parametrize("growth", [False, True])
@pytest.mark.parametrize("batch", [1, 4, 64])
@pytest.mark.parametrize("name", ["tc_uniform", "tc_rmat_count", "same_generation"])
def test_hash_set_rounds_batched(name, batch, growth):
    """Set heads held in hash tables (index mode 1) run batch rounds per host
    read, with the delta range on the device; with a tiny initial table the
    batches overflow and the host re-runs the round that stopped.  Rows,
    per-pass delta sizes and pass counts equal the round-by-round loop's."""
    wl = W.small_workloads()[name]()
    print(f"case: batched hash set rounds {name} batch={batch} growth={growth}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    opts = {"index_mode": 1, "batched_rounds": batch}
    if growth:
        opts["hash_min_log2"] = 10
    rels, stats, _ = engine_run(wl, options=opts)
    _compare(wl, rels, ref)
    base = engine_run(wl, options={"index_mode": 1, "batched_rounds": 0})[1]
    assert stats["delta_rows"] == base["delta_rows"] and stats["iterations"] == base["iterations"]
    if growth:
        assert stats["table_grows"] > 0


@pytest.mark.parametrize("batch", [0, 4, 64])
def test_hash_set_rounds_cap_and_round_count(batch):
    """A chain of n nodes closes in n - 1 passes: the iteration cap ends the
    run with XL_CONVERGENCE_FAILURE at the same pass batched or not, and with
    64 rounds per read the control bytes read do not grow with the number of
    rounds (chains of 20 and 50 nodes)."""
    from paper_2609_27203_amd import xlh
    reads = {}
    for n in (20, 50):
        src = np.arange(n - 1, dtype=np.int32)
        wl = W.Workload(f"chain{n}", W.TC_RULES, _edges(src, src + 1), {"path": ("i32", "i32")})
        print(f"case: hash chain n={n} batch={batch}", flush=True)
        opts = {"index_mode": 1, "batched_rounds": batch}
        rels, stats, _ = engine_run(wl, options=opts, workspace_bytes=256 << 20)
        assert len(rels["path"][0]) == n * (n - 1) // 2
        assert stats["iterations"] == n - 1 and stats["delta_rows"] == list(range(n - 1, -1, -1))
        reads[n] = stats["control_bytes_read"]
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, options=opts, max_iterations=n - 2, workspace_bytes=256 << 20)
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
        engine_run(wl, options=opts, max_iterations=n - 1, workspace_bytes=256 << 20)
    if batch == 64:
        assert reads[20] == reads[50]


def _value_workload(name):
    """A min/max/sum/logsumexp workload over the small layered DAG or the small
    SSSP graph (the aggregate heads of the batched keyed-table rounds)."""
    if name in ("sssp", "lse_dag"):
        return W.small_workloads()[name]()
    base = W.small_workloads()["lse_dag"]()
    if name in PULL_RULES:
        rules, idb = PULL_RULES[name]
        return W.Workload(name, rules, base.edb, idb)
    rules, idb = SUBTRACT_RULES[name]
    src, dst, _ = base.edb["edge"][1]
    edb = dict(base.edb)
    edb["iedge"] = (("i32", "i32", "i32"), [src, dst, ((src * 7 + dst * 3) % 9 + 1).astype(np.int32)])
    return W.Workload(name, rules, {k: v for k, v in edb.items() if k + "(" in rules}, idb)


def _compare_values(wl, rels, ref, where=""):
    for rel, types in wl.idb.items():
        tol = value_tolerance(wl.rules, rel)
        assert_same_relation(rel, types, rels[rel], ref.relations[rel][1], where,
                             tol=tol if tol[0] == LSE_TOL else (0.0, 0.0))


@pytest.mark.parametrize("growth", [False, True])
@pytest.mark.parametrize("batch", [1, 4, 64])
@pytest.mark.parametrize("name", ["sssp", "lse_dag", "npaths", "max_i32", "score_filtered"])
def test_hash_value_rounds_batched(name, batch, growth):
    """Min/max and sum/logsumexp heads held in hash tables (index mode 1) run
    batch rounds per host read: min/max candidates improve table values,
    sum/logsumexp candidates fold into per-slot accumulators, and each round's
    touched slots become the next delta on the device.  With a tiny initial
    table the batches overflow and the host re-runs the round that stopped.
    Min/max and integer sums match the oracle bit for bit, logsumexp within
    its tolerance; per-pass delta sizes and pass counts equal the
    round-by-round loop's."""
    wl = _value_workload(name)
    print(f"case: batched hash value rounds {name} batch={batch} growth={growth}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    opts = {"index_mode": 1, "batched_rounds": batch}
    if growth:
        opts["hash_min_log2"] = 10
    rels, stats, _ = engine_run(wl, options=opts)
    _compare_values(wl, rels, ref)
    base = engine_run(wl, options={"index_mode": 1, "batched_rounds": 0})[1]
    assert stats["delta_rows"] == base["delta_rows"] and stats["iterations"] == base["iterations"]
    if growth:
        assert stats["table_grows"] > 0


CHAIN_VALUE_RULES = {
    "min": (W.SSSP_RULES, {"dist": ("i32", "i32", "f32")}),
    "lse": (W.LSE_RULES, {"score": ("i32", "i32", "f32")}),
    "sum": (PULL_RULES["npaths"][0], {"npaths": ("i32", "i32", "i32")}),
}


@pytest.mark.parametrize("batch", [0, 4, 64])
@pytest.mark.parametrize("kind", list(CHAIN_VALUE_RULES))
def test_hash_value_rounds_cap_and_round_count(kind, batch):
    """A chain of n nodes from one source takes one pass per edge: in index
    mode 1 the iteration cap ends the run with XL_CONVERGENCE_FAILURE at the
    same pass batched or not, and with 64 rounds per read the control bytes
    read do not grow with the number of rounds (chains of 20 and 50 nodes)."""
    from paper_2609_27203_amd import xlh
    rules, idb = CHAIN_VALUE_RULES[kind]
    reads = {}
    for n in (20, 50):
        src = np.arange(n - 1, dtype=np.int32)
        w = np.full(n - 1, -0.5 if kind == "lse" else 1.5, np.float32)
        edb = {"source": (("i32",), [np.array([0], np.int32)]),
               "edge": (("i32", "i32", "f32"), [src, src + 1, w])}
        wl = W.Workload(f"{kind}_chain{n}", rules, edb, idb)
        print(f"case: hash value chain {kind} n={n} batch={batch}", flush=True)
        ref = evaluate(wl.rules, wl.edb, wl.idb)
        opts = {"index_mode": 1, "batched_rounds": batch}
        rels, stats, _ = engine_run(wl, options=opts, workspace_bytes=256 << 20)
        _compare_values(wl, rels, ref)
        base = engine_run(wl, options={"index_mode": 1, "batched_rounds": 0}, workspace_bytes=256 << 20)[1]
        passes = stats["iterations"]
        assert passes == base["iterations"] and stats["delta_rows"] == base["delta_rows"]
        assert passes >= n - 1
        reads[n] = stats["control_bytes_read"]
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, options=opts, max_iterations=passes - 1, workspace_bytes=256 << 20)
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
        engine_run(wl, options=opts, max_iterations=passes, workspace_bytes=256 << 20)
    if batch == 64:
        assert reads[20] == reads[50]


PARITY_RULES = """
odd(X,Y) :- edge(X,Y).
even(X,Y) :- odd(X,Z), edge(Z,Y).
odd(X,Y) :- even(X,Z), edge(Z,Y).
"""
PARITY_IDB = {"odd": ("i32", "i32"), "even": ("i32", "i32")}


@pytest.mark.parametrize("growth", [False, True])
@pytest.mark.parametrize("batch", [1, 4, 64])
@pytest.mark.parametrize("name", ["tc_uniform", "tc_rmat_count"])
def test_hash_mutual_recursion_batched(name, batch, growth):
    """Two set heads in one recursive stratum (walks of odd and of even
    length: each head's delta drives the other's rule), held in hash tables
    and batched: one row list, counter block and boundary list per head,
    rounds marked complete for both heads or for neither.  With a tiny
    initial table the batches overflow and the host re-runs the stopped
    round for both heads.  Rows, per-pass delta sizes and pass counts equal
    the round-by-round loop's; index mode 0 agrees too."""
    base = W.small_workloads()[name]()
    wl = W.Workload(f"parity_{name}", PARITY_RULES, {"edge": base.edb["edge"]}, PARITY_IDB)
    print(f"case: batched mutual recursion {name} batch={batch} growth={growth}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    opts = {"index_mode": 1, "batched_rounds": batch}
    if growth:
        opts["hash_min_log2"] = 10
    rels, stats, _ = engine_run(wl, options=opts)
    _compare(wl, rels, ref)
    round_by_round = engine_run(wl, options={"index_mode": 1, "batched_rounds": 0})[1]
    assert stats["delta_rows"] == round_by_round["delta_rows"]
    assert stats["iterations"] == round_by_round["iterations"]
    if growth:
        assert stats["table_grows"] > 0
    _compare(wl, engine_run(wl, options={"index_mode": 0})[0], ref, " (index mode 0)")


@pytest.mark.parametrize("batch", [0, 4, 64])
def test_hash_mutual_recursion_cap_and_control_reads(batch):
    """Odd/even walks along a chain of n nodes take n - 1 passes: the cap ends
    the run with XL_CONVERGENCE_FAILURE at the same pass batched or not, and
    at 64 rounds per read the control bytes read do not grow with the number
    of rounds (chains of 20 and 50 nodes)."""
    from paper_2609_27203_amd import xlh
    reads = {}
    for n in (20, 50):
        src = np.arange(n - 1, dtype=np.int32)
        wl = W.Workload(f"parity_chain{n}", PARITY_RULES, _edges(src, src + 1), PARITY_IDB)
        print(f"case: mutual recursion chain n={n} batch={batch}", flush=True)
        opts = {"index_mode": 1, "batched_rounds": batch}
        rels, stats, _ = engine_run(wl, options=opts, workspace_bytes=256 << 20)
        assert len(rels["odd"][0]) + len(rels["even"][0]) == n * (n - 1) // 2
        assert stats["iterations"] == n - 1 and stats["delta_rows"] == list(range(n - 1, -1, -1))
        reads[n] = stats["control_bytes_read"]
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, options=opts, max_iterations=n - 2, workspace_bytes=256 << 20)
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
        engine_run(wl, options=opts, max_iterations=n - 1, workspace_bytes=256 << 20)
    if batch == 64:
        assert reads[20] == reads[50]


@pytest.mark.parametrize("batch", [0, 4, 64])
def test_hash_same_generation_rounds_and_control_reads(batch):
    """Same generation in hash tables (index mode 1; the recursive rule joins
    both parent steps in one product launch): over two parallel chains under
    one root, pass k derives the pairs at depth k + 1, so the pass count
    grows with the depth while, at 64 rounds per read, the control bytes
    read do not (depths 10 and 30)."""
    reads = {}
    for depth in (10, 30):
        # node 0 is the root; chain a: 1..depth, chain b: depth+1..2*depth
        a = np.arange(1, depth + 1, dtype=np.int32)
        b = a + depth
        child = np.concatenate([a, b])
        par = np.concatenate([np.concatenate([[0], a[:-1]]), np.concatenate([[0], b[:-1]])]).astype(np.int32)
        wl = W.Workload(f"comb{depth}", W.SG_RULES, {"parent": (("i32", "i32"), [child, par])},
                        {"sg": ("i32", "i32")})
        print(f"case: hash same generation comb depth={depth} batch={batch}", flush=True)
        ref = evaluate(wl.rules, wl.edb, wl.idb)
        rels, stats, _ = engine_run(wl, options={"index_mode": 1, "batched_rounds": batch},
                                    workspace_bytes=256 << 20)
        _compare(wl, rels, ref)
        assert len(rels["sg"][0]) == 2 * depth
        assert stats["iterations"] == depth and stats["delta_rows"] == [2] * depth + [0]
        reads[depth] = stats["control_bytes_read"]
    if batch == 64:
        assert reads[10] == reads[30]


@pytest.mark.parametrize("batch", [0, 1, 4, 64])
@pytest.mark.parametrize("tiles", [-1, 0, 1, 7, 94])
def test_min_rounds_tiled_and_untiled(tiles, batch):
    """Carried min rule over a dense head: one workgroup per (source, tile of
    targets) with the tile in LDS (1 tile, 7 uneven tiles, the automatic
    choice, 94 tiles of 32 slots) or the untiled emission (-1), tiled rounds
    enqueued one at a time or in batches of 1, 4 or 64 per host read; all
    match the oracle bit for bit and give the same per-round delta sizes and
    pass count."""
    wl = W.small_workloads()["sssp"]()
    print(f"case: min tiles={tiles} batch={batch}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"dense_tiles": tiles, "batched_rounds": batch})
    assert_same_relation("dist", wl.idb["dist"], rels["dist"], ref.relations["dist"][1], tol=(0.0, 0.0))
    if tiles != -1 or batch:
        base = engine_run(wl, options={"dense_tiles": -1, "batched_rounds": 0})[1]
        assert stats["delta_rows"] == base["delta_rows"]
        assert stats["iterations"] == base["iterations"]


TILED_FORMS = {
    # Z in the edge relation's second column: the tiled index sorts the rows
    # by the whole (tile of Y, Z) key
    "swapped": ("dist(S,S,min(D)) :- source(S), D is 0.0.\n"
                "dist(S,Y,min(D)) :- dist(S,Z,D1), redge(Y,Z,W), D is D1 + W.", "redge", (1, 0, 2)),
    # a derived edge relation (a min head, not stored in sorted order)
    "derived": ("e2(Z,Y,min(W)) :- edge(Z,Y,W).\ndist(S,S,min(D)) :- source(S), D is 0.0.\n"
                "dist(S,Y,min(D)) :- dist(S,Z,D1), e2(Z,Y,W), D is D1 + W.", "edge", (0, 1, 2)),
}


@pytest.mark.parametrize("tiles", [0, 1, 7])
@pytest.mark.parametrize("form", list(TILED_FORMS))
def test_min_rounds_tiled_index_built_by_sort(form, tiles):
    """The tiled min rounds over an edge relation whose rows are not already
    in (Z, Y) order (Z in the second column, or a derived relation) build
    their (tile of Y, Z) index with a full key sort; they match the oracle bit
    for bit and the untiled emission's per-round delta sizes."""
    base_wl = W.small_workloads()["sssp"]()
    rules, name, perm = TILED_FORMS[form]
    types, cols = base_wl.edb["edge"]
    edb = {"source": base_wl.edb["source"],
           name: (tuple(types[k] for k in perm), [cols[k] for k in perm])}
    idb = {"dist": base_wl.idb["dist"]}
    if form == "derived":
        idb["e2"] = types
    wl = W.Workload(f"tiled_{form}", rules, edb, idb)
    print(f"case: tiled index by sort form={form} tiles={tiles}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"dense_tiles": tiles})
    assert_same_relation("dist", idb["dist"], rels["dist"], ref.relations["dist"][1], tol=(0.0, 0.0))
    base = engine_run(wl, options={"dense_tiles": -1, "batched_rounds": 0})[1]
    assert stats["iterations"] == base["iterations"]
    # the tiled rounds read their own (tile, Z) index; the untiled emission
    # builds an ordinary index of the edge relation
    assert stats["index_builds"] < base["index_builds"]


@pytest.mark.parametrize("batch", [0, 4])
def test_min_rounds_iteration_cap(batch):
    """A cap below the pass count is a convergence failure in both forms; the
    exact pass count converges."""
    from paper_2609_27203_amd import xlh
    wl = W.small_workloads()["sssp"]()
    print(f"case: min cap batch={batch}", flush=True)
    passes = engine_run(wl, options={"batched_rounds": 0})[1]["iterations"]
    for cap in (0, 1, passes - 1):
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, max_iterations=cap, options={"batched_rounds": batch})
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
    assert engine_run(wl, max_iterations=passes, options={"batched_rounds": batch})[1]["iterations"] == passes


@pytest.mark.parametrize("batch", [0, 1, 4, 64])
def test_pull_rounds_batched(batch):
    """Carried logsumexp rule over a dense head (one add, so the marks are the
    in-neighbours' delta presence): pull rounds one at a time or enqueued in
    batches of 1, 4 or 64 per host read with the key counts in device
    memory; the oracle's values within the logsumexp tolerance and the same
    per-round delta sizes and pass count either way."""
    wl = W.small_workloads()["lse_dag"]()
    print(f"case: pull rounds batch={batch}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"batched_rounds": batch, "profile": 1})
    _compare(wl, rels, ref)
    base = engine_run(wl, options={"batched_rounds": 0})[1]
    assert stats["delta_rows"] == base["delta_rows"]
    assert stats["iterations"] == base["iterations"] > 1
    # (one at a time, the last pass finds no marked key and launches nothing)
    assert stats["pull_launches"] == stats["iterations"] - (0 if batch else 1)


@pytest.mark.parametrize("batch", [0, 4])
def test_pull_rounds_iteration_cap(batch):
    """A cap below the pass count is a convergence failure in both forms; the
    exact pass count converges."""
    from paper_2609_27203_amd import xlh
    wl = W.small_workloads()["lse_dag"]()
    print(f"case: pull cap batch={batch}", flush=True)
    passes = engine_run(wl, options={"batched_rounds": 0})[1]["iterations"]
    for cap in (0, 1, passes - 1):
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, max_iterations=cap, options={"batched_rounds": batch})
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
    assert engine_run(wl, max_iterations=passes, options={"batched_rounds": batch})[1]["iterations"] == passes


SELF_JOIN_TC = """
path(X,Y) :- edge(X,Y).
path(X,Y) :- path(X,Z), path(Z,Y).
"""

SELF_JOIN_MIN = """
dist(X,Y,min(D)) :- edge(X,Y,D).
dist(X,Y,min(D)) :- dist(X,Z,D1), dist(Z,Y,D2), D is D1 + D2.
"""


@pytest.mark.parametrize("index_mode", [0, 1])
def test_self_join_closure_matches_oracle_and_doubles_path_length(index_mode):
    """Non-linear closure: two delta variants per round; after round k the
    relation holds every pair joined by a walk of length <= 2^k, so the
    per-round delta sizes equal the oracle's naive iterations."""
    base = W.tc_uniform(150, 600, 11)
    wl = W.Workload("tc_self_join", SELF_JOIN_TC, base.edb, {"path": ("i32", "i32")})
    print(f"case: self-join closure index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"index_mode": index_mode})
    _compare(wl, rels, ref)
    assert stats["delta_rows"] == _delta_levels(ref, "path")
    linear = evaluate(W.TC_RULES, base.edb, {"path": ("i32", "i32")})
    assert len(ref.sizes["path"]) < len(linear.sizes["path"])


@pytest.mark.parametrize("index_mode", [0, 1])
def test_self_join_min_matches_oracle(index_mode):
    """Non-linear shortest paths (dist joined with dist): integer-valued f32
    weights keep every sum exact, so the min fixpoint is compared bit for bit."""
    rng = np.random.default_rng(21)
    n, m = 120, 480
    src = rng.integers(0, n, 3 * m)
    dst = rng.integers(0, n, 3 * m)
    keep = src != dst
    pairs = np.unique(np.stack([src[keep], dst[keep]], 1), axis=0)[:m]
    wgt = rng.integers(1, 9, len(pairs)).astype(np.float32)
    edb = {"edge": (("i32", "i32", "f32"), [pairs[:, 0].astype(np.int32), pairs[:, 1].astype(np.int32), wgt])}
    wl = W.Workload("min_self_join", SELF_JOIN_MIN, edb, {"dist": ("i32", "i32", "f32")})
    print(f"case: self-join min index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, _, _ = engine_run(wl, options={"index_mode": index_mode})
    assert_same_relation("dist", wl.idb["dist"], rels["dist"], ref.relations["dist"][1], tol=(0.0, 0.0))


def _delta_levels(ref, name):
    sizes = ref.sizes[name]
    return [sizes[0]] + [b - a for a, b in zip(sizes, sizes[1:])]


def test_tc_delta_sizes_are_walk_levels():
    """Per-round |delta| of linear TC equals the number of pairs first joined at that walk length."""
    wl = W.small_workloads()["tc_uniform"]()
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    _, stats, _ = engine_run(wl)
    sizes = ref.sizes["path"]
    levels = [sizes[0]] + [b - a for a, b in zip(sizes, sizes[1:])]
    assert stats["delta_rows"] == levels
    assert stats["iterations"] == len(levels) - 1


# ------------------------------------------------------------- edge cases and errors
def test_empty_edb():
    wl = W.Workload("empty", W.TC_COUNT_RULES, _edges([], []),
                    {"path": ("i32", "i32"), "reach_count": ("i32", "i32")})
    rels, stats, _ = engine_run(wl, workspace_bytes=256 << 20)
    assert len(rels["path"][0]) == 0 and len(rels["reach_count"][0]) == 0
    assert stats["iterations"] == 0


@pytest.mark.parametrize("resident", [0, 1])
def test_closure_and_count_over_many_first_keys(resident):
    """20,000 first keys in chains of 8 nodes (a ragged last chain): the
    per-key row counts are scanned by one workgroup walking 4,096-value
    tiles (4,097 to 65,536 values), and the count head, 20,000 slots, is
    compacted in one pass with its row count and value bounds in one read."""
    n, chain = 20_000, 8
    src = np.array([i for i in range(n - 1) if (i + 1) % chain], np.int64)
    wl = W.Workload("chains", W.TC_COUNT_RULES, _edges(src, src + 1),
                    {"path": ("i32", "i32"), "reach_count": ("i32", "i32")})
    print(f"case: chains n={n} resident={resident}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"frontier_resident": resident})
    _compare(wl, rels, ref)
    assert stats["iterations"] == chain - 1
    counts = rels["reach_count"][1]
    assert counts.min() == 1 and counts.max() == chain - 1


@pytest.mark.parametrize("resident", [0, 1])
def test_closure_seeded_by_two_rules(resident):
    """The seed round of the closure has two rules (edge, then a second edge
    relation): the resident launch starts only after both have inserted, so
    paths that begin with an edge of the second relation are found too."""
    rng = np.random.default_rng(17)
    edb = _edges(rng.integers(0, 300, 1200), rng.integers(0, 300, 1200))
    edb["extra"] = (("i32", "i32"), [rng.integers(0, 300, 400).astype(np.int32),
                                     rng.integers(0, 300, 400).astype(np.int32)])
    rules = ("path(X, Y) :- edge(X, Y).\npath(X, Y) :- extra(X, Y).\n"
             "path(X, Z) :- path(X, Y), edge(Y, Z).")
    wl = W.Workload("two_seeds", rules, edb, {"path": ("i32", "i32")})
    print(f"case: closure seeded by two rules resident={resident}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"frontier_resident": resident, "profile": 1})
    _compare(wl, rels, ref)
    assert stats["iterations"] == len(ref.sizes["path"]) - 1
    assert stats["front_launches"] == (1 if resident else stats["iterations"])


@pytest.mark.parametrize("resident", [0, 1])
def test_closure_whose_seed_derives_nothing(resident):
    """A seed rule whose filter rejects every edge: the closure stays empty,
    no round runs, and the count stratum after it sees no rows."""
    wl = W.Workload("empty_seed", "path(X, Y) :- edge(X, Y), X > 1000.\n"
                                  "path(X, Z) :- path(X, Y), edge(Y, Z).\n"
                                  "reach_count(X, count(Y)) :- path(X, Y).",
                    _edges([1, 2, 3, 4], [2, 3, 4, 1]), {"path": ("i32", "i32"), "reach_count": ("i32", "i32")})
    print(f"case: closure with an empty seed resident={resident}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"frontier_resident": resident}, workspace_bytes=256 << 20)
    _compare(wl, rels, ref)   # both relations empty, as in the oracle
    assert stats["iterations"] == 0


def test_self_loop_and_duplicates():
    wl = W.Workload("loops", W.TC_RULES, _edges([0, 0, 1, 1, 2], [0, 1, 2, 2, 0]), {"path": ("i32", "i32")})
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, _, _ = engine_run(wl, workspace_bytes=256 << 20)
    _compare(wl, rels, ref)


@pytest.mark.parametrize("index_mode", [0, 1])
def test_negative_ids_and_wide_key_range(index_mode):
    """Keys spread over almost the whole int32 range: the join index is
    compacted (distinct keys found by binary search) instead of direct."""
    src = np.array([-2_000_000_000, -5, 7, 1_900_000_000], np.int32)
    dst = np.array([-5, 7, 1_900_000_000, -2_000_000_000], np.int32)
    wl = W.Workload("wide", W.TC_RULES, _edges(src, dst), {"path": ("i32", "i32")})
    print(f"case: wide key range index_mode={index_mode}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, _, _ = engine_run(wl, workspace_bytes=256 << 20, options={"index_mode": index_mode})
    _compare(wl, rels, ref)
    assert len(rels["path"][0]) == 16


def _relabel(wl, span, seed, cols_by_rel):
    """The workload with every node id i replaced by ids[i]: distinct values
    ascending in i, spread over [lo, lo + span) (order kept, so the rows map
    one to one)."""
    rng = np.random.default_rng(seed)
    n = max(int(c.max()) for name, cs in cols_by_rel.items() for j in cs for c in [wl.edb[name][1][j]]) + 1
    ids = np.sort(rng.choice(span, n, replace=False)).astype(np.int64) - span // 2
    ids = ids.astype(np.int32)
    edb = {}
    for name, (types, cols) in wl.edb.items():
        cols = [ids[c] if j in cols_by_rel.get(name, ()) else c for j, c in enumerate(cols)]
        edb[name] = (types, cols)
    return W.Workload(wl.name + "_sparse", wl.rules, edb, wl.idb)


SPARSE_CASES = {
    # (small workload, columns holding node ids per relation)
    "tc_uniform": ("tc_uniform", {"edge": (0, 1)}),
    "sssp": ("sssp", {"edge": (0, 1), "source": (0,)}),
    "lse_dag": ("lse_dag", {"edge": (0, 1), "source": (0,)}),
    "same_generation": ("same_generation", {"parent": (0, 1)}),
    "triangle": ("triangle", {"r": (0, 1), "s": (0, 1), "t": (0, 1)}),
}


@pytest.mark.parametrize("span", [1 << 28, 4_000_000_000])
@pytest.mark.parametrize("name", list(SPARSE_CASES))
def test_sparse_and_wide_node_ids(name, span):
    """The reduced workloads with node ids drawn sparsely from 2^28 values or
    from almost all of int32: joins go through compacted indexes (hash-table
    heads, since the key domains are far too wide for bitmaps)."""
    base, cols = SPARSE_CASES[name]
    wl = _relabel(W.small_workloads()[base](), span, 17, cols)
    print(f"case: sparse ids {name} span={span}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl)
    _compare(wl, rels, ref)
    assert stats["derived_tuples"] == sum(len(r[1][0]) for r in ref.relations.values())


def test_join_key_with_2_26_rows_is_refused():
    """One key holding 2^26 rows of the indexed relation would overflow the
    stage kernel's 32-bit match count per wavefront: the run reports
    XL_UNSUPPORTED (the kernel skips that key's matches, so nothing is read
    out of bounds), and one row fewer runs."""
    from paper_2609_27203_amd import xlh
    for n, ok in (((1 << 26) - 1, True), (1 << 26, False)):
        v = np.arange(n, dtype=np.int32)
        wl = W.Workload("hub", "out(V) :- d(K), e(K, V), V < 3.",
                        {"d": (("i32",), [np.zeros(1, np.int32)]), "e": (("i32", "i32"), [np.zeros(n, np.int32), v])},
                        {"out": ("i32",)})
        print(f"case: hub key with {n} rows", flush=True)
        if ok:
            rels, _, _ = engine_run(wl, workspace_bytes=8 << 30)
            assert rels["out"][0].tolist() == [0, 1, 2]
        else:
            with pytest.raises(xlh.XlError) as ei:
                engine_run(wl, workspace_bytes=8 << 30)
            assert ei.value.status_name == "XL_UNSUPPORTED" and "2^26" in str(ei.value)


def test_sparse_ids_self_join_and_later_stratum():
    """Self-joined recursion and a later join over the finished closure, with
    sparse ids: the head snapshots and the closure are indexed compacted."""
    wl0 = _relabel(W.small_workloads()["tc_uniform"](), 1 << 29, 5, {"edge": (0, 1)})
    rules = ("path(X,Y) :- edge(X,Y).\npath(X,Y) :- path(X,Z), path(Z,Y).\n"
             "into(Z) :- edge(_,Y), path(Z,Y).\nback(X,Z) :- edge(X,Y), path(Y,Z), Z < X.\n")
    wl = W.Workload("sparse_self_join", rules, wl0.edb,
                    {"path": ("i32", "i32"), "into": ("i32",), "back": ("i32", "i32")})
    print("case: sparse ids self-join", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, _, _ = engine_run(wl)
    _compare(wl, rels, ref)


@pytest.mark.parametrize("resident", [0, 1])
def test_iteration_cap_is_convergence_failure(resident):
    """A chain of 6 nodes needs 5 passes (deltas 4, 3, 2, 1, 0 after the
    seed): a cap of 5 converges, 4 and 0 do not."""
    from paper_2609_27203_amd import xlh
    n = 6
    wl = W.Workload("chain", W.TC_RULES, _edges(np.arange(n - 1), np.arange(1, n)), {"path": ("i32", "i32")})
    print(f"case: iteration cap resident={resident}", flush=True)
    opts = {"frontier_resident": resident}
    for cap in (0, 1, 4):
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, workspace_bytes=256 << 20, max_iterations=cap, options=opts)
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
    rels, stats, _ = engine_run(wl, workspace_bytes=256 << 20, max_iterations=5, options=opts)
    assert stats["iterations"] == 5 and stats["delta_rows"] == [5, 4, 3, 2, 1, 0]
    assert len(rels["path"][0]) == n * (n - 1) // 2


def test_capacity_and_workspace_errors():
    from paper_2609_27203_amd import xlh
    wl = W.small_workloads()["tc_uniform"]()
    ctx = xlh.Context(device=0, workspace_bytes=256 << 20)
    ctx.relation("edge", ("i32", "i32"))
    ctx.relation("path", ("i32", "i32"), max_rows=1000)
    with pytest.raises(xlh.XlError) as ei:
        engine_run(wl, ctx=ctx)
    assert ei.value.status_name == "XL_CAPACITY_EXCEEDED"
    small = xlh.Context(device=0, workspace_bytes=2 << 20)
    small.relation("edge", ("i32", "i32"))
    small.relation("path", ("i32", "i32"))
    with pytest.raises(xlh.XlError) as ei:
        engine_run(wl, ctx=small)
    assert ei.value.status_name == "XL_RESOURCE_EXHAUSTED"


def _gather_workload(variant):
    if variant.startswith("sg"):
        base = W.small_workloads()["same_generation"]()
        rules = base.rules if variant == "sg" else (
            "sg(X,Y) :- parent(X,P), parent(Y,P), X != Y.\nsg(X,Y) :- sg(A,B), parent(Y,B), parent(X,A).")
        return W.Workload(variant, rules, base.edb, base.idb), "sg"
    e_src, e_dst = W.uniform_graph(300, 900, 31)
    f_src, f_dst = W.uniform_graph(300, 600, 32)
    edb = {"e": (("i32", "i32"), [np.asarray(e_src, np.int32), np.asarray(e_dst, np.int32)]),
           "f": (("i32", "i32"), [np.asarray(f_src, np.int32), np.asarray(f_dst, np.int32)])}
    if variant == "func":  # e1 pairs every X with exactly one A (a random function, with cycles)
        g = np.random.default_rng(33)
        edb["p"] = (("i32", "i32"), [np.arange(300, dtype=np.int32), g.integers(0, 300, 300).astype(np.int32)])
    rules = {"dag": "h(X,Y) :- e(X,Y).\nh(X,Y) :- e(X,A), h(A,B), f(Y,B).",
             "dag_swapped": "h(X,Y) :- e(Y,X).\nh(X,Y) :- e(A,X), h(A,B), f(B,Y).",
             "func": "h(X,Y) :- e(X,Y).\nh(X,Y) :- p(X,A), h(A,B), f(Y,B)."}[variant]
    return W.Workload(variant, rules, edb, {"h": ("i32", "i32")}), "h"


@pytest.mark.parametrize("gather,batch", [(0, 4), (1, 0), (1, 1), (1, 4), (1, 64), (2, 0), (2, 4)])
@pytest.mark.parametrize("variant", ["sg", "sg_reordered", "dag", "dag_swapped", "func"])
def test_gathered_rounds(variant, gather, batch):
    """h(X,Y) :- e1(X,A), delta h(A,B), e2(Y,B) in gathered rounds (1: per
    delta row A, the union of its Y values ORed into the rows of A's X
    values; 2: head row X staged in LDS, the Y values of the B bits of its A
    values' delta rows set there; one round or 1, 4 or 64 rounds per host
    read) and in the generic join: the oracle's rows and per-round delta
    sizes either way,
    also over random graphs where an X has many A (several
    delta rows per head row, one delta row read for many X), where e1 is a
    random function (one A per X, cycles), and with the columns and atoms in
    other orders."""
    wl, head = _gather_workload(variant)
    print(f"case: gathered rounds {variant} gather={gather} batch={batch}", flush=True)
    ref = evaluate(wl.rules, wl.edb, wl.idb)
    rels, stats, _ = engine_run(wl, options={"gather_rounds": gather, "batched_rounds": batch, "profile": 1})
    _compare(wl, rels, ref)
    levels = _delta_levels(ref, head)
    assert stats["delta_rows"][:len(levels)] == levels
    assert stats["iterations"] == len(ref.sizes[head]) - 1
    if gather:
        assert stats["gather_launches"] == stats["iterations"] and stats["gather_new"] == sum(levels[1:])
    else:
        assert stats["gather_launches"] == 0


@pytest.mark.parametrize("batch", [0, 4])
def test_gathered_rounds_iteration_cap(batch):
    """Gathered rounds one at a time or batched: a cap below the pass count is
    a convergence failure, the exact pass count converges."""
    from paper_2609_27203_amd import xlh
    wl, _ = _gather_workload("sg")
    print(f"case: gathered cap batch={batch}", flush=True)
    passes = engine_run(wl, options={"batched_rounds": 0})[1]["iterations"]
    for cap in (0, 1, passes - 1):
        with pytest.raises(xlh.XlError) as ei:
            engine_run(wl, max_iterations=cap, options={"batched_rounds": batch})
        assert ei.value.status_name == "XL_CONVERGENCE_FAILURE"
    assert engine_run(wl, max_iterations=passes, options={"batched_rounds": batch})[1]["iterations"] == passes


def test_resume_from_fixpoint_is_idempotent():
    wl = W.small_workloads()["same_generation"]()
    rels, _, ctx = engine_run(wl)
    ctx.relations["sg"].load(rels["sg"])
    prog = ctx.compile(wl.rules)
    stats = prog.run()
    assert stats["delta_rows"][0] == 0 and stats["iterations"] == 0
    again = ctx.relations["sg"].read()
    assert all(np.array_equal(a, b) for a, b in zip(again, rels["sg"]))


def test_min_resume_from_fixpoint_is_idempotent():
    wl = W.small_workloads()["sssp"]()
    rels, _, ctx = engine_run(wl)
    ctx.relations["dist"].load(rels["dist"])
    stats = ctx.compile(wl.rules).run()
    assert stats["delta_rows"][0] == 0
    again = ctx.relations["dist"].read()
    assert all(np.array_equal(a.view(np.int32), b.view(np.int32)) for a, b in zip(again, rels["dist"]))


def test_repeat_runs_are_identical():
    for name in ("tc_rmat_count", "sssp", "lse_dag"):
        wl = W.small_workloads()[name]()
        a, _, ctx = engine_run(wl)
        b, _, _ = engine_run(wl, ctx=ctx)
        for rel in wl.idb:
            for x, y in zip(a[rel], b[rel]):
                assert np.array_equal(x.view(np.int32), y.view(np.int32)), (name, rel)


def test_device_columns_round_trip():
    import torch
    from paper_2609_27203_amd import xlh
    wl = W.small_workloads()["tc_uniform"]()
    ctx = xlh.Context(device=0, workspace_bytes=512 << 20)
    ctx.relation("edge", ("i32", "i32"))
    ctx.relation("path", ("i32", "i32"))
    src, dst = wl.edb["edge"][1]
    ctx.relations["edge"].load([torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda()])
    ctx.compile(wl.rules).run()
    dev = ctx.relations["path"].read_device()
    host = ctx.relations["path"].read()
    assert all(np.array_equal(d.cpu().numpy(), h) for d, h in zip(dev, host))
