"""Host-only checks (no GPU): the C-ABI library loads and exports what the
header declares, and the planner accepts, plans and rejects rule forms."""
import os
import re

import pytest

from paper_2609_27203_amd import workloads as W
from paper_2609_27203_amd import xlh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "xlh.h")).read()
    declared = set(re.findall(r"\b(xl_[a-z_]+)\s*\(", header))
    lib = xlh.lib()
    missing = [name for name in sorted(declared) if not hasattr(lib, name)]
    assert not missing, missing
    assert declared == set(xlh.EXPORTS)


def test_status_strings():
    lib = xlh.lib()
    for i, name in enumerate(xlh.STATUS):
        assert lib.xl_status_string(i).decode() == name


def _ctx(rels):
    c = xlh.Context(device=-1)
    for name, types in rels.items():
        c.relation(name, types)
    return c


@pytest.mark.parametrize("name", list(W.full_workloads()))
def test_workload_programs_compile(name):
    wl = W.small_workloads()[name]()
    c = _ctx({**{k: t for k, (t, _) in wl.edb.items()}, **wl.idb})
    plan = c.compile(wl.rules).explain()
    assert "recursive" in plan
    if name == "tc_rmat_count":
        assert plan.index("stratum 0 recursive heads: path") < plan.index("stratum 1 non-recursive heads: reach_count[count]")
    if name == "same_generation":   # delta variant joins parent twice, both by the parent column
        assert "delta sg(v0,v1) -> join parent on col 1=v0 (v2,_) -> join parent on col 1=v1 (v3,_)" in plan
        assert "[gathered by head row v2]" in plan  # h(X,Y) :- e1(X,A), delta h(A,B), e2(Y,B)
    if name == "tc_rmat_count":
        assert "[gathered" not in plan


def test_delta_variant_per_recursive_atom():
    c = _ctx({"e": ("i32", "i32"), "p": ("i32", "i32"), "q": ("i32", "i32")})
    plan = c.compile("p(X,Y) :- e(X,Y).\np(X,Y) :- q(X,Z), e(Z,Y).\nq(X,Y) :- p(X,Y).").explain()
    assert "stratum 0 recursive heads: p[set] q[set]" in plan or "stratum 0 recursive heads: q[set] p[set]" in plan
    assert plan.count("  delta rule") == 2


I2 = ("i32", "i32")
W3 = ("i32", "i32", "f32")


def test_negated_literals_are_planned_as_membership_tests():
    """A negated literal over a relation of an earlier stratum is a membership
    test on the constrained columns, after the atoms that bind them; a rule
    with one is not run in the grouped closure form."""
    c = _ctx({"e": I2, "b": ("i32",), "p": I2})
    plan = c.compile("b(X) :- e(X,X).\np(X,Y) :- e(X,Y), not b(Y).\n"
                     "p(X,Y) :- p(X,Z), e(Z,Y), not b(Y), not e(Y, 0).").explain()
    lines = plan.splitlines()
    assert lines[0].startswith("stratum 0") and "b[set]" in lines[0]
    assert any("-> not b(cols 0)" in ln and "seed" in ln for ln in lines)
    delta = [ln for ln in lines if ln.startswith("  delta rule")]
    assert len(delta) == 1 and "-> not b(cols 0) -> not e(cols 0 1)" in delta[0]
    assert "grouped" not in delta[0]


def test_triangle_rules_become_one_worst_case_optimal_join():
    """Any column order of the three atoms and any head order: the driver is
    the atom over the first two head variables."""
    c = _ctx({"r": I2, "s": I2, "t": I2, "tri": ("i32", "i32", "i32")})
    plan = c.compile("tri(Z,X,Y) :- s(Y,Z), r(X,Y), t(Z,X).").explain()
    line = [ln for ln in plan.splitlines() if "triangle join" in ln][0]
    # head columns (Z, X, Y) play the roles X, Y, Z: a = t over (Z, X), b = r
    # over (X, Y), c = s over (Z, Y)
    assert "t(X=col 0, Y=col 1) x r(Y=col 0, Z=col 1) x s(X=col 1, Z=col 0) -> tri(X,Y,Z)" in line


def test_self_join_gets_one_delta_variant_per_recursive_atom():
    """Alg. 1: a rule with two recursive atoms has two delta variants, each
    scanning the delta at one atom and joining the full relation at the other."""
    c = _ctx({"e": I2, "p": I2})
    plan = c.compile("p(X,Y) :- e(X,Y).\np(X,Y) :- p(X,Z), p(Z,Y).").explain()
    variants = [ln for ln in plan.splitlines() if ln.startswith("  delta rule")]
    assert len(variants) == 2
    assert "delta p(v0,v1) -> join p on col 0=v1" in variants[0]
    assert "delta p(v0,v1) -> join p on col 1=v0" in variants[1]


@pytest.mark.parametrize("rels,text,status", [
    ({"e": I2, "p": I2}, "p(X,Y) :- e(X,Y", "XL_PARSE_ERROR"),
    ({"e": I2, "p": I2}, "p(X,Y) :- e(X,Y) e(Y,Z).", "XL_PARSE_ERROR"),
    ({"e": I2, "p": I2}, "p(1,2).", "XL_PARSE_ERROR"),
    ({"e": I2, "p": I2}, "p(X,Y) :- nope(X,Y).", "XL_INVALID_ARGUMENT"),
    ({"e": I2, "p": I2}, "p(X,Y) :- e(X,Y,Z).", "XL_INVALID_ARGUMENT"),
    ({"e": I2, "p": I2}, "p(X,Y,count(Z)) :- e(X,Y), e(Y,Z).", "XL_INVALID_ARGUMENT"),
    ({"e": I2, "c": I2}, "c(X,count(Y)) :- c(X,Z), e(Z,Y).", "XL_UNSUPPORTED"),
    ({"w": W3, "s": W3}, "s(X,Y,logsumexp(P)) :- w(X,Y,P).\ns(X,Y,logsumexp(P)) :- s(X,Z,P1), s(Z,Y,P2), P is P1 + P2.",
     "XL_UNSUPPORTED"),
    ({"e": I2, "f": I2, "p": I2}, "p(X,Y) :- e(X,A), f(B,Y).", "XL_UNSUPPORTED"),
    ({"w": W3, "p": ("f32", "i32")}, "p(W,Y) :- w(X,Y,W).", "XL_UNSUPPORTED"),
    ({"w": W3, "p": I2}, "p(X,W) :- w(X,Y,W).", "XL_TYPE_MISMATCH"),
    ({"w": W3, "e": I2, "p": I2}, "p(X,Y) :- w(X,Y,W), e(W,Y).", "XL_TYPE_MISMATCH"),
    ({"w": W3, "p": W3}, "p(X,Y,logsumexp(D)) :- w(X,Y,W), D is W + 1.", "XL_TYPE_MISMATCH"),
    ({"w": W3, "p": ("i32", "i32", "i32")}, "p(X,Y,logsumexp(Y)) :- w(X,Y,_).", "XL_TYPE_MISMATCH"),
    ({"e": I2, "p": I2}, "p(X,Y) :- e(X,Y), Y is X + 1.", "XL_UNSUPPORTED"),
    ({"e": I2, "p": I2}, "p(X,Z) :- e(X,Y).", "XL_UNSUPPORTED"),
    ({"e": I2, "p": I2, "m": ("i32", "i32", "i32")},
     "m(X,Y,min(Y)) :- e(X,Y).\nm(X,Y,max(Y)) :- e(Y,X).", "XL_UNSUPPORTED"),
    # stratified negation: no negative edge inside a recursive component, every
    # variable of a negated literal bound positively, int32 columns, at most
    # two constrained columns and two negated literals per rule
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,_), not p(X).", "XL_UNSUPPORTED"),
    ({"e": I2, "p": ("i32",), "q": ("i32",)}, "p(X) :- e(X,_), not q(X).\nq(X) :- e(_,X), not p(X).",
     "XL_UNSUPPORTED"),
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,_), not e(X,Z).", "XL_UNSUPPORTED"),
    ({"w": W3, "p": ("i32",)}, "p(X) :- w(X,_,W), not w(X,_,W).", "XL_UNSUPPORTED"),
    ({"t": ("i32", "i32", "i32"), "p": ("i32",)}, "p(X) :- t(X,Y,Z), not t(Z,Y,X).", "XL_UNSUPPORTED"),
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,Y), not e(Y,X), not e(X,X), not e(Y,Y).", "XL_UNSUPPORTED"),
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,_), not nope(X).", "XL_INVALID_ARGUMENT"),
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,_), not e(X).", "XL_INVALID_ARGUMENT"),
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,_), not e(X, 1.5).", "XL_TYPE_MISMATCH"),
    # three-column heads: only one non-recursive triangle join rule
    ({"e": I2, "h": ("i32", "i32", "i32")}, "h(X,Y,Z) :- e(X,Y), e(Y,Z).", "XL_UNSUPPORTED"),
    ({"e": I2, "h": ("i32", "i32", "i32")}, "h(X,Y,Z) :- e(X,Y), e(Y,Z), e(X,Z), X != Z.", "XL_UNSUPPORTED"),
    ({"e": I2, "h": ("i32", "i32", "i32")},
     "h(X,Y,Z) :- e(X,Y), e(Y,Z), e(X,Z).\nh(X,Y,Z) :- e(Y,X), e(Y,Z), e(X,Z).", "XL_UNSUPPORTED"),
    ({"e": I2, "h": ("i32", "i32", "i32")}, "h(X,Y,Z) :- e(X,Y), e(Y,Z), h(X,Z,Y).", "XL_UNSUPPORTED"),
    ({"e": I2, "h": ("i32", "i32", "i32")}, "h(X,Y,Y) :- e(X,Y), e(Y,Y), e(X,Y).", "XL_UNSUPPORTED"),
    # a recursive sum carries the recursive atom's value unchanged, a
    # recursive logsumexp adds terms to it, and neither compares it: folding
    # each pass's contributions then gives the naive fixpoint's values
    ({"w": ("i32", "i32", "i32"), "s": ("i32", "i32", "i32")},
     "s(X,Y,sum(C)) :- w(X,Y,C).\ns(X,Y,sum(C)) :- s(X,Z,C1), w(Z,Y,K), C is C1 - K.", "XL_UNSUPPORTED"),
    ({"w": ("i32", "i32", "i32"), "s": ("i32", "i32", "i32")},
     "s(X,Y,sum(C)) :- w(X,Y,C).\ns(X,Y,sum(C)) :- s(X,Z,C1), w(Z,Y,C).", "XL_UNSUPPORTED"),
    ({"w": ("i32", "i32", "i32"), "s": ("i32", "i32", "i32")},
     "s(X,Y,sum(C)) :- w(X,Y,C).\ns(X,Y,sum(C)) :- s(X,Z,C1), w(Z,Y,_), C1 > 3, C is C1.", "XL_UNSUPPORTED"),
    ({"w": W3, "s": W3}, "s(X,Y,logsumexp(P)) :- w(X,Y,P).\ns(X,Y,logsumexp(P)) :- s(X,Z,P1), w(Z,Y,W), P is W - P1.",
     "XL_UNSUPPORTED"),
    ({"w": W3, "s": W3}, "s(X,Y,logsumexp(P)) :- w(X,Y,P).\ns(X,Y,logsumexp(P)) :- s(X,Z,_), w(Z,Y,P).",
     "XL_UNSUPPORTED"),
    # min and max: each carried value at most once, added, and not compared
    ({"w": W3, "d": W3}, "d(X,Y,min(D)) :- w(X,Y,D).\nd(X,Y,min(D)) :- d(X,Z,D1), w(Z,Y,W), D is W - D1.",
     "XL_UNSUPPORTED"),
    ({"w": W3, "d": W3}, "d(X,Y,min(D)) :- w(X,Y,D).\nd(X,Y,min(D)) :- d(X,Z,D1), w(Z,Y,W), D1 > 1.0, D is D1 + W.",
     "XL_UNSUPPORTED"),
    ({"w": W3, "d": W3}, "d(X,Y,max(D)) :- w(X,Y,D).\nd(X,Y,max(D)) :- d(X,Z,D1), w(Z,Y,_), D is D1 + D1.",
     "XL_UNSUPPORTED"),
])
def test_rejected_programs(rels, text, status):
    c = _ctx(rels)
    with pytest.raises(xlh.XlError) as ei:
        c.compile(text)
    assert ei.value.status_name == status, str(ei.value)


U2 = ("u64", "u64")


@pytest.mark.parametrize("rels,text,status", [
    # a variable keeps one declared type; constants must be values of the
    # column type they meet
    ({"e": U2, "f": I2, "p": ("u64",)}, "p(X) :- e(X,Y), f(Y,_).", "XL_TYPE_MISMATCH"),
    ({"e": U2, "p": ("i64",)}, "p(X) :- e(X,_).", "XL_TYPE_MISMATCH"),
    ({"e": ("u32", "u32"), "p": ("u32",)}, "p(X) :- e(X,-1).", "XL_TYPE_MISMATCH"),
    ({"e": I2, "p": ("i32",)}, "p(X) :- e(X,4294967296).", "XL_TYPE_MISMATCH"),
    ({"e": ("i64", "i64"), "p": ("i64",)}, "p(X) :- e(X,1.5).", "XL_TYPE_MISMATCH"),
    ({"e": ("i64", "i64"), "p": ("i64",)}, "p(X) :- e(X,9223372036854775808).", "XL_TYPE_MISMATCH"),
    ({"e": U2, "p": ("u64",)}, "p(X) :- e(X,18446744073709551616).", "XL_PARSE_ERROR"),
    ({"e": ("i32", "bool"), "p": ("i32",)}, "p(X) :- e(X,2).", "XL_TYPE_MISMATCH"),
    ({"e": ("f64", "f64"), "p": ("f64",)}, "p(X) :- e(X,1).", "XL_TYPE_MISMATCH"),
    ({"e": ("u64", "i32"), "p": ("u64",)}, "p(X) :- e(X,Y), X < Y.", "XL_TYPE_MISMATCH"),
    ({"e": U2, "p": ("u64",)}, "p(X) :- e(X,_), X > -3.", "XL_TYPE_MISMATCH"),
    # arithmetic, sum and logsumexp take i32 and f32 only; count is int32
    ({"e": ("i64", "i64"), "p": ("i64", "i64")}, "p(X,Z) :- e(X,Y), Z is Y + 1.", "XL_UNSUPPORTED"),
    ({"e": ("i32", "u32"), "p": ("i32", "u32")}, "p(X,sum(Y)) :- e(X,Y).", "XL_UNSUPPORTED"),
    ({"e": ("i32", "f64"), "p": ("i32", "f64")}, "p(X,logsumexp(Y)) :- e(X,Y).", "XL_TYPE_MISMATCH"),
    ({"e": U2, "p": ("u64", "i64")}, "p(X,count(Y)) :- e(X,Y).", "XL_TYPE_MISMATCH"),
])
def test_rejected_typed_programs(rels, text, status):
    c = _ctx(rels)
    with pytest.raises(xlh.XlError) as ei:
        c.compile(text)
    assert ei.value.status_name == status, str(ei.value)


@pytest.mark.parametrize("rels,text", [
    ({"e": U2, "p": U2}, "p(X,Y) :- e(X,Y).\np(X,Y) :- p(X,Z), e(Z,Y)."),
    ({"e": ("u32", "u32"), "p": ("u32",)}, "p(X) :- e(X,4294967295), X >= 2147483648."),
    ({"e": ("i64", "f64"), "m": ("i64", "f64")}, "m(X,min(W)) :- e(X,W), W < -0.0."),
    ({"e": ("i64", "f64"), "m": ("i64", "f64")}, "m(X,max(W)) :- e(X,W), W != 2.5."),
    ({"e": U2, "c": ("u64", "i32")}, "c(X,count(Y)) :- e(X,Y), Y != 18446744073709551615."),
    ({"e": ("i32", "bool"), "p": ("i32",), "q": ("i32",)}, "p(X) :- e(X,1).\nq(X) :- e(X,0), not p(X)."),
    ({"e": ("i64", "i64"), "p": ("i64",)}, "p(X) :- e(X,-9223372036854775808)."),
])
def test_accepted_typed_programs(rels, text):
    assert "stratum 0" in _ctx(rels).compile(text).explain()


def test_planning_context_refuses_data():
    c = _ctx({"e": I2})
    import numpy as np
    with pytest.raises(xlh.XlError) as ei:
        c.relations["e"].load([np.zeros(3, np.int32), np.ones(3, np.int32)])
    assert ei.value.status_name == "XL_INVALID_ARGUMENT"


def test_options():
    c = xlh.Context(device=-1)
    c.set_option("hash_min_log2", 12)
    c.set_option("profile", 1)
    c.set_option("pull_ratio", 0)
    c.set_option("dense_tiles", -1)
    c.set_option("frontier_resident", 0)
    c.set_option("index_cache_mb", 64)
    c.set_option("index_cache_mb", 0)
    c.set_option("product_joins", 0)
    c.set_option("batched_rounds", 8)
    for k, v in [("hash_min_log2", 3), ("nope", 1), ("profile", 7), ("pull_ratio", 2000),
                 ("index_mode", -1), ("dense_tiles", -2),
                 ("frontier_resident", 2), ("index_cache_mb", -1),
                 ("product_joins", 3), ("batched_rounds", 65)]:
        with pytest.raises(xlh.XlError):
            c.set_option(k, v)


@pytest.mark.parametrize("text", [
    "s(X,Y,sum(C)) :- w(X,Y,C).\ns(X,Y,sum(C)) :- s(X,Z,C1), w(Z,Y,_), C is C1.",
    "s(X,Y,sum(C1)) :- w(X,Y,C1).\ns(X,Y,sum(C1)) :- s(X,Z,C1), w(Z,Y,K), K > 0.",
])
def test_recursive_path_sums_are_accepted(text):
    _ctx({"w": ("i32", "i32", "i32"), "s": ("i32", "i32", "i32")}).compile(text)


@pytest.mark.parametrize("text", [
    "s(X,Y,min(P)) :- w(X,Y,P).\ns(X,Y,min(P)) :- s(X,Z,P1), w(Z,Y,W), P is P1 - W.",
    "s(X,Y,max(P)) :- w(X,Y,P).\ns(X,Y,max(P)) :- s(X,Z,_), w(Z,Y,P).",
    "s(X,Y,min(P)) :- w(X,Y,P).\ns(X,Y,min(P)) :- s(X,Z,P1), s(Z,Y,P2), P is P1 + P2.",
    "s(X,Y,logsumexp(P)) :- w(X,Y,P).\ns(X,Y,logsumexp(P)) :- s(X,Z,P1), w(Z,Y,W), P is P1 + W.",
    "s(X,Y,logsumexp(P)) :- w(X,Y,P).\ns(X,Y,logsumexp(P)) :- s(X,Z,P1), w(Z,Y,W), W > -2.0, P is P1 - W - 1.0.",
])
def test_recursive_log_domain_products_are_accepted(text):
    _ctx({"w": W3, "s": W3}).compile(text)
