"""Pins of the oracle's scalar types beyond i32 / f32 (the paper's type
system, Sec. 3.2): u32, i64, u64, bool and f64 with IEEE 754 totalOrder.

Two kinds of pin, neither of which re-derives the oracle's own formulas:
  * relabelling: every result of an order-based program (closure, count, min,
    max, comparisons with a constant) over node labels of a wider type must
    be the already-pinned int32 result with node i replaced by the i-th label,
    when the labels ascend in the type's order;
  * hand-written expectations from the types' definitions: the ascending
    order of boundary values, min/max of -0.0 and +0.0, which rows a
    comparison or an equality with a constant keeps.
"""
import math
import struct

import numpy as np
import pytest

import oracle.datalog as D
from oracle import evaluate
from paper_2609_27203_amd import workloads as W

PROGRAM = """
path(X,Y) :- e(X,Y).
path(X,Y) :- path(X,Z), e(Z,Y).
reach(X,count(Y)) :- path(X,Y).
low(X,min(Y)) :- path(X,Y).
high(X,max(Y)) :- path(X,Y).
above(X,Y) :- path(X,Y), Y > {c}.
notself(X) :- e(X,_), not path(X,X).
"""


def _literal(v, kind):
    return repr(float(v)) if kind == "f64" else str(int(v))


def _graph(n=40, m=90, seed=11):
    src, dst = W.uniform_graph(n, m, seed)
    return np.asarray(src, np.int64), np.asarray(dst, np.int64)


def _run(kind, n, src, dst, c_index):
    lab = W.typed_labels(kind, n) if kind != "i32" else np.arange(n, dtype=np.int32)
    t = (kind, kind)
    idb = {"path": t, "reach": (kind, "i32"), "low": t, "high": t, "above": t, "notself": (kind,)}
    text = PROGRAM.format(c=_literal(lab[c_index], kind))
    return evaluate(text, {"e": (t, [lab[src], lab[dst]])}, idb).relations, lab


def _relabel(rel, lab, kinds):
    types, cols = rel
    return [lab[c.astype(np.int64)] if k == "node" else c for c, k in zip(cols, kinds)]


@pytest.mark.parametrize("kind", W.TYPED_KINDS)
def test_labels_ascend_in_the_type_order(kind):
    lab = W.typed_labels(kind, 40)
    if kind == "f64":  # ascending by value, and -0.0 (sign bit set) right before +0.0
        v = [float(x) for x in lab]
        z = [k for k, x in enumerate(v) if x == 0.0]
        assert len(z) == 2 and math.copysign(1, v[z[0]]) < 0 < math.copysign(1, v[z[1]]) and z[1] == z[0] + 1
        assert all(a < b for a, b in zip(v[:z[0]], v[1:z[0] + 1])) and all(a < b for a, b in zip(v[z[1]:], v[z[1] + 1:]))
    else:
        v = [int(x) for x in lab]
        assert all(a < b for a, b in zip(v, v[1:]))


@pytest.mark.parametrize("kind", W.TYPED_KINDS)
def test_relabelled_program_equals_int32_program(kind):
    n = 40
    src, dst = _graph(n)
    c_index = 21  # the label right after the f64 zeros / the u32 sign boundary
    base, _ = _run("i32", n, src, dst, c_index)
    wide, lab = _run(kind, n, src, dst, c_index)
    expect = {
        "path": ("node", "node"), "reach": ("node", "count"), "low": ("node", "node"),
        "high": ("node", "node"), "above": ("node", "node"), "notself": ("node",),
    }
    for name, kinds in expect.items():
        want = _relabel(base[name], lab, kinds)
        got = wide[name][1]
        assert len(got[0]) == len(want[0]) > 0 or name == "notself", name
        for g, w in zip(got, want):
            if g.dtype == np.float64:  # identity, so -0.0 and +0.0 stay apart
                assert np.array_equal(g.view(np.int64), np.asarray(w, np.float64).view(np.int64)), name
            else:
                assert np.array_equal(g, w), name


def _sel(types, values, text, out_types=None):
    edb = {"r": (types, [np.array([1] * len(values), np.int32), np.array(values, dtype=D._NP[types[1]])])}
    res = evaluate(text, edb, {"q": out_types or types})
    return [c.tolist() for c in res.relations["q"][1]]


def _bits(x):
    return struct.unpack("<q", struct.pack("<d", x))[0]


F64_ASCENDING = [-1e300, -1.0, -5e-324, -0.0, 0.0, 5e-324, 1.0, 1e300]


def test_f64_total_order_sorts_rows():
    shuffled = [F64_ASCENDING[k] for k in (5, 0, 3, 7, 1, 4, 6, 2)]
    _, vals = _sel(("i32", "f64"), shuffled, "q(X,V) :- r(X,V).")
    assert [_bits(v) for v in vals] == [_bits(v) for v in F64_ASCENDING]


def test_f64_zeros_are_two_values():
    # min picks -0.0 and max +0.0; a comparison with 0.0 follows totalOrder;
    # an equality or a join with +0.0 does not meet -0.0
    _, lo = _sel(("i32", "f64"), [0.0, -0.0], "q(X,min(V)) :- r(X,V).")
    _, hi = _sel(("i32", "f64"), [-0.0, 0.0], "q(X,max(V)) :- r(X,V).")
    assert [_bits(v) for v in lo] == [_bits(-0.0)] and [_bits(v) for v in hi] == [_bits(0.0)]
    _, below = _sel(("i32", "f64"), F64_ASCENDING, "q(X,V) :- r(X,V), V < 0.0.")
    assert [_bits(v) for v in below] == [_bits(v) for v in F64_ASCENDING[:4]]
    _, eq = _sel(("i32", "f64"), F64_ASCENDING, "q(X,V) :- r(X,V), V == 0.0.")
    assert [_bits(v) for v in eq] == [_bits(0.0)]
    _, const = _sel(("i32", "f64"), F64_ASCENDING, "q(X,V) :- r(X,-0.0), r(X,V), V <= -0.0.")
    assert [_bits(v) for v in const] == [_bits(v) for v in F64_ASCENDING[:4]]
    edb = {"a": (("f64",), [np.array([-0.0])]), "b": (("f64",), [np.array([0.0])])}
    res = evaluate("q(V) :- a(V), b(V).", edb, {"q": ("f64",)})
    assert len(res.relations["q"][1][0]) == 0


@pytest.mark.parametrize("ty,ascending,text,kept", [
    ("u32", [0, 1, 2 ** 31 - 1, 2 ** 31, 2 ** 32 - 1], "q(X,V) :- r(X,V), V > 2147483647.", [2 ** 31, 2 ** 32 - 1]),
    ("i64", [-2 ** 63, -2 ** 32, -1, 0, 2 ** 32, 2 ** 63 - 1], "q(X,V) :- r(X,V), V < 0.", [-2 ** 63, -2 ** 32, -1]),
    ("u64", [0, 2 ** 63 - 1, 2 ** 63, 2 ** 64 - 1], "q(X,V) :- r(X,V), V >= 9223372036854775808.",
     [2 ** 63, 2 ** 64 - 1]),
    ("bool", [False, True], "q(X,V) :- r(X,V), V == 1.", [True]),
])
def test_integer_types_order_and_compare(ty, ascending, text, kept):
    shuffled = ascending[::-1]
    assert _sel(("i32", ty), shuffled, "q(X,V) :- r(X,V).")[1] == ascending
    assert _sel(("i32", ty), shuffled, text)[1] == kept
    assert _sel(("i32", ty), shuffled, "q(X,min(V)) :- r(X,V).")[1] == [ascending[0]]
    assert _sel(("i32", ty), shuffled, "q(X,max(V)) :- r(X,V).")[1] == [ascending[-1]]


@pytest.mark.parametrize("types,text", [
    (("i32", "i64"), "q(X,W) :- r(X,V), W is V + 1."),
    (("i32", "u64"), "q(X,sum(V)) :- r(X,V)."),
    (("i32", "u32"), "q(X,V) :- r(X,V), V > -1."),
    (("i32", "i32"), "q(X,V) :- r(X,V), V > 4294967296."),
    (("i32", "f64"), "q(X,V) :- r(X,V), V > 1."),
    (("i32", "bool"), "q(X,V) :- r(X,2)."),
])
def test_rejected_typed_forms(types, text):
    with pytest.raises(TypeError):
        _sel(types, [1], text)


def test_planted_mistake_f64_by_value_is_caught(monkeypatch):
    """An oracle that ordered f64 by IEEE value (-0.0 == +0.0) fails the pins."""
    monkeypatch.setattr(D, "_order", lambda c: np.asarray(c))
    with pytest.raises(AssertionError):
        test_f64_zeros_are_two_values()
