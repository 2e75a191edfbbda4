"""The allocation-free context (xl_context_create_static) against the
workspace context (xl_context_create): same programs, same inputs, same
results, through the C ABI.  The static workspace keeps the previous call's
contents, so every case runs a larger input first and a smaller one after it
(stale tables, bitmaps and counters from the first must not leak into the
second)."""
import numpy as np
import pytest

from helpers import assert_same_relation, value_tolerance
from paper_2609_27203_amd import workloads as W
from paper_2609_27203_amd import xlh

pytestmark = pytest.mark.gpu


def _run(wl, ctx):
    for name, (types, cols) in wl.edb.items():
        rel = ctx.relations.get(name) or ctx.relation(name, types)
        rel.load(cols)
    for name, types in wl.idb.items():
        rel = ctx.relations.get(name) or ctx.relation(name, types)
        rel.clear()
    stats = ctx.compile(wl.rules).run()
    return {n: ctx.relations[n].read() for n in wl.idb}, stats


def _same(wl, got, ref):
    for name, types in wl.idb.items():
        tol = value_tolerance(wl.rules, name)
        assert_same_relation(name, types, got[name], ref[name], " (static vs workspace context)",
                             tol=tol if tol[1] else (0.0, 0.0))
        assert len(got[name][0]) > 0, name


PAIRS = {
    "closure_count": (lambda: W.tc_rmat(10, 1 << 13, seed=15), lambda: W.tc_rmat(9, 3000, seed=3)),
    "min": (lambda: W.sssp(3000, 30_000, 16, seed=12), lambda: W.sssp(1000, 6000, 4, seed=9)),
    "logsumexp": (lambda: W.layered_dag(8, 300, 8, 32, seed=13), lambda: W.layered_dag(5, 100, 4, 8, seed=2)),
    "same_generation": (lambda: W.same_generation(1500, seed=14), lambda: W.same_generation(400, seed=5)),
}


@pytest.mark.parametrize("name", list(PAIRS))
def test_static_context_matches_workspace_context_twice(name):
    """Two static contexts in a row on device 0 (the second on a smaller
    input), each against the workspace context's result; the second static
    context also runs its input twice."""
    for k, make in enumerate(PAIRS[name]):
        wl = make()
        print(f"case: no-alloc {name} call {k + 1} {wl.name}", flush=True)
        ref, ref_stats = _run(wl, xlh.Context(device=0, workspace_bytes=256 << 20))
        ctx = xlh.Context(device=0, static=True)
        try:
            got, stats = _run(wl, ctx)
            _same(wl, got, ref)
            assert stats["derived_tuples"] == ref_stats["derived_tuples"]
            assert stats["iterations"] == ref_stats["iterations"]
            if k == 1:
                again, _ = _run(wl, ctx)
                _same(wl, again, ref)
        finally:
            ctx.close()


def test_one_static_context_per_device():
    print("case: no-alloc second static context refused", flush=True)
    first = xlh.Context(device=0, static=True)
    try:
        with pytest.raises(xlh.XlError) as ei:
            xlh.Context(device=0, static=True)
        assert ei.value.status_name == "XL_RESOURCE_EXHAUSTED"
    finally:
        first.close()
    xlh.Context(device=0, static=True).close()   # free again once the first is gone


def test_static_workspace_limit_is_a_clear_error():
    """A load larger than the 64 MiB static workspace is refused with
    XL_RESOURCE_EXHAUSTED before any device work; the context stays usable."""
    print("case: no-alloc workspace limit", flush=True)
    ctx = xlh.Context(device=0, static=True)
    try:
        n = 20_000_000   # each int32 column alone is 80 MB
        big = ctx.relation("big", ("i32", "i32"))
        with pytest.raises(xlh.XlError) as ei:
            big.load([np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32)])
        assert ei.value.status_name == "XL_RESOURCE_EXHAUSTED"
        assert "workspace exhausted" in str(ei.value)
        wl = W.tc_rmat(9, 3000, seed=3)
        got, _ = _run(wl, ctx)
        ref, _ = _run(wl, xlh.Context(device=0, workspace_bytes=256 << 20))
        _same(wl, got, ref)
    finally:
        ctx.close()
