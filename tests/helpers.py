"""Shared helpers for the GPU parity tests: run a workload through the engine
(via the C ABI binding) and compare with the CPU oracle."""
from __future__ import annotations

import numpy as np

LSE_TOL = 1e-5   # |gpu - ref| <= LSE_TOL * max(1, |ref|)
MIN_TOL = 1e-6   # relative; the f32 min fixpoint is expected to be bit-exact


def engine_run(wl, workspace_bytes=1 << 30, options=None, max_iterations=10_000, edb=None,
               ctx=None):
    """Evaluate a workload on cuda:0; returns (relations, stats, ctx)."""
    from paper_2609_27203_amd import xlh
    if ctx is None:
        ctx = xlh.Context(device=0, workspace_bytes=workspace_bytes)
        for k, v in (options or {}).items():
            ctx.set_option(k, v)
        for name, (types, _) in wl.edb.items():
            ctx.relation(name, types)
        for name, types in wl.idb.items():
            ctx.relation(name, types)
    for name, (_, cols) in (edb or wl.edb).items():
        ctx.relations[name].load(cols)
    for name in wl.idb:
        ctx.relations[name].clear()
    prog = ctx.compile(wl.rules)
    stats = prog.run(max_iterations)
    rels = {name: ctx.relations[name].read() for name in wl.idb}
    return rels, stats, ctx


def value_tolerance(rules: str, name: str):
    """(tolerance, floor) for the f32 value column of relation `name`.

    logsumexp: |gpu - ref| <= 1e-5 * max(1, |ref|); min/sum: 1e-6 relative.
    """
    for line in rules.splitlines():
        if line.strip().startswith(name + "(") and "logsumexp(" in line.split(":-")[0]:
            return LSE_TOL, 1.0
    return MIN_TOL, 0.0


def assert_same_relation(name, types, got, ref, where="", tol=(MIN_TOL, 0.0)):
    """Keys bit-exact; f32 value column within the aggregate's tolerance."""
    n_ref = len(ref[0])
    assert len(got[0]) == n_ref, f"{name}{where}: {len(got[0])} rows, oracle {n_ref}"
    for j, t in enumerate(types):
        g, r = got[j], ref[j]
        if t == "f64":  # values come from the data only: identical bits
            g, r = np.asarray(g).view(np.int64), np.asarray(r).view(np.int64)
        if t != "f32":
            bad = np.flatnonzero(g != r)
            assert bad.size == 0, f"{name}{where} column {j}: first mismatch at row {bad[0]}: {g[bad[0]]} vs {r[bad[0]]}"
        else:
            rel, floor = tol
            scale = np.maximum(floor, np.abs(r.astype(np.float64)))
            err = np.abs(g.astype(np.float64) - r.astype(np.float64))
            both_inf = np.isinf(g) & np.isinf(r) & (np.sign(g) == np.sign(r))
            err[both_inf] = 0.0
            worst = int(np.argmax(err - rel * scale)) if len(err) else 0
            assert np.all(err <= rel * scale), \
                f"{name}{where} column {j}: row {worst} gpu {g[worst]!r} oracle {r[worst]!r}"


def select_rows(cols, col, values):
    keep = np.isin(cols[col], np.asarray(values))
    return [c[keep] for c in cols]
