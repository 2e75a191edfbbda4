"""Seeded synthetic inputs for the semi-naive fixpoint engine.

This module only draws random relations and holds the rule texts that are
evaluated over them; it contains none of the evaluation arithmetic, so both
the GPU engine's tests and the CPU oracle's tests can use it without sharing
any code of the method itself.

The paper evaluates its Datalog engine on program-analysis and hub-skewed
graph shapes (Sec. 4.4, Sec. 10) whose datasets are not available here.  The
five workloads below stand in for them: uniform random graphs, a layered DAG,
a bounded-depth forest and an R-MAT power-law graph.  Every generator takes an
explicit seed and uses numpy's PCG64, so the same seed always yields the same
bytes.

Relations are returned as ``{name: (types, [column arrays])}`` where types is
a tuple of "i32" / "f32" strings and the columns are numpy int32 / float32
arrays of equal length.  Every relation is a set (no duplicate rows).
"""
from __future__ import annotations

import hashlib
from collections import deque
from dataclasses import dataclass, field

import numpy as np

TC_RULES = """
path(X,Y) :- edge(X,Y).
path(X,Y) :- path(X,Z), edge(Z,Y).
"""

TC_COUNT_RULES = TC_RULES + """
reach_count(X,count(Y)) :- path(X,Y).
"""

SSSP_RULES = """
dist(S,S,min(D)) :- source(S), D is 0.0.
dist(S,Y,min(D)) :- dist(S,Z,D1), edge(Z,Y,W), D is D1 + W.
"""

LSE_RULES = """
score(S,Y,logsumexp(P)) :- source(S), edge(S,Y,P).
score(S,Y,logsumexp(P)) :- score(S,Z,P1), edge(Z,Y,W), P is P1 + W.
"""

TRIANGLE_RULES = """
tri(X,Y,Z) :- r(X,Y), s(Y,Z), t(X,Z).
"""

SG_RULES = """
sg(X,Y) :- parent(X,P), parent(Y,P), X != Y.
sg(X,Y) :- parent(X,A), sg(A,B), parent(Y,B).
"""


@dataclass
class Workload:
    """One evaluation problem: rule text, input relations and output schema."""

    name: str
    rules: str
    edb: dict
    idb: dict  # name -> types of the derived relations
    params: dict = field(default_factory=dict)

    def digest(self) -> str:
        """SHA-256 over every input column, so runs can prove identical inputs."""
        h = hashlib.sha256()
        for name in sorted(self.edb):
            types, cols = self.edb[name]
            h.update(name.encode())
            for t, c in zip(types, cols):
                h.update(t.encode())
                h.update(np.ascontiguousarray(c).tobytes())
        return h.hexdigest()


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _collect_distinct(draw, target: int, batch: int):
    """Accumulate distinct non-loop (u, v) pairs in first-appearance order."""
    seen_u = np.empty(0, np.int64)
    seen_v = np.empty(0, np.int64)
    while seen_u.size < target:
        u, v = draw(batch)
        keep = u != v
        u = np.concatenate([seen_u, u[keep].astype(np.int64)])
        v = np.concatenate([seen_v, v[keep].astype(np.int64)])
        key = (u << 32) | v
        _, first = np.unique(key, return_index=True)
        first.sort()
        seen_u, seen_v = u[first], v[first]
    return seen_u[:target].astype(np.int32), seen_v[:target].astype(np.int32)


def uniform_graph(n_nodes: int, n_edges: int, seed: int):
    """n_edges distinct directed edges, endpoints uniform on [0, n_nodes), no self-loops."""
    rng = _rng(seed)

    def draw(m):
        return rng.integers(0, n_nodes, m), rng.integers(0, n_nodes, m)

    return _collect_distinct(draw, n_edges, max(1024, n_edges // 2))


def tc_uniform(n_nodes: int = 1000, n_edges: int = 4000, seed: int = 1) -> Workload:
    """Transitive closure over a uniform random graph (the 1k-node / 4k-edge workload)."""
    src, dst = uniform_graph(n_nodes, n_edges, seed)
    return Workload(
        name=f"tc_uniform_n{n_nodes}_e{n_edges}",
        rules=TC_RULES,
        edb={"edge": (("i32", "i32"), [src, dst])},
        idb={"path": ("i32", "i32")},
        params=dict(n_nodes=n_nodes, n_edges=n_edges, seed=seed),
    )


def _weights_1_10(rng, m: int) -> np.ndarray:
    """f32 weights 1 + 9u, u in [0,1) drawn in f64; values that round to 10 are redrawn."""
    w = (1.0 + 9.0 * rng.random(m)).astype(np.float32)
    bad = w >= np.float32(10.0)
    while bad.any():
        w[bad] = (1.0 + 9.0 * rng.random(int(bad.sum()))).astype(np.float32)
        bad = w >= np.float32(10.0)
    return w


def sssp(n_nodes: int = 100_000, n_edges: int = 1_000_000, n_sources: int = 64,
         seed: int = 2) -> Workload:
    """Multi-source shortest paths with a min aggregate over a uniform random graph."""
    rng = _rng(seed)

    def draw(m):
        return rng.integers(0, n_nodes, m), rng.integers(0, n_nodes, m)

    src, dst = _collect_distinct(draw, n_edges, max(1024, n_edges // 2))
    w = _weights_1_10(rng, n_edges)
    sources = np.sort(rng.choice(n_nodes, n_sources, replace=False)).astype(np.int32)
    return Workload(
        name=f"sssp_n{n_nodes}_e{n_edges}_s{n_sources}",
        rules=SSSP_RULES,
        edb={"edge": (("i32", "i32", "f32"), [src, dst, w]),
             "source": (("i32",), [sources])},
        idb={"dist": ("i32", "i32", "f32")},
        params=dict(n_nodes=n_nodes, n_edges=n_edges, n_sources=n_sources, seed=seed),
    )


def layered_dag(n_layers: int = 20, width: int = 5000, out_degree: int = 8,
                n_sources: int = 256, seed: int = 3) -> Workload:
    """Probabilistic reachability (logsumexp) over a layered DAG.

    Node id = layer * width + index.  Every node outside the last layer has
    out_degree distinct targets in the next layer, each with an f32 log
    probability log(0.05 + 0.95 v), v uniform on [0, 1).
    """
    assert out_degree <= width
    rng = _rng(seed)
    n_src_nodes = (n_layers - 1) * width
    tgt = rng.integers(0, width, (n_src_nodes, out_degree))
    while True:
        s = np.sort(tgt, axis=1)
        dup = (s[:, 1:] == s[:, :-1]).any(axis=1)
        if not dup.any():
            break
        tgt[dup] = rng.integers(0, width, (int(dup.sum()), out_degree))
    src_ids = np.repeat(np.arange(n_src_nodes, dtype=np.int64), out_degree)
    layer = src_ids // width
    dst_ids = (layer + 1) * width + tgt.reshape(-1)
    v = rng.random(src_ids.size)
    w = np.log(0.05 + 0.95 * v).astype(np.float32)
    sources = np.sort(rng.choice(width, n_sources, replace=False)).astype(np.int32)
    return Workload(
        name=f"lse_dag_l{n_layers}_w{width}_d{out_degree}_s{n_sources}",
        rules=LSE_RULES,
        edb={"edge": (("i32", "i32", "f32"),
                      [src_ids.astype(np.int32), dst_ids.astype(np.int32), w]),
             "source": (("i32",), [sources])},
        idb={"score": ("i32", "i32", "f32")},
        params=dict(n_layers=n_layers, width=width, out_degree=out_degree,
                    n_sources=n_sources, seed=seed),
    )


def forest(n_nodes: int = 20_000, max_depth: int = 8, mean_children: float = 3.0,
           max_roots: int = 8, seed: int = 4):
    """Bounded-depth random forest; returns (child, parent, depth, root) arrays.

    Starts with U{1..max_roots} roots and grows breadth-first: every node above
    max_depth draws Poisson(mean_children) children, clipped so the total never
    exceeds n_nodes.  If the frontier empties early a further root is added
    (never more than max_roots in total).  Ids follow creation order.
    """
    rng = _rng(seed)
    n_roots = int(rng.integers(1, max_roots + 1))
    depth = [0] * n_roots
    root = list(range(n_roots))
    child, par = [], []
    queue = deque(range(n_roots))
    n = n_roots
    while n < n_nodes:
        if not queue:
            if n_roots >= max_roots:
                break
            depth.append(0)
            root.append(n)
            queue.append(n)
            n += 1
            n_roots += 1
            continue
        v = queue.popleft()
        if depth[v] >= max_depth:
            continue
        k = min(int(rng.poisson(mean_children)), n_nodes - n)
        for _ in range(k):
            child.append(n)
            par.append(v)
            depth.append(depth[v] + 1)
            root.append(root[v])
            queue.append(n)
            n += 1
    return (np.asarray(child, np.int32), np.asarray(par, np.int32),
            np.asarray(depth, np.int32), np.asarray(root, np.int32))


def same_generation(n_nodes: int = 20_000, seed: int = 4) -> Workload:
    """Same-generation (a non-linear three-atom join) over a bounded-depth forest."""
    child, par, depth, root = forest(n_nodes, seed=seed)
    return Workload(
        name=f"sg_forest_n{n_nodes}",
        rules=SG_RULES,
        edb={"parent": (("i32", "i32"), [child, par])},
        idb={"sg": ("i32", "i32")},
        params=dict(n_nodes=n_nodes, seed=seed, depth=depth, root=root),
    )


def rmat_graph(scale: int, n_edges: int, seed: int,
               a: float = 0.57, b: float = 0.19, c: float = 0.19):
    """R-MAT edges: per level pick a quadrant (a: 00, b: 01, c: 10, d: 11).

    No noise and no relabelling; duplicates and self-loops are dropped and
    drawing continues until exactly n_edges distinct edges exist.
    """
    rng = _rng(seed)

    def draw(m):
        r = rng.random((m, scale))
        src_bit = r >= a + b                      # quadrants c, d
        dst_bit = ((r >= a) & (r < a + b)) | (r >= a + b + c)  # quadrants b, d
        weights = (1 << np.arange(scale - 1, -1, -1)).astype(np.int64)
        return src_bit.astype(np.int64) @ weights, dst_bit.astype(np.int64) @ weights

    return _collect_distinct(draw, n_edges, max(1024, n_edges))


def tc_rmat(scale: int = 14, n_edges: int = 1 << 18, seed: int = 5,
            with_count: bool = True) -> Workload:
    """Transitive closure plus per-source reach count over an R-MAT graph."""
    src, dst = rmat_graph(scale, n_edges, seed)
    idb = {"path": ("i32", "i32")}
    if with_count:
        idb["reach_count"] = ("i32", "i32")
    return Workload(
        name=f"tc_rmat_s{scale}_e{n_edges}",
        rules=TC_COUNT_RULES if with_count else TC_RULES,
        edb={"edge": (("i32", "i32"), [src, dst])},
        idb=idb,
        params=dict(scale=scale, n_edges=n_edges, seed=seed),
    )


# The five full-size workloads, in the order they are listed for this engine.
def _distinct_pairs(fixed, parts, rng):
    """Distinct (a, b) pairs: the fixed pairs first, then for each (count,
    draw) of parts, drawn pairs not seen before until count of them are
    added (draw(rng, k) returns k candidate pairs)."""
    seen = set(zip(fixed[0].tolist(), fixed[1].tolist()))
    out_a, out_b = [fixed[0].tolist()], [fixed[1].tolist()]
    for count, draw in parts:
        added = 0
        while added < count:
            a, b = draw(rng, 2 * (count - added) + 16)
            for u, v in zip(a.tolist(), b.tolist()):
                if (u, v) not in seen:
                    seen.add((u, v))
                    out_a[0].append(u)
                    out_b[0].append(v)
                    added += 1
                    if added == count:
                        break
    return np.array(out_a[0], np.int32), np.array(out_b[0], np.int32)


def triangle(rows: int = 1 << 16, core: int = 161, hubs: int = 8, seed: int = 6,
             core_frac: float = 0.4, hub_frac: float = 0.3) -> Workload:
    """Three-way triangle join tri(X,Y,Z) :- r(X,Y), s(Y,Z), t(X,Z) over three
    relations of `rows` distinct pairs each, shaped so that every join
    variable has a small hot domain.

    The paper's fixture (three relations of 65,536 rows, about 4.19 M output
    triples, hot domains that make a binary-join plan's intermediate far
    larger than the result; Sec. 10, WCOJ ablation) is not available; this
    stands in for it.  Values 0..core-1 form a hot core: each relation holds
    min(core_frac * rows, core^2) distinct core x core pairs drawn without
    replacement (all of them at the defaults, which alone close
    161^3 = 4,173,281 triangles).  Values core..core+hubs-1 are hubs:
    hub_frac of r's rows pair a cold X with a hub Y and hub_frac of s's rows
    pair a hub Y with a cold Z, so r joined with s on Y is large while t,
    which holds no hub rows, closes few of those pairs.  The remaining rows
    are uniform over the cold values [core + hubs, rows).
    """
    rng = _rng(seed)
    lo_cold = core + hubs
    n_core = min(int(round(core_frac * rows)), core * core)
    n_hub = int(round(hub_frac * rows))
    if n_core + n_hub > rows or lo_cold >= rows:
        raise ValueError("triangle: core and hub rows exceed the relation size")

    def core_pairs():
        k = rng.choice(core * core, n_core, replace=False)
        return k // core, k % core

    def cold_pairs(g, k):
        return g.integers(lo_cold, rows, k), g.integers(lo_cold, rows, k)

    def cold_hub(g, k):
        return g.integers(lo_cold, rows, k), g.integers(core, lo_cold, k)

    def hub_cold(g, k):
        return g.integers(core, lo_cold, k), g.integers(lo_cold, rows, k)

    r = _distinct_pairs(core_pairs(), [(n_hub, cold_hub), (rows - n_core - n_hub, cold_pairs)], rng)
    s_ = _distinct_pairs(core_pairs(), [(n_hub, hub_cold), (rows - n_core - n_hub, cold_pairs)], rng)
    t = _distinct_pairs(core_pairs(), [(rows - n_core, cold_pairs)], rng)
    i2 = ("i32", "i32")
    return Workload("triangle", TRIANGLE_RULES,
                    {"r": (i2, list(r)), "s": (i2, list(s_)), "t": (i2, list(t))},
                    {"tri": ("i32", "i32", "i32")},
                    {"rows": rows, "core": core, "hubs": hubs, "seed": seed})


# ---------------------------------------------------------------- typed labels
TYPED_KINDS = ("u32", "i64", "u64", "f64")


def typed_labels(kind: str, n: int, extremes: bool = True) -> np.ndarray:
    """n distinct values of a column type in strictly ascending order of that
    type (f64: IEEE totalOrder), spread over the type's range: the extremes,
    values either side of the signed/unsigned boundary, and for f64 both
    zeros (-0.0 before +0.0), subnormals and negatives.  Node i of a graph
    drawn over 0..n-1 becomes label i, so any order-based result over the
    labels is the i32 result relabelled."""
    assert n >= 8
    h = n // 2
    i = np.arange(n, dtype=object)
    if kind == "u32":
        vals = [2 ** 31 - 3 * h + 3 * int(k) for k in i]
        if extremes:
            vals[0], vals[-1] = 0, 2 ** 32 - 1
        return np.array(vals, dtype=np.uint64).astype(np.uint32)
    if kind == "i64":
        vals = [(int(k) - h) * 2 ** 34 + 11 for k in i]
        vals[0], vals[-1] = -2 ** 63, 2 ** 63 - 1
        return np.array(vals, dtype=np.int64)
    if kind == "u64":
        vals = [2 ** 63 - h * 2 ** 20 + int(k) * 2 ** 20 for k in i]
        vals[0], vals[-1] = 0, 2 ** 64 - 1
        return np.array(vals, dtype=np.uint64)
    if kind == "f64":
        neg = [-(h - 1 - k) * 0.75 - 5e-324 for k in range(h - 1)]   # ascending negatives
        pos = [5e-324] + [(k + 1) * 1.25 for k in range(n - h - 2)]
        vals = neg[:-1] + [-5e-324, -0.0, 0.0] + pos
        assert len(vals) == n, len(vals)
        vals[0] = -1.7976931348623157e308
        vals[-1] = 1.7976931348623157e308
        return np.array(vals, dtype=np.float64)
    raise KeyError(kind)


def full_workloads():
    return {
        "tc_uniform": tc_uniform,
        "sssp": sssp,
        "lse_dag": layered_dag,
        "same_generation": same_generation,
        "tc_rmat_count": tc_rmat,
        "triangle": triangle,
    }


# Reduced versions of the same recipes, small enough for an exhaustive
# oracle comparison in seconds while still spanning many GPU tiles.
def small_workloads():
    return {
        "tc_uniform": lambda: tc_uniform(300, 1200, seed=11),
        "sssp": lambda: sssp(3000, 30_000, 16, seed=12),
        "lse_dag": lambda: layered_dag(8, 300, 8, 32, seed=13),
        "same_generation": lambda: same_generation(1500, seed=14),
        "tc_rmat_count": lambda: tc_rmat(10, 1 << 13, seed=15),
        "triangle": lambda: triangle(rows=4096, core=40, hubs=4, seed=16),
    }
