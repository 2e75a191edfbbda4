"""Full-size certificates for the five workloads, computed on the CPU from
textbook routines (no oracle, no engine): they decide every row of a
full-size result, where the naive oracle is too slow to run per test.

* closure (transitive closure, R-MAT and uniform): breadth-first search from
  every node at once, with the frontier of all sources held as one bit per
  (node, source); level k holds the pairs first joined by a walk of k edges,
  so the level sizes are the per-pass delta sizes of linear semi-naive
  evaluation (Sec. 4.1, Algorithm 1).
* min (shortest paths): the binary32 Bellman equations.  d(s, s) = 0, and
  for every other y, d(s, y) = min over in-edges (z, y, w) of fl32(d(s, z) +
  w) (+inf when there is none).  With weights >= 1 and distances far below
  2^24, fl32(x + w) > x, so the equations have one solution, and it is the
  fixpoint of the min rule (and binary32 Dijkstra).
* logsumexp over a DAG: the layer-by-layer forward pass in probability space
  in float64 (path mass = product of exp(weight)); the score of (s, y) is the
  log of the total mass of the paths of >= 1 edge from s to y.
* same generation over a forest: (x, y) with x != y, both with a parent, in
  the same tree at the same depth.
"""
from __future__ import annotations

import hashlib

import numpy as np
import scipy.sparse as sp


def row_digest(cols) -> str:
    """SHA-256 over rows in the given order, each row as its columns' 4-byte
    little-endian images one after another (int32 as is, float32 by bits)."""
    h = hashlib.sha256()
    n = len(cols[0])
    step = 1 << 24
    for lo in range(0, n, step):
        part = [np.ascontiguousarray(c[lo:lo + step]).view(np.uint32) for c in cols]
        h.update(np.stack(part, axis=1).astype("<u4").tobytes())
    return h.hexdigest()


def _in_edge_segments(n, src, dst):
    order = np.argsort(dst, kind="stable")
    starts = np.searchsorted(dst[order], np.arange(n + 1))
    return order, starts


def closure_bits(n, src, dst, block=1024):
    """Breadth-first search from every node at once.

    Returns (reached, levels): reached is uint64[n, ceil(n / 64)] with bit x of
    row y set iff a walk of >= 1 edge leads from x to y; levels[k - 1] is the
    number of pairs whose shortest such walk has k edges, and the list ends
    with the 0 of the first empty level."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    words = (n + 63) // 64
    order, starts = _in_edge_segments(n, src, dst)
    zs = src[order]
    one = np.uint64(1)
    delta = np.zeros((n, words), np.uint64)
    np.bitwise_or.at(delta, (dst, src >> 6), np.left_shift(one, (src & 63).astype(np.uint64)))
    reached = delta.copy()
    levels = [int(np.bitwise_count(delta).sum())]
    while levels[-1]:
        nxt = np.zeros_like(delta)
        for lo in range(0, n, block):
            hi = min(n, lo + block)
            e0, e1 = starts[lo], starts[hi]
            if e0 == e1:
                continue
            # one zero row after the block's edges, so that every segment start
            # (an empty segment's included) is a valid index
            g = np.concatenate([delta[zs[e0:e1]], np.zeros((1, words), np.uint64)])
            red = np.bitwise_or.reduceat(g, starts[lo:hi] - e0, axis=0)
            red[starts[lo + 1:hi + 1] == starts[lo:hi]] = 0   # targets without in-edges
            nxt[lo:hi] = red
        delta = nxt & ~reached
        reached |= delta
        levels.append(int(np.bitwise_count(delta).sum()))
    return reached, levels


def reached_matrix(reached, n):
    """Boolean matrix m[x, y] = (y reachable from x) from closure_bits' rows."""
    bits = np.unpackbits(reached.view(np.uint8), axis=1, bitorder="little")[:, :n]   # [y, x]
    return bits.T.astype(bool)


def check_closure_rows(m, x, y):
    """The rows (x, y) are strictly ascending and are exactly the true cells of m."""
    n = m.shape[0]
    key = x.astype(np.int64) * n + y.astype(np.int64)
    if len(key) > 1 and not np.all(key[1:] > key[:-1]):
        raise AssertionError("rows are not strictly ascending")
    if not m.ravel()[key].all():
        bad = int(np.flatnonzero(~m.ravel()[key])[0])
        raise AssertionError(f"row ({x[bad]}, {y[bad]}) is not in the closure")
    total = int(m.sum())
    if total != len(key):
        raise AssertionError(f"{len(key)} rows, closure has {total}")


def bellman_check(n, src, dst, w, sources, s_col, y_col, d_col, chunk=8):
    """Raise unless the rows (s, y, d) solve the binary32 Bellman equations for
    every source (rows absent = +inf)."""
    sources = np.asarray(sources)
    rank = np.searchsorted(sources, s_col)
    if not np.array_equal(sources[np.minimum(rank, len(sources) - 1)], s_col):
        raise AssertionError("a row's first column is not a source")
    key = rank.astype(np.int64) * n + y_col
    if len(key) > 1 and not np.all(key[1:] > key[:-1]):
        raise AssertionError("rows are not strictly ascending")
    D = np.full((len(sources), n), np.inf, np.float32)
    D[rank, y_col] = d_col
    finite = D[np.isfinite(D)]
    if finite.size and not (finite.min() >= 0 and finite.max() < 2.0 ** 20):
        raise AssertionError("distances outside the range where the equations have one solution")
    w = np.asarray(w, np.float32)
    if w.size and w.min() < 1:
        raise AssertionError("weights below 1")
    order, starts = _in_edge_segments(n, np.asarray(src, np.int64), np.asarray(dst, np.int64))
    zs, ws = np.asarray(src)[order], w[order]
    no_in = starts[1:] == starts[:-1]
    for c0 in range(0, len(sources), chunk):
        c1 = min(len(sources), c0 + chunk)
        cand = D[c0:c1][:, zs] + ws                       # one binary32 add per edge
        # one +inf column after the edges: every segment start is a valid index
        cand = np.concatenate([cand, np.full((c1 - c0, 1), np.inf, np.float32)], axis=1)
        best = np.minimum.reduceat(cand, starts[:-1], axis=1)
        best[:, no_in] = np.inf
        for i in range(c0, c1):
            s = int(sources[i])
            best[i - c0, s] = min(np.float32(0.0), best[i - c0, s])
        sub = D[c0:c1]
        if not np.array_equal(sub.view(np.int32), best.astype(np.float32).view(np.int32)):
            r, y = np.argwhere(sub.view(np.int32) != best.astype(np.float32).view(np.int32))[0]
            raise AssertionError(f"source {sources[c0 + r]} node {y}: row {sub[r, y]!r}, equations {best[r, y]!r}")


def forward_scores(n, src, dst, w, sources, n_layers):
    """float64 total path mass of the paths of >= 1 edge from each source:
    array [n, len(sources)]; score = log(mass), absent where mass is 0."""
    A = sp.csr_matrix((np.exp(np.asarray(w, np.float64)), (src, dst)), shape=(n, n))
    AT = A.T.tocsr()
    mass = np.zeros((n, len(sources)))
    mass[np.asarray(sources), np.arange(len(sources))] = 1.0
    total = np.zeros_like(mass)
    for _ in range(n_layers - 1):
        mass = AT @ mass
        total += mass
    return total


def check_scores(total, sources, s_col, y_col, p_col, tol=1e-5):
    """Every row within tol * max(1, |ref|) of log(total mass); the rows are
    exactly the (source, node) pairs with positive mass."""
    rank = np.searchsorted(sources, s_col)
    if not np.array_equal(np.asarray(sources)[np.minimum(rank, len(sources) - 1)], s_col):
        raise AssertionError("a row's first column is not a source")
    mass = total[y_col, rank]
    if not np.all(mass > 0):
        raise AssertionError("a row for a pair without paths")
    if len(s_col) != int(np.count_nonzero(total)):
        raise AssertionError(f"{len(s_col)} rows, {int(np.count_nonzero(total))} pairs with paths")
    ref = np.log(mass)
    err = np.abs(p_col.astype(np.float64) - ref)
    lim = tol * np.maximum(1.0, np.abs(ref))
    if not np.all(err <= lim):
        i = int(np.argmax(err - lim))
        raise AssertionError(f"({s_col[i]}, {y_col[i]}): {p_col[i]!r} vs {ref[i]!r}")
    return float(np.max(err / np.maximum(1.0, np.abs(ref)))) if len(err) else 0.0


def same_generation_keys(child, depth, root, n):
    """Sorted x * n + y of every (x, y), x != y, both with a parent, same tree, same depth."""
    has_parent = np.zeros(len(depth), bool)
    has_parent[child] = True
    nodes = np.flatnonzero(has_parent)
    group = root[nodes].astype(np.int64) * 64 + depth[nodes]
    order = np.lexsort((nodes, group))
    nodes, group = nodes[order], group[order]
    bounds = np.flatnonzero(np.diff(group)) + 1
    keys = []
    for g in np.split(nodes, bounds):
        xs = np.repeat(g, len(g)).astype(np.int64)
        ys = np.tile(g, len(g)).astype(np.int64)
        keep = xs != ys
        keys.append(xs[keep] * n + ys[keep])
    return np.sort(np.concatenate(keys)) if keys else np.zeros(0, np.int64)
