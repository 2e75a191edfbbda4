"""CPU oracle, semi-naive mode: Algorithm 1 (Sec. 4.1) over the naive oracle's
own T_P pieces.

TEST INFRASTRUCTURE ONLY, like datalog.py: nothing in the engine imports it;
the test suite checks it against the naive definition, and the benchmark's
CPU-baseline leg times it on all host cores.

Per stratum (strongly connected component of the IDB dependency graph, in
dependency order):

* seed (iteration 0): every rule of the stratum is applied once to the
  relations as they stand (the stratum's own heads empty); the result is the
  first delta and the first full relation;
* each pass then applies, for every rule and every body atom whose
  predicate is a head of this stratum, the rule with that one atom reading
  the previous pass's delta and every other atom reading the full relations
  as they stood when the pass began (one delta variant per recursive atom);
* the pass's results are merged into the full relations, per head kind
  (the readings of aggregate deltas the engine takes too):
  - set heads: delta = results not already in the relation; relation |= delta;
  - min / max heads: delta = the keys whose folded value is new or strictly
    better than the relation's; the relation takes those values;
  - sum / logsumexp heads: delta = the pass's fold per key (the contributions
    derived from the previous delta); the relation's value becomes the
    relation's value folded with it.  This equals the naive fixpoint when
    every recursive rule carries the recursive atom's value through a
    semiring product: for sum the head's value must be that value itself
    (path sums), for logsumexp that value plus further terms (a log-domain
    product).  A term added to a sum's value would be added once per pass in
    which the key's value changes rather than once; such rules are the ones
    the engine refuses;
* the stratum ends after the first pass whose deltas are all empty; passes
  are counted as the engine counts them (the seed is iteration 0, the final
  empty pass counts).

Sum and logsumexp values are accumulated across passes in float64 and rounded
to float32 once at the end; each pass's delta is rounded to float32 before the
next pass reads it, as a float32 relation column would be.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .datalog import (ConvergenceFailure, OracleResult, _NP, _apply_rules, _bits, _canonical, _empty, _order,
                      _strata, parse)

__all__ = ["evaluate_semi_naive"]

_DELTA = "\x00delta:"  # prefix of the names the delta relations take in a pass's view


def _key_codes(a_keys, b_keys):
    """Codes such that equal codes <=> equal key tuples, for two key lists:
    the key columns' bits packed into one integer when they fit 64 bits,
    else dense ranks of the distinct tuples."""
    na = len(a_keys[0]) if a_keys else 0
    if not a_keys:
        return np.zeros(na, np.int64), np.zeros(len(b_keys[0]) if b_keys else 0, np.int64)
    narrow = all(np.asarray(a).dtype.itemsize <= 4 for a in a_keys) and len(a_keys) <= 2
    if narrow:
        def pack(keys):
            code = np.zeros(len(keys[0]), np.uint64)
            for k in keys:
                v = _bits(np.asarray(k)).astype(np.int64).astype(np.uint64) & np.uint64(0xFFFFFFFF)
                code = (code << np.uint64(32)) | v
            return code
        return pack(a_keys), pack(b_keys)
    cols = [np.concatenate([_bits(np.asarray(a)).astype(np.int64), _bits(np.asarray(b)).astype(np.int64)])
            for a, b in zip(a_keys, b_keys)]
    _, inv = np.unique(np.stack(cols, axis=1), axis=0, return_inverse=True)
    inv = inv.reshape(-1)
    return inv[:na], inv[na:]


def _locate(have, new):
    """For each code of `new`, its index in `have` (distinct codes), or -1."""
    order = np.argsort(have, kind="stable")
    sh = have[order]
    pos = np.searchsorted(sh, new)
    pos_c = np.minimum(pos, max(len(sh) - 1, 0))
    hit = (pos < len(sh)) & (sh[pos_c] == new) if len(sh) else np.zeros(len(new), bool)
    return np.where(hit, order[pos_c] if len(sh) else 0, -1).astype(np.int64)


def _lse2(a, b):
    m = np.maximum(a, b)
    with np.errstate(invalid="ignore"):
        out = m + np.log1p(np.exp(-np.abs(a - b)))
    return np.where(np.isneginf(a), b, np.where(np.isneginf(b), a, out))


class _Head:
    """The full relation of one head of the running stratum."""

    def __init__(self, name, types, agg):
        self.name, self.types, self.agg = name, tuple(types), agg
        self.nkey = len(types) - (1 if agg else 0)
        self.keys = [np.empty(0, _NP[t]) for t in types[: self.nkey]]
        self.vals = np.empty(0, np.float64 if agg in ("sum", "logsumexp") and types[-1] == "f32"
                             else (_NP[types[-1]] if agg else np.int32))

    def rows(self):
        """The relation's rows in no particular order (no duplicates)."""
        if not self.agg:
            return (self.types, list(self.keys))
        vals = self.vals
        if self.agg in ("sum", "logsumexp") and self.types[-1] == "f32":
            vals = vals.astype(np.float32)
        return (self.types, list(self.keys) + [np.asarray(vals, _NP[self.types[-1]])])

    def relation(self):
        if not self.agg:
            return _canonical(self.types, self.keys)
        vals = self.vals
        if self.agg in ("sum", "logsumexp") and self.types[-1] == "f32":
            vals = vals.astype(np.float32)
        return _canonical(self.types, self.keys + [np.asarray(vals, _NP[self.types[-1]])])

    def merge(self, cand):
        """Merge one pass's folded results; returns the delta relation."""
        types, cols = cand
        if len(cols[0]) == 0:
            return _empty(self.types)
        ck = cols[: self.nkey]
        have, new = _key_codes(self.keys, ck)
        idx = _locate(have, new)
        fresh = idx < 0
        if not self.agg:
            self.keys = [np.concatenate([k, c[fresh]]) for k, c in zip(self.keys, ck)]
            return _canonical(self.types, [c[fresh] for c in ck])
        cv = cols[self.nkey]
        if self.agg in ("min", "max"):
            better = np.zeros(len(cv), bool)
            old = self.vals[np.maximum(idx, 0)]
            if self.agg == "min":
                better[~fresh] = _order(cv[~fresh]) < _order(old[~fresh])
            else:
                better[~fresh] = _order(cv[~fresh]) > _order(old[~fresh])
            self.vals[idx[better]] = cv[better]
            self.keys = [np.concatenate([k, c[fresh]]) for k, c in zip(self.keys, ck)]
            self.vals = np.concatenate([self.vals, cv[fresh]])
            take = fresh | better
            return _canonical(self.types, [c[take] for c in ck] + [cv[take]])
        if self.agg in ("sum", "logsumexp"):
            wide = self.vals.dtype
            add = np.asarray(cv, wide)
            if self.agg == "sum" and wide != np.float64:
                cur = self.vals[idx[~fresh]].astype(np.int64) + add[~fresh].astype(np.int64)
                self.vals[idx[~fresh]] = ((cur + 2 ** 31) % 2 ** 32 - 2 ** 31).astype(wide)
            elif self.agg == "sum":
                self.vals[idx[~fresh]] = self.vals[idx[~fresh]] + add[~fresh]
            else:
                self.vals[idx[~fresh]] = _lse2(self.vals[idx[~fresh]], add[~fresh])
            self.keys = [np.concatenate([k, c[fresh]]) for k, c in zip(self.keys, ck)]
            self.vals = np.concatenate([self.vals, add[fresh]])
            return _canonical(self.types, list(ck) + [cv])  # the pass's fold is the delta
        raise ValueError(f"{self.agg} inside a recursive stratum is not supported")

    def seed(self, cand):
        types, cols = cand
        self.keys = [c.copy() for c in cols[: self.nkey]]
        if self.agg:
            self.vals = np.asarray(cols[self.nkey], self.vals.dtype).copy()
        return cand


def _restricted(cand, restrict, head):
    if not restrict or head not in restrict:
        return cand
    col, allowed = restrict[head]
    t, cs = cand
    keep = np.isin(cs[col], np.asarray(allowed))
    return (t, [c[keep] for c in cs])


def evaluate_semi_naive(rules_text: str, edb: dict, idb: dict, max_iterations: int = 10_000,
                        restrict: dict | None = None) -> OracleResult:
    """Semi-naive evaluation to the least fixpoint (same arguments and result
    as datalog.evaluate; `iterations` counts passes as the engine does)."""
    rules = parse(rules_text)
    rels = {k: _canonical(t, c) for k, (t, c) in edb.items()}
    for r in rules:
        if r.head not in idb:
            raise KeyError(f"rule head {r.head} has no declared schema")
    iterations, sizes = {}, {h: [] for h in idb}
    for comp in _strata(rules, idb):
        mine = [r for r in rules if r.head in comp]
        heads = {}
        for h in comp:
            aggs = {r.agg[0] for r in mine if r.head == h and r.agg}
            heads[h] = _Head(h, idb[h], aggs.pop() if aggs else None)
        # seed: every rule over the relations as they stand (the heads empty)
        view = dict(rels)
        view.update({h: _empty(idb[h]) for h in comp})
        delta = {}
        for h in comp:
            hr = [r for r in mine if r.head == h]
            cand = _apply_rules(h, tuple(idb[h]), hr, view) if hr else _empty(idb[h])
            delta[h] = heads[h].seed(_restricted(cand, restrict, h))
            sizes[h].append(len(delta[h][1][0]))
        variants = []
        for r in mine:
            for i, (pred, terms) in enumerate(r.atoms):
                if pred in comp:
                    atoms = list(r.atoms)
                    atoms[i] = (_DELTA + pred, terms)
                    variants.append(dataclasses.replace(r, atoms=atoms))
        passes = 0
        while variants and any(len(d[1][0]) for d in delta.values()):
            if passes >= max_iterations:
                raise ConvergenceFailure(f"no fixpoint for {comp} within {max_iterations} passes")
            passes += 1
            view = dict(rels)
            for h in comp:
                view[h] = heads[h].rows()
                view[_DELTA + h] = delta[h]
            nxt = {}
            for h in comp:
                hv = [v for v in variants if v.head == h]
                cand = _apply_rules(h, tuple(idb[h]), hv, view) if hv else _empty(idb[h])
                nxt[h] = heads[h].merge(_restricted(cand, restrict, h))
                sizes[h].append(len(heads[h].keys[0]) if heads[h].keys else 0)
            delta = nxt
        iterations[tuple(comp)] = passes
        for h in comp:
            rels[h] = heads[h].relation()
    return OracleResult({h: rels[h] for h in idb}, iterations, sizes)
