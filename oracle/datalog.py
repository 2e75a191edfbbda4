"""CPU oracle: plain naive bottom-up evaluation of the rule subset.

TEST INFRASTRUCTURE ONLY.  Nothing in the engine imports this module; only the
test suite, the smoke check and the benchmark's CPU-baseline leg call it.  It
shares no code with the GPU engine (its parser, joins and folds are written
here from the definitions below), and it is deliberately slow and direct.

What it computes (the plain definition the semi-naive method reaches):

* Relations are sets of typed tuples (Sec. 3.1-3.2 of the paper).  Column
  types are the paper's scalar types other than symbol (Sec. 3.2, type
  system): "i32", "u32", "i64", "u64" (integers of those widths), "bool"
  (false < true), "f32" and "f64" (IEEE-754 binary32 / binary64).  Values of
  every type but f32 are equal when identical and ordered by the type's
  order; for f64 that order is IEEE 754 totalOrder, so -0.0 < +0.0 and the two
  are different values.  f32 keeps IEEE comparison (-0.0 == +0.0).  A
  constant must be a value of the column type it meets (an integer literal in
  the column's range, a decimal literal for a float column).  ``is``
  arithmetic, sum and logsumexp take i32 and f32 values only.
* The immediate-consequence operator T_P(I) enumerates every derivation of a
  rule -- one fact per body atom, all agreeing on shared variables, all
  comparison filters true -- against the input relations plus I, computes the
  ``is`` arithmetic, and emits the head.  A set head keeps the distinct emitted
  tuples.  An aggregate head (Sec. 3.5: count, sum, min, max, logsumexp in the
  last head position) groups the derivations by the other head columns and
  folds the aggregated variable over all derivations of the group.
* Naive evaluation: I_0 = empty, I_{k+1} = T_P(I_k), stop at the first k with
  I_{k+1} identical to I_k (bitwise, float values included).  Strata (strongly
  connected components of the predicate dependency graph) run in dependency
  order (Sec. 2.4 and Sec. 4.1).  For set heads the result is the least
  fixpoint that Algorithm 1 (semi-naive evaluation) also reaches.
* Precision: ``is`` arithmetic keeps the operands' scalar type (Sec. 3.2), so
  an expression is evaluated left to right and every add or subtract of f32
  values is one binary32 operation (computed in float64 and rounded once to
  float32, which equals the binary32 operation exactly because binary64 has
  more than twice the precision plus two bits); i32 arithmetic wraps modulo
  2^32.  Aggregate folds over f32 values (sum) are taken in float64 and
  rounded once to float32: the exact sum, correctly rounded.  logsumexp uses
  the max-shifted form m + log(sum(exp(x - m))) in float64; a group whose
  values are all -inf folds to -inf.

* Stratified negation (Sec. 3, completeness over finite domains: explicit
  stratified negation-as-failure; Sec. 2, program to GPU plan: negative
  dependency edges in the SCC analysis).  A body literal ``not q(t1, .., tk)``
  holds for a derivation when no row of q agrees with it on every column
  given by a variable or a constant (``_`` columns are unconstrained).  Every
  variable of a negated literal must occur in a positive atom or an ``is``
  of the same rule, and q must be complete before the rule runs: a negative
  dependency inside one strongly connected component is rejected.

Readings where the paper is silent are listed with the engine's design notes;
the ones that change results here are: aggregates fold over derivations (so
count(Y) with body path(X,Y) counts distinct Y per X), groups without
derivations produce no row, and ``is`` / comparisons are applied after all
body atoms have been joined.
"""
from __future__ import annotations

import re
from dataclasses import dataclass, field

import numpy as np

__all__ = ["parse", "evaluate", "ConvergenceFailure", "OracleResult"]


class ConvergenceFailure(RuntimeError):
    """Raised when the iteration cap is reached before the fixpoint."""


# --------------------------------------------------------------------------
# Parsing.  Grammar (the paper's surface syntax, restricted):
#   rule    := atom ':-' literal (',' literal)* '.'
#   atom    := name '(' term (',' term)* ')'
#   head    := name '(' term (',' term)* [',' agg '(' Var ')'] ')'
#   literal := atom | Var 'is' term (('+'|'-') term)* | term cmp term
#   term    := Var | '_' | integer | float
# --------------------------------------------------------------------------
_TOKEN = re.compile(r"""
    (?P<ws>\s+|//[^\n]*)
  | (?P<num>\d+\.\d+(?:[eE][-+]?\d+)?|\d+[eE][-+]?\d+|\d+)
  | (?P<name>[A-Za-z_][A-Za-z0-9_]*)
  | (?P<op>:-|!=|==|<=|>=|<|>|[(),.+-])
""", re.VERBOSE)

AGGREGATES = ("count", "sum", "min", "max", "logsumexp")
CMP_OPS = ("!=", "==", "<", "<=", ">", ">=")


@dataclass
class Rule:
    head: str
    head_terms: list          # ('var', name) entries
    agg: tuple | None         # (op, var) or None
    atoms: list = field(default_factory=list)    # (pred, [terms])
    assigns: list = field(default_factory=list)  # (var, [(sign, term)])
    filters: list = field(default_factory=list)  # (op, term, term)
    negs: list = field(default_factory=list)     # (pred, [terms]) of 'not' literals


def _tokens(text):
    pos = 0
    out = []
    while pos < len(text):
        m = _TOKEN.match(text, pos)
        if not m:
            raise SyntaxError(f"unexpected character at {pos}: {text[pos:pos + 10]!r}")
        pos = m.end()
        if m.lastgroup != "ws":
            out.append((m.lastgroup, m.group()))
    return out


def _term(tok):
    kind, s = tok
    if kind == "num":
        return ("float", float(s)) if any(c in s for c in ".eE") else ("int", int(s))
    if kind == "name":
        if s == "_":
            return ("anon",)
        if s[0].isupper() or s[0] == "_":
            return ("var", s)
    raise SyntaxError(f"expected a term, got {s!r}")


def parse(text: str) -> list:
    toks = _tokens(text)
    i = 0
    rules = []

    def expect(s):
        nonlocal i
        if i >= len(toks) or toks[i][1] != s:
            got = toks[i][1] if i < len(toks) else "end of input"
            raise SyntaxError(f"expected {s!r}, got {got!r}")
        i += 1

    def term():
        nonlocal i
        neg = toks[i][1] == "-" and i + 1 < len(toks) and toks[i + 1][0] == "num"
        if neg:
            i += 1
        t = _term(toks[i])
        i += 1
        return (t[0], -t[1]) if neg else t

    def atom_args():
        nonlocal i
        expect("(")
        args = []
        while True:
            if toks[i][1] in AGGREGATES and i + 1 < len(toks) and toks[i + 1][1] == "(":
                op = toks[i][1]
                i += 2
                var = _term(toks[i])
                i += 1
                expect(")")
                args.append(("agg", op, var))
            else:
                args.append(term())
            if toks[i][1] == ")":
                i += 1
                return args
            expect(",")

    while i < len(toks):
        name = toks[i][1]
        i += 1
        args = atom_args()
        aggs = [a for a in args if a[0] == "agg"]
        if aggs and args[-1][0] != "agg" or len(aggs) > 1:
            raise SyntaxError("an aggregate may only appear once, in the last head position")
        agg = (aggs[0][1], aggs[0][2][1]) if aggs else None
        rule = Rule(head=name, head_terms=args[:-1] if agg else args, agg=agg)
        expect(":-")
        while True:
            t0 = toks[i]
            if t0 == ("name", "not") and toks[i + 1][0] == "name" and toks[i + 2][1] == "(":
                pred = toks[i + 1][1]
                i += 2
                rule.negs.append((pred, atom_args()))
            elif t0[0] == "name" and not (t0[1][0].isupper() or t0[1][0] == "_") \
                    and toks[i + 1][1] == "(":
                i += 1
                rule.atoms.append((t0[1], atom_args()))
            elif i + 1 < len(toks) and toks[i + 1][1] == "is":
                var = _term(t0)
                if var[0] != "var":
                    raise SyntaxError("the left side of 'is' must be a variable")
                i += 2
                parts = [(1, term())]
                while toks[i][1] in ("+", "-"):
                    sign = 1 if toks[i][1] == "+" else -1
                    i += 1
                    parts.append((sign, term()))
                rule.assigns.append((var[1], parts))
            else:
                lhs = term()
                op = toks[i][1]
                if op not in CMP_OPS:
                    raise SyntaxError(f"cannot parse body literal near {op!r}")
                i += 1
                rule.filters.append((op, lhs, term()))
            if toks[i][1] == ".":
                i += 1
                break
            expect(",")
        rules.append(rule)
    return rules


# --------------------------------------------------------------------------
# Relations: (types, [columns]) with numpy columns of the types' dtypes.
# --------------------------------------------------------------------------
_NP = {"i32": np.int32, "f32": np.float32, "u32": np.uint32, "i64": np.int64, "u64": np.uint64,
       "f64": np.float64, "bool": np.bool_}
_INT_RANGE = {"i32": (-2 ** 31, 2 ** 31 - 1), "u32": (0, 2 ** 32 - 1), "i64": (-2 ** 63, 2 ** 63 - 1),
              "u64": (0, 2 ** 64 - 1), "bool": (0, 1)}
_SIGN64 = np.uint64(1 << 63)


def _const(t, ty):
    """Constant term t as a value of column type ty; TypeError if it is not one."""
    if ty in ("f32", "f64"):
        if t[0] != "float":
            raise TypeError(f"constant {t[1]!r} is not a {ty} value")
        return np.asarray(t[1], _NP[ty])
    lo, hi = _INT_RANGE[ty]
    if t[0] != "int" or not lo <= t[1] <= hi:
        raise TypeError(f"constant {t[1]!r} is not a {ty} value")
    return np.asarray(t[1], _NP[ty])


def _order(c):
    """Keys whose numeric order is the column type's order: f64 values by IEEE
    754 totalOrder (negative values: every bit flipped; others: the sign bit
    set, as unsigned 64-bit integers); other types as they are."""
    c = np.asarray(c)
    if c.dtype == np.float64:
        b = c.view(np.uint64)
        return np.where((b & _SIGN64) != 0, ~b, b | _SIGN64)
    return c


def _from_order(k):
    """Inverse of _order for f64 keys."""
    k = np.asarray(k, np.uint64)
    return np.where((k & _SIGN64) != 0, k & ~_SIGN64, ~k).view(np.float64)


def _eq(col, val):
    """Equality of values: identity for f64, IEEE equality for f32."""
    return _bits(col) == _bits(np.asarray(val, col.dtype)) if col.dtype == np.float64 else col == val


def _empty(types):
    return (tuple(types), [np.empty(0, _NP[t]) for t in types])


def _canonical(types, cols):
    """Distinct rows in ascending lexicographic order (each column in its
    type's order; f32 by value)."""
    cols = [np.asarray(c, _NP[t]) for t, c in zip(types, cols)]
    if len(cols[0]) == 0:
        return (tuple(types), cols)
    order = np.lexsort([_order(c) for c in cols][::-1])
    cols = [c[order] for c in cols]
    keep = np.ones(len(cols[0]), bool)
    same = np.ones(len(cols[0]) - 1, bool)
    for c in cols:
        same &= _bits(c)[1:] == _bits(c)[:-1]
    keep[1:] = ~same
    return (tuple(types), [c[keep] for c in cols])


def _bits(c):
    if c.dtype == np.float32:
        return c.view(np.int32)
    return c.view(np.int64) if c.dtype == np.float64 else c


def _identical(a, b):
    return all(len(x) == len(y) and np.array_equal(_bits(x), _bits(y))
               for x, y in zip(a[1], b[1]))


def _join_codes(left, right):
    """Dense integer codes such that equal codes <=> equal values in every column."""
    nl = len(left[0]) if left else 0
    code = None
    def ident(c):  # equal entries <=> equal values (f32 by IEEE value, f64 by identity)
        if c.dtype == np.float32:
            return np.asarray(c, np.float64)
        if c.dtype in (np.float64, np.uint64):
            return c.view(np.int64)
        return np.asarray(c, np.int64)

    for lc, rc in zip(left, right):
        vals = np.concatenate([ident(lc), ident(rc)])
        _, inv = np.unique(vals, return_inverse=True)
        inv = inv.astype(np.int64)
        code = inv if code is None else np.unique(code * (inv.max() + 1) + inv,
                                                  return_inverse=True)[1].astype(np.int64)
    return code[:nl], code[nl:]


def _eval_body(rule, rels, var_types):
    """All derivations of the rule body: dict var -> column, plus the count."""
    binding = {}
    n = 1
    for pred, terms in rule.atoms:
        types, cols = rels[pred]
        if len(terms) != len(types):
            raise TypeError(f"{pred}/{len(types)} used with {len(terms)} arguments")
        m = len(cols[0])
        mask = np.ones(m, bool)
        first = {}
        for j, t in enumerate(terms):
            if t[0] in ("int", "float"):
                mask &= _eq(cols[j], _const(t, types[j]))
            elif t[0] == "var":
                if var_types.setdefault(t[1], types[j]) != types[j]:
                    raise TypeError(f"variable {t[1]} used at two types")
                if t[1] in first:
                    mask &= cols[j] == cols[first[t[1]]]
                else:
                    first[t[1]] = j
        rows = [c[mask] for c in cols]
        shared = [v for v in first if v in binding]
        if shared:
            lcode, rcode = _join_codes([binding[v] for v in shared],
                                       [rows[first[v]] for v in shared])
            order = np.argsort(rcode, kind="stable")
            rs = rcode[order]
            lo = np.searchsorted(rs, lcode, "left")
            hi = np.searchsorted(rs, lcode, "right")
            cnt = hi - lo
            li = np.repeat(np.arange(n), cnt)
            start = np.cumsum(cnt) - cnt
            ri = order[lo[li] + np.arange(li.size) - start[li]]
        else:  # no shared variable: every pairing
            li = np.repeat(np.arange(n), len(rows[0]))
            ri = np.tile(np.arange(len(rows[0])), n)
        binding = {v: c[li] for v, c in binding.items()}
        for v, j in first.items():
            if v not in binding:
                binding[v] = rows[j][ri]
        n = li.size
    atom_vars = {t[1] for _, terms in rule.atoms for t in terms if t[0] == "var"}
    for var, parts in rule.assigns:
        if var in atom_vars:
            raise ValueError(f"{var} is both an 'is' result and an atom argument")
        ptypes = set()
        vals = []
        for sign, t in parts:
            if t[0] == "var":
                if t[1] not in binding:
                    raise ValueError(f"{t[1]} is unbound in an 'is' expression")
                ptypes.add(var_types[t[1]])
                vals.append((sign, binding[t[1]]))
            elif t[0] in ("int", "float"):
                ptypes.add("f32" if t[0] == "float" else "i32")
                vals.append((sign, t[1]))
            else:
                raise ValueError("'_' cannot appear in arithmetic")
        if len(ptypes) != 1:
            raise TypeError(f"mixed-type arithmetic for {var}")
        ty = ptypes.pop()
        if ty not in ("i32", "f32"):
            raise TypeError(f"arithmetic on {ty} values is not supported")
        # Left to right, one operation at a time, each result a value of the
        # operands' type (Sec. 3.2: arithmetic keeps scalar types): an f32
        # add or subtract is done in float64 and rounded to float32 at once,
        # which is the binary32 operation itself; i32 wraps modulo 2^32.  A
        # leading minus is 0 - x.
        wide = np.float64 if ty == "f32" else np.int64
        acc = None
        for sign, v in vals:
            t = np.broadcast_to(np.asarray(v, wide), (n,))
            if acc is None:
                acc = t.copy() if sign > 0 else np.zeros(n, wide) - t
            else:
                acc = acc + t if sign > 0 else acc - t
            if ty == "f32":
                acc = acc.astype(np.float32).astype(np.float64)
            else:
                acc = (acc + 2 ** 31) % 2 ** 32 - 2 ** 31
        if var_types.setdefault(var, ty) != ty:
            raise TypeError(f"variable {var} used at two types")
        binding[var] = acc.astype(np.float32) if ty == "f32" else acc.astype(np.int32)
    mask = np.ones(n, bool)
    for pred, terms in rule.negs:
        mask &= ~_negated_match(pred, terms, rels, binding, var_types, n)
    for op, a, b in rule.filters:
        ta = var_types[a[1]] if a[0] == "var" else None
        tb = var_types[b[1]] if b[0] == "var" else None
        if ta and tb and ta != tb:
            raise TypeError(f"comparison between {ta} and {tb}")
        ty = ta or tb
        if ty is None:  # two constants: their natural types
            ty = "f32" if a[0] == "float" else "i32"
            if ("f32" if b[0] == "float" else "i32") != ty:
                raise TypeError("comparison between i32 and f32")
        av = binding[a[1]] if a[0] == "var" else _const(a, ty)
        bv = binding[b[1]] if b[0] == "var" else _const(b, ty)
        mask &= {"!=": np.not_equal, "==": np.equal, "<": np.less, "<=": np.less_equal,
                 ">": np.greater, ">=": np.greater_equal}[op](_order(av), _order(bv))
    return {v: c[mask] for v, c in binding.items()}, int(mask.sum())


def _negated_match(pred, terms, rels, binding, var_types, n):
    """For each of the n derivations: does some row of pred agree with it on
    every variable and constant column of the negated literal?"""
    types, cols = rels[pred]
    if len(terms) != len(types):
        raise TypeError(f"{pred}/{len(types)} used with {len(terms)} arguments")
    mask = np.ones(len(cols[0]), bool)
    first = {}
    for j, t in enumerate(terms):
        if t[0] in ("int", "float"):
            mask &= _eq(cols[j], _const(t, types[j]))
        elif t[0] == "var":
            if t[1] not in binding:
                raise ValueError(f"{t[1]} occurs only in a negated literal")
            if var_types[t[1]] != types[j]:
                raise TypeError(f"variable {t[1]} used at two types")
            if t[1] in first:
                mask &= cols[j] == cols[first[t[1]]]
            else:
                first[t[1]] = j
    rows = [c[mask] for c in cols]
    if not first:  # only constants and '_': the literal fails iff such a row exists
        return np.full(n, len(rows[0]) > 0)
    if len(rows[0]) == 0 or n == 0:
        return np.zeros(n, bool)
    vs = list(first)
    lcode, rcode = _join_codes([binding[v] for v in vs], [rows[first[v]] for v in vs])
    return np.isin(lcode, rcode)


def _fold(op, keys, vals, ty):
    """Group rows by the key columns and fold vals over each group's derivations."""
    if len(vals) == 0:
        return keys, vals
    order = np.lexsort([_order(k) for k in keys][::-1]) if keys else np.arange(len(vals))
    keys = [k[order] for k in keys]
    vals = vals[order]
    start = np.ones(len(vals), bool)
    if keys:
        start[1:] = False
        for k in keys:
            start[1:] |= _bits(k)[1:] != _bits(k)[:-1]
    else:
        start[1:] = False
    idx = np.flatnonzero(start)
    gkeys = [k[idx] for k in keys]
    if op == "count":
        out = np.diff(np.append(idx, len(vals))).astype(np.int32)
    elif op in ("min", "max") and ty == "f64":  # by totalOrder
        red = np.minimum if op == "min" else np.maximum
        out = _from_order(red.reduceat(_order(vals), idx))
    elif op == "min":
        out = np.minimum.reduceat(vals, idx)
    elif op == "max":
        out = np.maximum.reduceat(vals, idx)
    elif op in ("sum", "logsumexp") and ty not in ("i32", "f32"):
        raise TypeError(f"{op} over {ty} values is not supported")
    elif op == "sum":
        if ty == "f32":
            out = np.add.reduceat(vals.astype(np.float64), idx).astype(np.float32)
        else:
            out = np.add.reduceat(vals.astype(np.int64), idx).astype(np.int32)
    elif op == "logsumexp":
        x = vals.astype(np.float64)
        m = np.maximum.reduceat(x, idx)
        seg = np.repeat(np.arange(len(idx)), np.diff(np.append(idx, len(x))))
        finite = np.isfinite(m)
        shift = np.where(finite, m, 0.0)
        s = np.add.reduceat(np.exp(x - shift[seg]), idx)
        with np.errstate(divide="ignore"):
            out = np.where(finite, m + np.log(s), m).astype(np.float32)
    else:
        raise ValueError(op)
    return gkeys, out


def _apply_rules(head, htypes, rules, rels):
    """T_P restricted to one head predicate."""
    keys_parts, vals_parts = [], []
    agg = None
    for r in rules:
        var_types = {}
        b, n = _eval_body(r, rels, var_types)
        for t in r.head_terms:
            if t[0] != "var" or t[1] not in b:
                raise ValueError(f"head {head}: every head argument must be a body variable")
        keys_parts.append([b[t[1]] for t in r.head_terms])
        if r.agg:
            agg = r.agg[0]
            vals_parts.append(b[r.agg[1]] if r.agg[0] != "count" else np.zeros(n, np.int32))
    nkey = len(htypes) - (1 if agg else 0)
    keys = [np.concatenate([p[j] for p in keys_parts]).astype(_NP[htypes[j]])
            for j in range(nkey)]
    if agg is None:
        return _canonical(htypes, keys)
    vtype = htypes[-1]
    vals = np.concatenate(vals_parts)
    if agg != "count":
        vals = vals.astype(_NP[vtype])
    gkeys, out = _fold(agg, keys, vals, vtype)
    return _canonical(htypes, gkeys + [np.asarray(out, _NP[vtype])])


def _strata(rules, idb):
    """Strongly connected components of the IDB dependency graph, dependencies first."""
    deps = {h: set() for h in idb}
    negdeps = []
    for r in rules:
        for pred, _ in r.atoms:
            if pred in idb:
                deps[r.head].add(pred)
        for pred, _ in r.negs:
            if pred in idb:
                deps[r.head].add(pred)
                negdeps.append((r.head, pred))
    index, low, stack, on, out = {}, {}, [], set(), []

    def visit(v):
        index[v] = low[v] = len(index)
        stack.append(v)
        on.add(v)
        for w in sorted(deps[v]):
            if w not in index:
                visit(w)
                low[v] = min(low[v], low[w])
            elif w in on:
                low[v] = min(low[v], index[w])
        if low[v] == index[v]:
            comp = []
            while True:
                w = stack.pop()
                on.discard(w)
                comp.append(w)
                if w == v:
                    break
            out.append(sorted(comp))

    for v in sorted(idb):
        if v not in index:
            visit(v)
    comp_of = {h: k for k, comp in enumerate(out) for h in comp}
    for head, pred in negdeps:
        if comp_of[head] == comp_of[pred]:
            raise ValueError(f"{head} depends negatively on {pred} inside one recursive component "
                             "(negation is stratified)")
    return out  # Tarjan emits components in reverse topological order of deps


@dataclass
class OracleResult:
    relations: dict                      # name -> (types, [columns]) canonical
    iterations: dict                     # stratum (tuple of heads) -> T_P applications
    sizes: dict                          # head -> row count after each application


def evaluate(rules_text: str, edb: dict, idb: dict, max_iterations: int = 10_000,
             restrict: dict | None = None) -> OracleResult:
    """Naive evaluation to the least fixpoint.

    edb: {name: (types, [columns])}; idb: {name: types}.
    restrict: optional {head: (column, allowed values)}.  After every
    application of T_P the head keeps only rows whose column lies in the
    allowed set.  This is only meaningful when the allowed set is closed under
    the rules' dependencies (for example when the column is passed unchanged
    from the recursive atom into the head); callers use it to compute selected
    rows of a large fixpoint one by one.
    """
    rules = parse(rules_text)
    rels = {k: _canonical(t, c) for k, (t, c) in edb.items()}
    for r in rules:
        if r.head not in idb:
            raise KeyError(f"rule head {r.head} has no declared schema")
    iterations, sizes = {}, {h: [] for h in idb}
    for comp in _strata(rules, idb):
        cur = {h: _empty(idb[h]) for h in comp}
        for k in range(1, max_iterations + 1):
            view = dict(rels)
            view.update(cur)
            nxt = {}
            for h in comp:
                nxt[h] = _apply_rules(h, tuple(idb[h]), [r for r in rules if r.head == h], view)
                if restrict and h in restrict:
                    col, allowed = restrict[h]
                    t, cs = nxt[h]
                    keep = np.isin(cs[col], np.asarray(allowed))
                    nxt[h] = (t, [c[keep] for c in cs])
                sizes[h].append(len(nxt[h][1][0]))
            done = all(_identical(nxt[h], cur[h]) for h in comp)
            cur = nxt
            if done:
                iterations[tuple(comp)] = k
                break
        else:
            raise ConvergenceFailure(f"no fixpoint for {comp} within {max_iterations} iterations")
        rels.update(cur)
    return OracleResult({h: rels[h] for h in idb}, iterations, sizes)
