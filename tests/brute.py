"""Nested-loop reference for tiny star schemas (pure Python, no numpy logic).

For every fact row it scans every row of every joined dimension, counts the
rows whose key equals the fact key, and keeps the fact row only if exactly one
such row exists and passes that dimension's predicates (a second match is an
error: dimension keys are primary keys). Sums are Python integers reduced
modulo 2**64 at the end. It shares nothing with the oracle, so agreement
between the two on many random schemas pins the oracle's join, filter and
grouping logic.
"""

from __future__ import annotations


class BruteDuplicateKey(Exception):
    pass


def _holds(x: int, p: dict) -> bool:
    op, lo, hi = p["op"], int(p["lo"]), p.get("hi")
    if op == "eq":
        return x == lo
    if op == "ne":
        return not x == lo
    if op == "lt":
        return x < lo
    if op == "le":
        return not x > lo
    if op == "gt":
        return x > lo
    if op == "ge":
        return not x < lo
    if op == "between":
        return lo <= x and x <= int(hi)
    raise ValueError(op)


def nested_loop_query(fact, dims, dim_keys, query):
    """Returns (rows, n_live) with rows = sorted [(key tuple, signed sum, count)]."""
    fcols = {k: [int(x) for x in v] for k, v in fact.items()}
    n = len(next(iter(fcols.values()))) if fcols else 0
    dcols = {d: {k: [int(x) for x in v] for k, v in t.items()} for d, t in dims.items()}
    joins = query.get("joins", [])

    def join_pos(ref):
        if isinstance(ref, int):
            return ref
        for j, jd in enumerate(joins):
            if jd["dim"] == ref:
                return j
        raise KeyError(ref)

    groups = {}
    n_live = 0
    for i in range(n):
        ok = all(_holds(fcols[p["col"]][i], p) for p in query.get("fact_preds", []))
        if not ok:
            continue
        matched = []
        for jd in joins:
            t = dcols[jd["dim"]]
            keycol = t[dim_keys[jd["dim"]]]
            want = fcols[jd["fact_key"]][i]
            hits = [r for r in range(len(keycol)) if keycol[r] == want]
            if len(hits) > 1:
                raise BruteDuplicateKey(jd["dim"])
            if not hits:
                ok = False
                break
            r = hits[0]
            if not all(_holds(t[p["col"]][r], p) for p in jd.get("preds", [])):
                ok = False
                break
            matched.append(r)
        if not ok:
            continue
        n_live += 1
        key = tuple(dcols[joins[join_pos(ref)]["dim"]][payload][matched[join_pos(ref)]]
                    for ref, payload in query.get("group_by", []))
        agg = query["agg"]
        a = fcols[agg["a"]][i]
        if agg["kind"] == "col":
            v = a
        else:
            b = fcols[agg["b"]][i]
            v = {"mul": a * b, "sub": a - b, "add": a + b}[agg["kind"]]
        s, c = groups.get(key, (0, 0))
        groups[key] = (s + v, c + 1)

    def signed64(x):
        x %= 1 << 64
        return x - (1 << 64) if x >= 1 << 63 else x

    if not query.get("group_by"):
        s, c = groups.get((), (0, 0))
        return [((), signed64(s), c)], n_live
    return sorted((k, signed64(s), c) for k, (s, c) in groups.items()), n_live


def has_duplicate_keys(dims, dim_keys, query) -> bool:
    for jd in query.get("joins", []):
        ks = [int(x) for x in dims[jd["dim"]][dim_keys[jd["dim"]]]]
        if len(set(ks)) != len(ks):
            return True
    return False
