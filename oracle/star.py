"""Plain numpy oracle for one star-schema query (test infrastructure only).

What it computes (the query shape the paper executes, Sections 3.3 and 4.2):

    live(i) = AND over fact predicates of pred(fact column value of row i)
              AND, for every join j, there is exactly one row r_j of dimension j
                  with key_j[r_j] == fact_key_j[i] that passes all predicates of
                  dimension j                          (inner join, Section 4.2)
    key(i)  = the group attributes payload(r_j), in GROUP BY order
    v(i)    = a | a*b | a-b | a+b over int64 operands, wrapping modulo 2**64
    result  = for every distinct key among live rows: (key, sum of v, count),
              sorted lexicographically by key; a query without GROUP BY returns
              one row (sum, count) even when no row is live.

Integer sums modulo 2**64 do not depend on the order of addition, so this is
the one correct answer for any execution order (the paper accepts a GPU result
only if its 64-bit integer equals the reference's bit for bit, Section 2.2).

How: each dimension is sorted by key once (a library sort); a fact key is
looked up by binary search (``numpy.searchsorted``) and accepted only on an
exact key match; predicates are evaluated on int64 copies of the columns in the
order the query lists them; groups are formed with ``numpy.unique`` over the
key tuples and summed with ``numpy.add.at`` in uint64. A BETWEEN predicate is
the conjunction of its two inclusive bounds (Section 4.2). Duplicate dimension
keys make the join ambiguous and raise ``DuplicateKeyError``.

This module is test infrastructure: it shares no code with the GPU library and
is imported only by the tests, the smoke entry point and the benchmark's
CPU-baseline measurement.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

class DuplicateKeyError(ValueError):
    """A dimension table holds the same key in more than one row."""


@dataclass
class OracleResult:
    keys: np.ndarray      # int64 [n_groups, n_keys], lexicographically sorted rows
    sums: np.ndarray      # int64 [n_groups], each the wrapped 64-bit sum
    counts: np.ndarray    # int64 [n_groups], live rows per group (>= 1 when grouped)
    n_live: int           # live fact rows in total

    def as_rows(self):
        return [(tuple(int(x) for x in k), int(s), int(c))
                for k, s, c in zip(self.keys, self.sums, self.counts)]


def eval_pred(values: np.ndarray, pred: dict) -> np.ndarray:
    """Boolean mask of one comparison of a column against int64 literals."""
    x = np.asarray(values).astype(np.int64)
    op, lo, hi = pred["op"], int(pred["lo"]), pred.get("hi")
    if op == "eq":
        return x == lo
    if op == "ne":
        return x != lo
    if op == "lt":
        return x < lo
    if op == "le":
        return x <= lo
    if op == "gt":
        return x > lo
    if op == "ge":
        return x >= lo
    if op == "between":
        return (x >= lo) & (x <= int(hi))
    raise ValueError(f"unknown predicate op {op!r}")


def _all_preds(table: dict, preds: list, n: int) -> np.ndarray:
    mask = np.ones(n, dtype=bool)
    for p in preds:
        mask &= eval_pred(table[p["col"]], p)
    return mask


@dataclass
class _DimIndex:
    sorted_keys: np.ndarray   # int64, ascending
    row_of: np.ndarray        # row number of each sorted key
    passes: np.ndarray        # bool per dimension row


def _index_dimension(dim: dict, key_col: str, preds: list) -> _DimIndex:
    keys = np.asarray(dim[key_col]).astype(np.int64)
    order = np.argsort(keys, kind="stable")
    sk = keys[order]
    if sk.size > 1 and np.any(sk[1:] == sk[:-1]):
        raise DuplicateKeyError(f"dimension key column {key_col!r} is not unique")
    return _DimIndex(sk, order, _all_preds(dim, preds, keys.size))


def _probe(idx: _DimIndex, fact_keys: np.ndarray) -> np.ndarray:
    """Row of the dimension whose key equals each fact key, or -1."""
    fk = np.asarray(fact_keys).astype(np.int64)
    m = idx.sorted_keys.size
    if m == 0:
        return np.full(fk.size, -1, dtype=np.int64)
    pos = np.searchsorted(idx.sorted_keys, fk, side="left")
    pos_c = np.minimum(pos, m - 1)
    hit = idx.sorted_keys[pos_c] == fk
    return np.where(hit, idx.row_of[pos_c], -1)


def _aggregate_operands(fact: dict, agg: dict, rows: np.ndarray) -> np.ndarray:
    a = np.asarray(fact[agg["a"]])[rows].astype(np.int64)
    kind = agg["kind"]
    if kind == "col":
        return a
    b = np.asarray(fact[agg["b"]])[rows].astype(np.int64)
    with np.errstate(over="ignore"):
        if kind == "mul":
            return a * b
        if kind == "sub":
            return a - b
        if kind == "add":
            return a + b
    raise ValueError(f"unknown aggregate {kind!r}")


def _join_index_of(query: dict, ref) -> int:
    if isinstance(ref, (int, np.integer)):
        return int(ref)
    for j, jd in enumerate(query["joins"]):
        if jd["dim"] == ref:
            return j
    raise KeyError(f"group key names dimension {ref!r}, which the query does not join")


def star_query(fact: dict, dims: dict, dim_keys: dict, query: dict) -> OracleResult:
    """Evaluate ``query`` over the fact columns ``fact`` and dimension tables ``dims``."""
    cols = [np.asarray(v) for v in fact.values()]
    n = int(cols[0].size) if cols else 0

    live = _all_preds(fact, query.get("fact_preds", []), n)

    matched_rows = []
    for jd in query.get("joins", []):
        dim = dims[jd["dim"]]
        idx = _index_dimension(dim, dim_keys[jd["dim"]], jd.get("preds", []))
        r = _probe(idx, fact[jd["fact_key"]])
        found = r >= 0
        passes = np.zeros(n, dtype=bool)
        passes[found] = idx.passes[r[found]]
        live &= passes
        matched_rows.append(r)

    rows = np.flatnonzero(live)
    v = _aggregate_operands(fact, query["agg"], rows)
    vu = v.view(np.uint64)

    group_by = query.get("group_by", [])
    if not group_by:
        total = np.array([vu.sum(dtype=np.uint64)], dtype=np.uint64).view(np.int64)
        return OracleResult(np.zeros((1, 0), dtype=np.int64), total,
                            np.array([rows.size], dtype=np.int64), int(rows.size))

    key_cols = []
    for ref, payload in group_by:
        j = _join_index_of(query, ref)
        dim = dims[query["joins"][j]["dim"]]
        key_cols.append(np.asarray(dim[payload]).astype(np.int64)[matched_rows[j][rows]])
    keys = np.stack(key_cols, axis=1) if rows.size else np.zeros((0, len(key_cols)), np.int64)

    uniq, inverse = np.unique(keys, axis=0, return_inverse=True)
    inverse = inverse.reshape(-1)
    sums = np.zeros(uniq.shape[0], dtype=np.uint64)
    np.add.at(sums, inverse, vu)
    counts = np.bincount(inverse, minlength=uniq.shape[0]).astype(np.int64)
    return OracleResult(uniq.astype(np.int64), sums.view(np.int64), counts, int(rows.size))

