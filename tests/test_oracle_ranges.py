"""Pins for the oracle over row ranges (oracle/ranges.py).

The merge of partial results over disjoint row ranges must equal the oracle
over the whole table (a SUM and a COUNT are additive over disjoint row sets,
modulo 2**64 for the sums), and must equal a plain Python dict merge. The
worker-pool runners must return what the oracle returns in this process.
"""

import numpy as np
import pytest

import datagen
from datagen.star import CHUNK, random_tiny_workload
import oracle
from oracle import ranges


def _dict_merge(parts):
    acc = {}
    for r in parts:
        for k, s, c in r.as_rows():
            s0, c0 = acc.get(k, (0, 0))
            acc[k] = ((s0 + s) % (1 << 64), c0 + c)
    return sorted((k, s - (1 << 64) if s >= 1 << 63 else s, c) for k, (s, c) in acc.items())


def _parts(w, cuts):
    out = []
    for lo, hi in zip(cuts[:-1], cuts[1:]):
        part = {k: v[lo:hi] for k, v in w.fact.items()}
        out.append(oracle.star_query(part, w.dims, w.dim_keys, w.query))
    return out


@pytest.mark.parametrize("name,n", [("c1_scalar_scan", 300_001), ("c2_join_group", 400_003),
                                    ("c3_star3", 500_009)])
def test_merge_of_ranges_equals_whole(name, n):
    w = datagen.make_workload(name, n_fact=n)
    whole = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    cuts = [0, 1, 77_777, 77_777, n // 2 + 3, n]          # an empty range and a 1-row range included
    parts = _parts(w, cuts)
    m = ranges.merge(parts)
    assert m.as_rows() == whole.as_rows()
    assert m.n_live == whole.n_live
    assert m.as_rows() == _dict_merge(parts)


@pytest.mark.parametrize("seed", range(40))
def test_merge_on_tiny_schemas(seed):
    w = random_tiny_workload(seed)          # distinct dimension keys (tests/test_datagen.py)
    whole = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    n = w.n_fact
    rng = np.random.default_rng(seed)
    cuts = sorted([0, n] + [int(x) for x in rng.integers(0, n + 1, size=3)])
    parts = _parts(w, cuts)
    m = ranges.merge(parts)
    assert m.as_rows() == whole.as_rows()
    assert m.n_live == whole.n_live
    if w.query["group_by"]:
        assert m.as_rows() == _dict_merge(parts)


def test_merge_wraps_modulo_2_64():
    """Two parts whose sums overflow int64 when added merge to the wrapped value."""
    big = oracle.OracleResult(np.array([[1], [2]]), np.array([(1 << 63) - 5, -7], dtype=np.int64),
                              np.array([3, 1]), 4)
    big2 = oracle.OracleResult(np.array([[1], [3]]), np.array([10, 4], dtype=np.int64),
                               np.array([2, 2]), 4)
    m = ranges.merge([big, big2])
    assert m.as_rows() == [((1,), (1 << 63) + 5 - (1 << 64), 5), ((2,), -7, 1), ((3,), 4, 2)]
    assert m.n_live == 8


def test_row_ranges_cover_and_align():
    for n, parts in [(0, 4), (1, 4), (CHUNK, 3), (10 * CHUNK + 5, 4), (600_000_000, 16)]:
        rr = ranges.row_ranges(n, parts, CHUNK)
        assert len(rr) <= max(1, parts)
        assert rr[0][0] == 0 and rr[-1][1] == n
        for (a, b), (c, _) in zip(rr[:-1], rr[1:]):
            assert b == c and b % CHUNK == 0 and a < b


def test_pool_runners_equal_the_oracle_in_process():
    """Both runners on two worker processes from the fork server: the merged
    result equals the in-process oracle, the column sums equal numpy's."""
    ranges.start_forkserver()
    name, n = "c2_join_group", 2 * CHUNK + 12_345
    w = datagen.make_workload(name, n_fact=n)
    whole = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    want_sums = {k: int(v.astype(np.int64).sum()) for k, v in w.fact.items()}
    with ranges.pool(2) as ex:
        got, sums = ranges.run(name, n, ex, task_rows=CHUNK)
    assert got.as_rows() == whole.as_rows() and sums == want_sums
    got, sums, info = ranges.run_timed(name, n, workers=2)
    assert got.as_rows() == whole.as_rows() and sums == want_sums
    assert info["workers"] == 2 and info["wall_s"] > 0 and len(info["worker_oracle_s"]) == 2
