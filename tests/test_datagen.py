"""The seeded generators: determinism, row-range regeneration, value ranges."""

import numpy as np
import pytest

import datagen
from datagen.star import CONFIGS, random_tiny_workload


def test_same_seed_same_rows_and_ranges_regenerate():
    a = datagen.fact_column("c3_star3", "cust_key", 0, 9_000_000, threads=4)
    b = datagen.fact_column("c3_star3", "cust_key", 0, 9_000_000, threads=1)
    assert np.array_equal(a, b)
    c = datagen.fact_column("c3_star3", "cust_key", 4_194_300, 4_194_400)
    assert np.array_equal(c, a[4_194_300:4_194_400])


@pytest.mark.parametrize("name", list(CONFIGS))
def test_value_ranges(name):
    cfg = CONFIGS[name]
    rows = datagen.fact_rows(name, 0, 200_000)
    for col in cfg.fact_cols:
        v = rows[col.name]
        assert v.dtype == np.int32 and v.size == 200_000
        if col.dist[0] == "uniform":
            assert v.min() >= col.dist[1] and v.max() <= col.dist[2]
        if col.dist[0] == "zipf":
            assert v.min() >= 0 and v.max() < col.dist[1]
        if col.dist[0] == "ramp":
            assert np.all(np.diff(v) >= 0) and v[0] == col.dist[1]


def test_date_sorted_variant():
    """The date-sorted c3 variant: every day holds an equal run of rows (up to
    one row), in ascending order; the other columns follow c3's recipe with
    seeds of their own."""
    n = 600_000_000
    ends = datagen.fact_column("c3d_star3_date_sorted", "date_key", n - 5, n)
    assert list(ends) == [2555] * 5
    mid = datagen.fact_column("c3d_star3_date_sorted", "date_key", 300_000_000 - 2, 300_000_000 + 2)
    assert list(mid) == [1277, 1277, 1278, 1278]            # 2556 days: row 3e8 starts day 1278
    a = datagen.fact_column("c3d_star3_date_sorted", "cust_key", 0, 100_000)
    assert a.min() >= 0 and a.max() <= 2_999_999 and np.unique(a).size > 95_000


def test_date_dimension_recipe():
    w = datagen.make_workload("c1_scalar_scan", n_fact=10)
    d = w.dims["date"]
    assert np.array_equal(d["date_key"], np.arange(2556))
    assert d["year"][0] == 1992 and d["year"][364] == 1992 and d["year"][365] == 1993
    assert d["year"][2554] == 1998 and d["year"][2555] == 1999


def test_tiny_workloads_have_distinct_dimension_keys():
    for s in range(100):
        w = random_tiny_workload(s)
        for d, t in w.dims.items():
            k = t[w.dim_keys[d]]
            assert np.unique(k).size == k.size
