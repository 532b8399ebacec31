"""Pins for the CPU oracle: checks against things other than the oracle itself.

* hand-derived worked examples of the query shapes the paper prints
  (tests/golden/*.json, each citing its section);
* a pure-Python nested-loop join on hundreds of random tiny schemas;
* invariants: group counts add up to an independently counted live mask, group
  sums add up to the ungrouped sum, results do not depend on the order of
  predicates or joins, and row ranges add up;
* special cases that reduce to a library routine (numpy take/where/sum/add.at);
* closed forms for the synthetic generators' expected counts and sums;
* planted mistakes: altered copies of the oracle must fail at least one pin.
"""

import glob
import json
import math
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st, HealthCheck

import datagen
from datagen.star import random_tiny_workload
import oracle
import oracle.star as ostar
from brute import nested_loop_query

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(res):
    return res.as_rows()


def _cmp(w):
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    rows, n_live = nested_loop_query(w.fact, w.dims, w.dim_keys, w.query)
    return _rows(res), res.n_live, rows, n_live


# ---------------------------------------------------------------- golden

@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(GOLDEN, "*example*.json"))))
def test_hand_derived_examples(path):
    g = json.load(open(path))
    fact = {k: np.array(v, dtype=np.int32) for k, v in g["fact"].items()}
    dims = {d: {k: np.array(v, dtype=np.int32) for k, v in t.items()} for d, t in g["dims"].items()}
    res = oracle.star_query(fact, dims, g["dim_keys"], g["query"])
    want = [(tuple(k), s, c) for k, s, c in g["expected"]["rows"]]
    assert _rows(res) == want
    assert res.n_live == g["expected"]["n_live"]
    # the nested-loop checker agrees with the hand derivation too
    rows, n_live = nested_loop_query(fact, dims, g["dim_keys"], g["query"])
    assert rows == want and n_live == g["expected"]["n_live"]


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("block", range(8))
def test_oracle_equals_nested_loop(block):
    for seed in range(block * 40, block * 40 + 40):
        w = random_tiny_workload(seed, max_fact=300, max_dim_rows=60)
        got, got_live, want, want_live = _cmp(w)
        assert got == want, f"seed {seed}"
        assert got_live == want_live, f"seed {seed}"


@settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(min_value=10_000, max_value=2**31 - 1),
       n=st.integers(min_value=0, max_value=120))
def test_oracle_equals_nested_loop_hypothesis(seed, n):
    w = random_tiny_workload(seed, max_fact=n, max_dim_rows=40, n_fact=n)
    got, got_live, want, want_live = _cmp(w)
    assert got == want and got_live == want_live


def test_duplicate_dimension_key_is_an_error():
    fact = {"fk": np.array([1, 2], np.int32), "v": np.array([5, 6], np.int32)}
    dims = {"d": {"k": np.array([1, 2, 1], np.int32), "a": np.array([0, 1, 2], np.int32)}}
    q = {"fact_preds": [], "joins": [{"fact_key": "fk", "dim": "d", "preds": [], "payloads": []}],
         "group_by": [], "agg": {"kind": "col", "a": "v", "b": None}}
    with pytest.raises(oracle.DuplicateKeyError):
        oracle.star_query(fact, dims, {"d": "k"}, q)


def test_empty_fact_table():
    w = datagen.make_workload("c3_star3", n_fact=0)
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    assert res.keys.shape == (0, 3) and res.n_live == 0
    w1 = datagen.make_workload("c1_scalar_scan", n_fact=0)
    r1 = oracle.star_query(w1.fact, w1.dims, w1.dim_keys, w1.query)
    assert _rows(r1) == [((), 0, 0)]


def test_literals_beyond_int32_range():
    v = np.array([-(2**31), -1, 0, 1, 2**31 - 1], dtype=np.int32)
    assert list(oracle.eval_pred(v, {"op": "lt", "lo": 2**31 + 5})) == [True] * 5
    assert list(oracle.eval_pred(v, {"op": "gt", "lo": -(2**31) - 1})) == [True] * 5
    assert list(oracle.eval_pred(v, {"op": "ge", "lo": 2**31})) == [False] * 5
    assert list(oracle.eval_pred(v, {"op": "between", "lo": 1, "hi": 0})) == [False] * 5
    assert list(oracle.eval_pred(v, {"op": "ne", "lo": 2**40})) == [True] * 5
    assert list(oracle.eval_pred(v, {"op": "le", "lo": -(2**31)})) == [True, False, False, False, False]


# ---------------------------------------------------------------- invariants

def _independent_live_mask(w):
    """Live mask of a dense-key workload computed by direct indexing (no sort, no search)."""
    n = w.n_fact
    live = np.ones(n, dtype=bool)
    for p in w.query["fact_preds"]:
        x = w.fact[p["col"]].astype(np.int64)
        lo = p["lo"]
        live &= {"eq": lambda: x == lo, "lt": lambda: x < lo,
                 "between": lambda: (lo <= x) & (x <= p["hi"])}[p["op"]]()
    for jd in w.query["joins"]:
        dim = w.dims[jd["dim"]]
        keys = dim[w.dim_keys[jd["dim"]]]
        assert np.array_equal(keys, np.arange(keys.size)), "dense identity keys expected"
        ok = np.ones(keys.size, dtype=bool)
        for p in jd["preds"]:
            x = dim[p["col"]].astype(np.int64)
            ok &= (x == p["lo"]) if p["op"] == "eq" else ((p["lo"] <= x) & (x <= p["hi"]))
        live &= np.take(ok, w.fact[jd["fact_key"]])
    return live


@pytest.mark.parametrize("name,n", [("c1_scalar_scan", None), ("c2_join_group", 2_000_000),
                                    ("c3_star3", 2_000_000), ("c4_star4_zipf", 2_000_000)])
def test_counts_add_up_to_live_rows(name, n):
    w = datagen.make_workload(name, n_fact=n)
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    live = _independent_live_mask(w)
    assert int(res.counts.sum()) == int(live.sum()) == res.n_live


@pytest.mark.parametrize("name", ["c2_join_group", "c3_star3", "c4_star4_zipf"])
def test_group_sums_add_up_to_ungrouped_sum(name):
    w = datagen.make_workload(name, n_fact=1_000_000)
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    q2 = dict(w.query, group_by=[])
    tot = oracle.star_query(w.fact, w.dims, w.dim_keys, q2)
    assert int(res.sums.view(np.uint64).sum(dtype=np.uint64)) == int(tot.sums.view(np.uint64)[0])
    assert int(res.counts.sum()) == int(tot.counts[0])


def test_order_of_predicates_and_joins_does_not_matter():
    for seed in range(60):
        w = random_tiny_workload(seed + 500, max_fact=400, max_dim_rows=80)
        base = _rows(oracle.star_query(w.fact, w.dims, w.dim_keys, w.query))
        q = json.loads(json.dumps(w.query))
        q["fact_preds"] = q["fact_preds"][::-1]
        q["joins"] = q["joins"][::-1]
        # group_by names dimensions, so reordering joins keeps key order
        assert _rows(oracle.star_query(w.fact, w.dims, w.dim_keys, q)) == base, seed


def test_row_ranges_add_up():
    w = datagen.make_workload("c3_star3", n_fact=1_500_000)
    full = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    acc = {}
    for lo, hi in [(0, 333_333), (333_333, 1_000_001), (1_000_001, 1_500_000)]:
        part = {k: v[lo:hi] for k, v in w.fact.items()}
        for k, s, c in oracle.star_query(part, w.dims, w.dim_keys, w.query).as_rows():
            s0, c0 = acc.get(k, (0, 0))
            acc[k] = ((s0 + s) % (1 << 64), c0 + c)
    merged = sorted((k, s - (1 << 64) if s >= 1 << 63 else s, c) for k, (s, c) in acc.items())
    assert merged == full.as_rows()


# ---------------------------------------------------------------- library routines

def test_scalar_query_equals_numpy_where_sum():
    w = datagen.make_workload("c1_scalar_scan")
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    year_of_key = w.dims["date"]["year"]                       # key == row index
    mask = (np.take(year_of_key, w.fact["date_key"]) == 1994)
    mask &= (w.fact["disc"] >= 2) & (w.fact["disc"] <= 4) & (w.fact["qty"] < 30)
    prod = w.fact["price"].astype(np.int64) * w.fact["disc"].astype(np.int64)
    assert int(res.sums[0]) == int(np.sum(np.where(mask, prod, 0), dtype=np.int64))
    assert int(res.counts[0]) == int(mask.sum())


def test_single_key_group_equals_numpy_add_at():
    w = datagen.make_workload("c2_join_group", n_fact=3_000_000)
    q = dict(w.query, group_by=[["supplier", "nation"]])
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, q)
    sup = w.dims["supplier"]
    ok = np.take(sup["region"] == 2, w.fact["supp_key"])
    nation = np.take(sup["nation"], w.fact["supp_key"])
    out = np.zeros(25, dtype=np.int64)
    np.add.at(out, nation[ok], w.fact["revenue"][ok].astype(np.int64))
    cnt = np.bincount(nation[ok], minlength=25)
    present = np.flatnonzero(cnt)
    assert [k[0] for k in res.keys] == list(present)
    assert list(res.sums) == list(out[present])
    assert list(res.counts) == list(cnt[present])


# ---------------------------------------------------------------- closed forms

def test_c1_closed_form_count_and_sum():
    w = datagen.make_workload("c1_scalar_scan")
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    n = w.n_fact
    p = (365 / 2556) * (3 / 11) * (29 / 50)
    mean = n * p
    sd = math.sqrt(n * p * (1 - p))
    assert abs(int(res.counts[0]) - mean) < 5 * sd, (int(res.counts[0]), mean)
    # E[price*disc | disc in {2,3,4}] = E[price] * 3 with price ~ U[90000, 10^7]
    mu_price = (90_000 + 10_000_000) / 2
    var_price = ((10_000_000 - 90_000 + 1) ** 2 - 1) / 12
    e_v = mu_price * 3
    e_v2 = (var_price + mu_price ** 2) * (4 + 9 + 16) / 3
    sd_sum = math.sqrt(n * (p * e_v2 - (p * e_v) ** 2))
    assert abs(int(res.sums[0]) - n * p * e_v) < 5 * sd_sum


def test_c2_closed_form_group_counts():
    n = 3_000_000
    w = datagen.make_workload("c2_join_group", n_fact=n)
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    sup = w.dims["supplier"]
    # supplier share per nation among region-2 suppliers, counted from the table itself
    share = np.bincount(sup["nation"][sup["region"] == 2], minlength=25) / sup["nation"].size
    days = {y: 365 for y in range(1992, 1999)}
    days[1999] = 1
    got = {k: c for k, _, c in res.as_rows()}
    assert len(got) == 25 * 8
    for nation in range(25):
        for year, nd in days.items():
            p = share[nation] * nd / 2556
            mean, sd = n * p, math.sqrt(n * p * (1 - p))
            c = got[(nation, year)]
            assert abs(c - mean) < 6 * sd + 3, (nation, year, c, mean)


def test_c3_closed_form_survivors():
    """c3's fact keys are uniform over the dimension keys, so a row survives
    with the product of the three dimensions' pass fractions (customer and
    supplier region 2, about 1/5 each; 1992-1997, 2190 of 2556 days): about
    3.43% of the rows, 20.56M of 600M. The oracle's total count and sum on a
    2M-row head agree within 6 standard deviations, and every group key lies
    in the payload domains (250 cities, six years)."""
    n = 2_000_000
    w = datagen.make_workload("c3_star3", n_fact=n)
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    p_c = float(np.mean(w.dims["customer"]["region"] == 2))
    p_s = float(np.mean(w.dims["supplier"]["region"] == 2))
    p_d = 6 * 365 / 2556
    p = p_c * p_s * p_d
    assert abs(p - 0.0343) < 0.001
    mean, sd = n * p, math.sqrt(n * p * (1 - p))
    total = int(np.sum(res.counts))
    assert abs(total - mean) < 6 * sd, (total, mean)
    # revenue ~ U[1, 10^6] independent of the keys
    e_v, var_v = (1 + 1_000_000) / 2, (1_000_000 ** 2 - 1) / 12
    sd_sum = math.sqrt(n * (p * (var_v + e_v ** 2) - (p * e_v) ** 2))
    assert abs(int(np.sum(res.sums)) - n * p * e_v) < 6 * sd_sum
    keys = np.array(res.keys)
    assert keys[:, 0].min() >= 0 and keys[:, 0].max() <= 249 and keys[:, 1].max() <= 249
    assert set(keys[:, 2].tolist()) == set(range(1992, 1998))


def test_c5_closed_form_survivors():
    """Every c5 fact key exists in the dimension (its keys are a permutation of
    0..2^24-1) and half of the dimension rows pass: about half of the fact
    rows survive, 300M of 600M, about 4,578 per group of 65,536; the oracle's
    totals on a 2M-row head agree within 6 standard deviations."""
    n = 2_000_000
    w = datagen.make_workload("c5_hash_stress", n_fact=n)
    res = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    p = float(np.mean(w.dims["big"]["flag"] == 1))
    mean, sd = n * p, math.sqrt(n * p * (1 - p))
    total = int(np.sum(res.counts))
    assert abs(total - mean) < 6 * sd, (total, mean)
    assert abs(600_000_000 * p / 65536 - 4578) < 10
    e_v, var_v = (1 + 1_000_000) / 2, (1_000_000 ** 2 - 1) / 12
    sd_sum = math.sqrt(n * (p * (var_v + e_v ** 2) - (p * e_v) ** 2))
    assert abs(int(np.sum(res.sums)) - n * p * e_v) < 6 * sd_sum
    assert len(res.counts) <= 65536 and np.array(res.keys)[:, 0].max() <= 65535


def test_c4_zipf_head_mass():
    cdf = datagen.zipf_cdf(1_400_000, 1.1)
    h = np.sum(np.arange(1, 1_400_001, dtype=np.float64) ** -1.1)
    assert abs(h - 8.1557) < 1e-3
    assert abs(cdf[0] - 0.1226) < 1e-3 and abs(cdf[9] - 0.329) < 1e-3 and abs(cdf[99] - 0.525) < 1e-3
    z = datagen.fact_column("c4_star4_zipf", "part_key", 0, 2_000_000)
    assert abs((z == 0).mean() - cdf[0]) < 5 * math.sqrt(cdf[0] * (1 - cdf[0]) / z.size)


def test_c5_keys_are_a_permutation_and_half_pass():
    w = datagen.make_workload("c5_hash_stress", n_fact=1000)
    k = w.dims["big"]["key"]
    assert np.array_equal(np.sort(k), np.arange(1 << 24, dtype=np.int32))
    assert abs(w.dims["big"]["flag"].mean() - 0.5) < 0.001


# ---------------------------------------------------------------- planted mistakes

def _pins_catch(monkeypatch, name, fake):
    """Run the brute-force pin with a broken oracle piece; return True if a mismatch shows."""
    with monkeypatch.context() as m:
        m.setattr(ostar, name, fake)
        for seed in range(200):
            w = random_tiny_workload(seed, max_fact=200, max_dim_rows=40)
            try:
                got, got_live, want, want_live = _cmp(w)
            except Exception:
                return True
            if got != want or got_live != want_live:
                return True
        for path in sorted(glob.glob(os.path.join(GOLDEN, "*example*.json"))):
            g = json.load(open(path))
            fact = {k: np.array(v, dtype=np.int32) for k, v in g["fact"].items()}
            dims = {d: {k: np.array(v, dtype=np.int32) for k, v in t.items()}
                    for d, t in g["dims"].items()}
            res = ostar.star_query(fact, dims, g["dim_keys"], g["query"])
            if res.as_rows() != [(tuple(k), s, c) for k, s, c in g["expected"]["rows"]]:
                return True
    return False


def test_planted_mistakes_are_caught(monkeypatch):
    real_eval = ostar.eval_pred
    real_agg = ostar._aggregate_operands
    real_probe = ostar._probe
    real_index = ostar._index_dimension

    def lt_as_le(values, pred):
        if pred["op"] == "lt":
            return real_eval(values, dict(pred, op="le"))
        return real_eval(values, pred)

    def between_exclusive(values, pred):
        if pred["op"] == "between":
            x = np.asarray(values).astype(np.int64)
            return (x > pred["lo"]) & (x < pred["hi"])
        return real_eval(values, pred)

    def sub_reversed(fact, agg, rows):
        if agg["kind"] == "sub":
            return real_agg(fact, dict(agg, a=agg["b"], b=agg["a"]), rows)
        return real_agg(fact, agg, rows)

    def mul_in_int32(fact, agg, rows):
        v = real_agg(fact, agg, rows)
        return v.astype(np.int32).astype(np.int64) if agg["kind"] == "mul" else v

    def probe_ignores_key_match(idx, fact_keys):
        fk = np.asarray(fact_keys).astype(np.int64)
        m = idx.sorted_keys.size
        if m == 0:
            return np.full(fk.size, -1, dtype=np.int64)
        pos = np.minimum(np.searchsorted(idx.sorted_keys, fk), m - 1)
        return idx.row_of[pos]

    def dims_unfiltered(dim, key_col, preds):
        return real_index(dim, key_col, [])

    for name, fake in [("eval_pred", lt_as_le), ("eval_pred", between_exclusive),
                       ("_aggregate_operands", sub_reversed),
                       ("_aggregate_operands", mul_in_int32),
                       ("_probe", probe_ignores_key_match),
                       ("_index_dimension", dims_unfiltered)]:
        assert _pins_catch(monkeypatch, name, fake), f"planted mistake {fake.__name__} not caught"
    assert ostar.eval_pred is real_eval and ostar._probe is real_probe
