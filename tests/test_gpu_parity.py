"""GPU parity: the HIP path through the C ABI against the CPU oracle, exactly.

All arithmetic is integer, so every group key, sum and count must be equal bit
for bit. Sizes here let the oracle finish in seconds while still spanning many
blocks, tiles and a ragged tail; the full 600M-row shapes are covered in
test_gpu_fullsize.py.
"""

import numpy as np
import pytest

import datagen
import oracle
from datagen.star import random_tiny_workload
from gpu_util import assert_same, oracle_rows, require_gpu, run_gpu, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


SIZES = {"c1_scalar_scan": None, "c2_join_group": 4_000_003, "c3_star3": 4_000_001,
         "c4_star4_zipf": 4_000_002, "c5_hash_stress": 2_000_003}

_cache = {}
_want = {}


def workload(name):
    if name not in _cache:
        _cache[name] = datagen.make_workload(name, n_fact=SIZES[name])
    return _cache[name]


def want_rows(name):
    """The oracle's result of workload(name), computed once per session."""
    if name not in _want:
        _want[name] = oracle_rows(workload(name))
    return _want[name]


@pytest.mark.parametrize("name", list(SIZES))
def test_config_parity(name):
    w = workload(name)
    want = want_rows(name)
    got, q = run_gpu(w)
    print(name, w.n_fact, "rows;", len(want), "groups;", q.plan_obj.terminal, q.plan_obj.ipt)
    assert_same(got.as_rows(), want, name)


@pytest.mark.parametrize("name", ["c2_join_group", "c3_star3", "c4_star4_zipf"])
@pytest.mark.parametrize("force", [
    {"order": True}, {"vector": -1}, {"ipt": 1}, {"ipt": 4}, {"terminal": "global"},
    {"ipt": 4, "vector": -1, "terminal": "global"}, {"grid": 7}, {"grid": 1, "ipt": 2},
    {"terminal": "part"}, {"terminal": "part", "ipt": 1}, {"terminal": "part", "ipt": 4, "vector": -1},
    {"terminal": "part", "grid": 5},
    {"eager": 4}, {"eager": 4, "ipt": 1}, {"eager": 2, "terminal": "part"}, {"eager": 1, "terminal": "global", "grid": 3},
    {"eager": -1}, {"block": 1024}, {"block": 1024, "ipt": 1, "terminal": "part"}, {"block": 512, "ipt": 1},
    {"block": 64, "ipt": 2, "terminal": "global"}, {"lds": 2}, {"lds": 2, "terminal": "part"},
    {"lds": 3}, {"lds": 3, "terminal": "global"}, {"lds": 3, "ipt": 1, "terminal": "part"},
    {"ipt": 1, "block": 1024, "terminal": "global"},
    {"coarse": 1}, {"coarse": 2}, {"coarse": 3, "terminal": "global"}, {"coarse": 5, "ipt": 1, "block": 1024},
    {"coarse": 2, "lds": -1}, {"coarse": 4, "block": 1024, "terminal": "part"},
])
def test_forced_plans_agree(name, force):
    w = workload(name)
    want = want_rows(name)
    got, _ = run_gpu(w, force=force)
    assert_same(got.as_rows(), want, f"{name} {force}")


# every terminal a workload's query admits: the scalar terminal needs a query
# without GROUP BY, and c3's 375,000 groups do not fit the LDS terminal
_UNROLL_CASES = [(name, terminal) for name in ["c1_scalar_scan", "c2_join_group", "c3_star3"]
                 for terminal in ["auto", "scalar", "lds", "global", "part"]
                 if not (terminal == "scalar" and name != "c1_scalar_scan")
                 and not (terminal == "lds" and name == "c3_star3")]


@pytest.mark.parametrize("name,terminal", _UNROLL_CASES)
def test_unrolled_stage_loop_agrees(name, terminal):
    # the instance with the stage loop written out against the loop, per terminal
    w = workload(name)
    want = want_rows(name)
    force = {} if terminal == "auto" else {"terminal": terminal}
    got_u, qu = run_gpu(w, force=force)
    got_l, ql = run_gpu(w, force={**force, "unroll": -1})
    assert ql.plan_obj.unroll == 0
    if terminal == "auto":
        assert qu.plan_obj.unroll == 1
    assert_same(got_u.as_rows(), want, f"{name} {terminal} unrolled")
    assert_same(got_l.as_rows(), want, f"{name} {terminal} loop")


@pytest.mark.parametrize("mode", ["per_operator", "global_handoff"])
@pytest.mark.parametrize("name", list(SIZES))
def test_baselines_agree(name, mode):
    from paper_2607_07632_amd import sdb
    w = workload(name)
    fact, dims = upload(w)
    q = sdb.StarQuery(fact, sdb.build_dims(dims, w.dim_keys, w.query), w.query)
    assert_same(q.execute(baseline=mode).as_rows(), want_rows(name), f"{name} {mode}")


@pytest.mark.parametrize("mode", ["per_operator", "global_handoff"])
@pytest.mark.parametrize("n", [0, 1, 5, 257, 4097])
def test_baselines_small_and_tiny_schemas(n, mode):
    from paper_2607_07632_amd import sdb
    for seed in (5, 17):
        w = random_tiny_workload(seed, n_fact=n)
        fact, dims = upload(w)
        q = sdb.StarQuery(fact, sdb.build_dims(dims, w.dim_keys, w.query), w.query)
        assert_same(q.execute(baseline=mode).as_rows(), oracle_rows(w), f"{mode} seed {seed} n {n}")


@pytest.mark.parametrize("force", [
    {"ipt": 2, "block": 512}, {"ipt": 2, "block": 1024}, {"ipt": 4}, {"vector": -1}, {"terminal": "global"},
    {"terminal": "global", "xcd": -1}, {"eager": 2, "ipt": 1, "block": 512}, {"grid": 3}, {"order": True},
    {"slice": 1}, {"slice": 1, "terminal": "global"}, {"slice": 1, "terminal": "global", "xcd": -1},
    {"slice": 1, "vector": -1}, {"slice": 1, "grid": 3}, {"slice": 1, "ipt": 2, "block": 512},
    {"slice": 1, "ipt": 4, "block": 256}, {"slice": 1, "terminal": "part", "grid": 5},
])
def test_c5_forced_plans_agree(force):
    w = workload("c5_hash_stress")
    got, q = run_gpu(w, force=force)
    assert bool(q.plan_obj.slice_bits) == bool(force.get("slice"))
    assert_same(got.as_rows(), want_rows("c5_hash_stress"), f"c5 {force}")


def _sliceable(w, load_factor=0.5, keep_agg=False):
    """w's query narrowed to the shape a sliced hash probe serves: its first
    join only, as a hash table, group keys from that join, and (unless
    keep_agg) SUM of one column (the fact predicates stay)."""
    import copy
    q = copy.deepcopy(w.query)
    j = dict(q["joins"][0], kind="hash", load_factor=load_factor)
    q["joins"] = [j]
    q["group_by"] = [g for g in q["group_by"] if g[0] == j["dim"]]
    if not keep_agg:
        q["agg"] = {"kind": "col", "a": q["agg"]["a"], "b": None}
    return datagen.Workload(w.name, w.n_fact, w.fact, w.dims, w.dim_keys, q)


@pytest.mark.parametrize("n", [1, 16_385, 70_001, 400_003])
@pytest.mark.parametrize("kind", ["mul", "sub", "add"])
def test_sliced_probe_with_two_column_aggregates(n, kind):
    """Sliced probes whose aggregate combines two columns (both operands travel
    with the key through the scatter pass): random one-join schemas, every
    terminal shape, against the oracle."""
    done = 0
    for seed in range(60):
        w0 = random_tiny_workload(3000 + seed, n_fact=n, max_dim_rows=3000)
        if not w0.query["joins"] or len(w0.fact) < 3:
            continue
        w = _sliceable(w0, load_factor=(0.5, 0.25, 0.9)[seed % 3], keep_agg=True)
        vals = [c for c in w.fact if c.startswith("v")]
        w.query["agg"] = {"kind": kind, "a": vals[0], "b": vals[-1]}
        want = oracle_rows(w)
        for force in ({"slice": 1}, {"slice": 1, "terminal": "global"}, {"slice": 1, "terminal": "part"}):
            got, q = run_gpu(w, force=force)
            assert q.plan_obj.slice_bits > 0, (seed, force)
            assert_same(got.as_rows(), want, f"seed {seed} n {n} {kind} {force}")
        done += 1
        if done == 2:
            break
    assert done == 2


def test_sliced_probe_c5_with_a_difference():
    """c5's shape with SUM(value - key) through the sliced probe, both
    operands in the partitioned records (64-bit record values)."""
    w0 = workload("c5_hash_stress")
    w = datagen.Workload("c5 difference", w0.n_fact, w0.fact, w0.dims, w0.dim_keys,
                         {**w0.query, "agg": {"kind": "sub", "a": "value", "b": "key"}})
    got, q = run_gpu(w, force={"slice": 1})
    assert q.plan_obj.slice_bits > 0
    assert_same(got.as_rows(), oracle_rows(w), "c5 value - key, sliced")


# row counts around the passes' 16,384-row chunks, up to many blocks
@pytest.mark.parametrize("n", [0, 1, 5, 16_383, 16_384, 16_385, 70_001, 400_003])
def test_sliced_probe_on_random_tiny_schemas(n):
    """Sliced probes (forced) over random one-join schemas with fact
    predicates, negative keys and values, misses and filtered rows: the
    oracle's groups, sums and counts exactly."""
    from paper_2607_07632_amd import sdb
    done = 0
    for seed in range(40):
        w0 = random_tiny_workload(1000 + seed, n_fact=n, max_dim_rows=3000)
        if not w0.query["joins"]:
            continue
        w = _sliceable(w0, load_factor=(0.5, 0.25, 0.9)[seed % 3])
        for force in ({"slice": 1}, {"slice": 1, "terminal": "global"}, {"slice": 1, "order": True}):
            got, q = run_gpu(w, force=force)
            assert q.plan_obj.slice_bits > 0 or n == 0, (seed, force)
            assert_same(got.as_rows(), oracle_rows(w), f"seed {seed} n {n} {force}")
        done += 1
        if done == 3:
            break
    assert done == 3


def test_sliced_probe_at_every_slice_count():
    """The partition count follows the table size (slices of 2 MiB, at
    least 2): one-join schemas with 2^9 ... 2^24 dimension rows (keys with
    gaps and negative values, half filtered out) give 1 ... 8 slice bits,
    each with the oracle's result."""
    rng = np.random.default_rng([2607, 7632, 61])
    n = 300_007
    seen = set()
    for m, lf in ((1 << 9, 0.5), (1 << 18, 0.5), (1 << 19, 0.5), (1 << 20, 0.5), (1 << 22, 0.5),
                  (1 << 24, 0.25)):
        keys = (rng.permutation(2 * m)[:m] - m).astype(np.int32)
        dims = {"big": {"key": keys, "flag": rng.integers(0, 2, m, dtype=np.int32),
                        "attr": rng.integers(0, 1000, m, dtype=np.int32)}}
        fact = {"key": rng.integers(-m - 10, m + 10, n, dtype=np.int32),
                "value": rng.integers(-10**6, 10**6, n, dtype=np.int32)}
        query = {"fact_preds": [{"col": "value", "op": "ge", "lo": -900_000, "hi": None}],
                 "joins": [{"fact_key": "key", "dim": "big", "preds": [{"col": "flag", "op": "eq", "lo": 1, "hi": None}],
                            "payloads": ["attr"], "kind": "hash", "load_factor": lf}],
                 "group_by": [["big", "attr"]], "agg": {"kind": "col", "a": "value", "b": None}}
        w = datagen.Workload(f"one hash join, {m} rows", n, fact, dims, {"big": "key"}, query)
        got, sq = run_gpu(w, force={"slice": 1})
        bits = sq.plan_obj.slice_bits
        seen.add(bits)
        assert_same(got.as_rows(), oracle_rows(w), f"{m} dimension rows, {bits} slice bits")
    assert seen == {1, 2, 3, 5, 8}, seen


def _filter_words(table):
    """The pass filter of a built hash table, copied from its workspace."""
    import torch
    from paper_2607_07632_amd import sdb
    nbytes = sdb.dim_info(table)["filter_bytes"]
    off = table.handle.filter - table.workspace.data_ptr()
    return table.workspace[off:off + nbytes].view(torch.int32).cpu().numpy().view(np.uint32)


def _bitmap_words(keys, key_min, n_bits):
    bits = np.zeros((n_bits + 31) // 32 * 32, dtype=bool)
    bits[keys.astype(np.int64) - key_min] = True
    return np.packbits(bits, bitorder="little").view(np.uint32)


def _bloom_words(keys, n_words):
    """The blocked Bloom filter the header documents, written out in numpy:
    word m mod n_words of m = mix(key) holds three bits picked by
    t = rotl(m, 16) * 0x9E3779B1."""
    m = keys.astype(np.int32).view(np.uint32).copy()
    m = (m ^ (m >> np.uint32(16))) * np.uint32(0x85EBCA6B)
    m ^= m >> np.uint32(13)
    m *= np.uint32(0xC2B2AE35)
    m ^= m >> np.uint32(16)
    t = ((m << np.uint32(16)) | (m >> np.uint32(16))) * np.uint32(0x9E3779B1)
    one = np.uint32(1)
    mask = (np.left_shift(one, t >> np.uint32(27)) | np.left_shift(one, (t >> np.uint32(22)) & np.uint32(31)) |
            np.left_shift(one, (t >> np.uint32(17)) & np.uint32(31)))
    out = np.zeros(n_words, dtype=np.uint32)
    np.bitwise_or.at(out, m & np.uint32(n_words - 1), mask)
    return out


def _one_hash_join(m, n, key_span, seed, lf=0.5):
    """One hash join over m dimension rows whose distinct keys are drawn from
    key_span values around 0 (half of the rows filtered out), n fact rows
    with 80% hits, a fact predicate, SUM(value) by one payload."""
    rng = np.random.default_rng([2607, 7632, 71, seed])
    keys = (rng.choice(key_span, m, replace=False) - key_span // 2).astype(np.int32)
    dims = {"big": {"key": keys, "flag": rng.integers(0, 2, m, dtype=np.int32),
                    "attr": rng.integers(0, 700, m, dtype=np.int32)}}
    hit = keys[rng.integers(0, m, n)]
    miss = rng.integers(-key_span // 2 - 10, key_span // 2 + 10, n).astype(np.int32)
    fact = {"key": np.where(rng.random(n) < 0.8, hit, miss).astype(np.int32),
            "value": rng.integers(-10**6, 10**6, n, dtype=np.int32)}
    query = {"fact_preds": [{"col": "value", "op": "ge", "lo": -900_000, "hi": None}],
             "joins": [{"fact_key": "key", "dim": "big", "preds": [{"col": "flag", "op": "eq", "lo": 1, "hi": None}],
                        "payloads": ["attr"], "kind": "hash", "load_factor": lf}],
             "group_by": [["big", "attr"]], "agg": {"kind": "col", "a": "value", "b": None}}
    return datagen.Workload(f"one hash join, {m} rows over {key_span} keys", n, fact, dims, {"big": "key"}, query)


def test_hash_pass_filter_words():
    """A hash table's pass filter holds exactly its passing keys: c5's table
    and a permuted key range as a bitmap over the key range (built through a
    byte per key, or with atomics where those bytes do not fit the slot
    region), keys spread over 2^31 values as the documented Bloom filter
    (word for word)."""
    from paper_2607_07632_amd import sdb
    w = workload("c5_hash_stress")
    _, dims = upload(datagen.Workload(w.name, 0, {k: v[:0] for k, v in w.fact.items()}, w.dims, w.dim_keys,
                                      w.query))
    t = sdb.build_dims(dims, w.dim_keys, w.query)[0]
    info = sdb.dim_info(t)
    assert info["kind"] == "hash" and info["filter"] == "bitmap" and info["filter_bytes"] == 2 << 20
    big = w.dims["big"]
    want = _bitmap_words(big["key"][big["flag"] == 1], info["key_min"], info["key_max"] - info["key_min"] + 1)
    assert np.array_equal(_filter_words(t), want)
    # (two rows over 1000 keys: a bitmap whose bytes do not fit the 4-slot
    # table's region, so the inserts set its bits with atomics)
    for m, span, kind in ((3000, 7000, "bitmap"), (5000, 1 << 31, "bloom"), (1, 1, "bitmap"), (2, 1000, "bitmap")):
        wj = _one_hash_join(m, 0, span, seed=m)
        _, dj = upload(wj)
        tj = sdb.build_dims(dj, wj.dim_keys, wj.query)[0]
        ij = sdb.dim_info(tj)
        assert ij["filter"] == kind, (m, span, ij)
        passing = wj.dims["big"]["key"][wj.dims["big"]["flag"] == 1]
        if kind == "bitmap":
            want = _bitmap_words(passing, ij["key_min"], ij["key_max"] - ij["key_min"] + 1)
        else:
            assert ij["filter_bytes"] == 8192                     # 8 bits per row, a power of two
            want = _bloom_words(passing, ij["filter_bytes"] // 4)
        assert np.array_equal(_filter_words(tj), want), (m, span)


@pytest.mark.parametrize("n", [1, 16_385, 300_007])
@pytest.mark.parametrize("span", [7000, 1 << 31])
def test_prefilter_agrees_with_the_oracle(n, span):
    """The sliced probe with its pre-filter (bitmap or Bloom filter) and
    without, every terminal shape and a two-column aggregate, against the
    oracle."""
    w = _one_hash_join(3000, n, span, seed=n + span)
    want = oracle_rows(w)
    for force in ({"slice": 1, "prefilter": 1}, {"slice": 1, "prefilter": 1, "terminal": "global"},
                  {"slice": 1, "prefilter": 1, "terminal": "part"}, {"slice": 1, "prefilter": -1}):
        got, q = run_gpu(w, force=force)
        assert q.plan_obj.slice_bits > 0 and q.plan_obj.slice_prefilter == (force["prefilter"] == 1)
        assert_same(got.as_rows(), want, f"{w.name}, {n} rows, {force}")
    w2 = datagen.Workload(w.name, w.n_fact, w.fact, w.dims, w.dim_keys,
                          {**w.query, "agg": {"kind": "sub", "a": "value", "b": "key"}})
    got, q = run_gpu(w2, force={"slice": 1, "prefilter": 1})
    assert q.plan_obj.slice_prefilter == 1
    assert_same(got.as_rows(), oracle_rows(w2), f"{w.name}, {n} rows, value - key")


@pytest.mark.parametrize("n", [0, 5, 16_383, 16_384, 70_001])
def test_prefilter_on_random_tiny_schemas(n):
    """Forced pre-filters over random one-join schemas (fact predicates,
    misses, filtered rows, every aggregate kind) at row counts around the
    passes' chunks: the oracle's groups, sums and counts exactly."""
    done = 0
    for seed in range(60):
        w0 = random_tiny_workload(5000 + seed, n_fact=n, max_dim_rows=3000)
        if not w0.query["joins"]:
            continue
        w = _sliceable(w0, load_factor=(0.5, 0.25, 0.9)[seed % 3], keep_agg=seed % 2 == 1)
        for force in ({"slice": 1, "prefilter": 1}, {"slice": 1, "prefilter": 1, "order": True}):
            got, q = run_gpu(w, force=force)
            assert q.plan_obj.slice_prefilter == (1 if n else 0), (seed, force)
            assert_same(got.as_rows(), oracle_rows(w), f"seed {seed} n {n} {force}")
        done += 1
        if done == 3:
            break
    assert done == 3


def test_c5_prefilter_is_the_planners_choice():
    """c5 (half of the table's rows filtered out): the planner takes the
    pre-filter; with it and without, the oracle's result."""
    w = workload("c5_hash_stress")
    want = want_rows("c5_hash_stress")
    got, q = run_gpu(w, force={"slice": 1})
    assert q.plan_obj.slice_prefilter == 1
    from paper_2607_07632_amd import sdb
    assert sdb.plan_summary(q.plan_obj, w.query)["stages"][-1].get("prefilter") is True
    assert_same(got.as_rows(), want, "c5 pre-filtered")
    got, q = run_gpu(w, force={"slice": 1, "prefilter": -1})
    assert q.plan_obj.slice_prefilter == 0
    assert_same(got.as_rows(), want, "c5 without the pre-filter")


def test_c1_forced_plans_agree():
    w = workload("c1_scalar_scan")
    want = want_rows("c1_scalar_scan")
    for force in [{"ipt": 1}, {"ipt": 2}, {"ipt": 4}, {"vector": -1}, {"order": True},
                  {"terminal": "global"}, {"terminal": "lds"}, {"grid": 3}]:
        got, _ = run_gpu(w, force=force)
        assert_same(got.as_rows(), want, f"c1 {force}")


def test_table_kinds_agree():
    w = datagen.make_workload("c2_join_group", n_fact=1_000_005)
    want = oracle_rows(w)
    for kinds in [("hash", "hash"), ("dense", "hash"), ("hash", "dense")]:
        q = dict(w.query)
        q["joins"] = [dict(j, kind=k) for j, k in zip(w.query["joins"], kinds)]
        w2 = datagen.Workload(w.name, w.n_fact, w.fact, w.dims, w.dim_keys, q)
        got, qq = run_gpu(w2)
        assert [t.kind for t in qq.tables] == list(kinds)
        assert_same(got.as_rows(), want, f"c2 {kinds}")


def test_c5_dense_and_low_load_factor_agree():
    w = datagen.make_workload("c5_hash_stress", n_fact=500_001)
    want = oracle_rows(w)
    for kind, lf in [("dense", 0.0), ("hash", 0.25), ("auto", 0.0)]:
        q = dict(w.query)
        q["joins"] = [dict(w.query["joins"][0], kind=kind, load_factor=lf)]
        w2 = datagen.Workload(w.name, w.n_fact, w.fact, w.dims, w.dim_keys, q)
        got, _ = run_gpu(w2)
        assert_same(got.as_rows(), want, f"c5 {kind} {lf}")


@pytest.mark.parametrize("block", range(6))
def test_random_tiny_schemas(block):
    for seed in range(block * 50, block * 50 + 50):
        w = random_tiny_workload(seed, max_fact=3000, max_dim_rows=400)
        want = oracle_rows(w)
        got, _ = run_gpu(w)
        assert_same(got.as_rows(), want, f"tiny seed {seed}")


@pytest.mark.parametrize("seed", [7, 19, 23])
def test_random_tiny_schemas_forced(seed):
    w = random_tiny_workload(seed + 1000, max_fact=5000, max_dim_rows=500, n_fact=4099)
    want = oracle_rows(w)
    for force in [{"vector": -1}, {"ipt": 1, "grid": 2}, {"ipt": 4}, {"order": True},
                  {"terminal": "global"}, {"terminal": "part", "ipt": 1}, {"terminal": "part", "vector": -1, "grid": 3},
                  {"eager": 4}, {"eager": 3, "ipt": 1, "terminal": "part"}, {"eager": -1},
                  {"block": 1024, "ipt": 1}, {"block": 1024, "terminal": "part", "grid": 2}, {"lds": 2},
                  {"lds": 3}, {"lds": 3, "terminal": "part", "grid": 3},
                  {"lds": -1, "terminal": "part"}, {"lds": -1, "coarse": 1}, {"lds": -1, "coarse": 3, "ipt": 1},
                  {"lds": -1, "coarse": 5, "vector": -1}, {"coarse": 2, "terminal": "part"}]:
        got, _ = run_gpu(w, force=force)
        assert_same(got.as_rows(), want, f"tiny {seed} {force}")


@pytest.mark.parametrize("n", [0, 1, 3, 4, 5, 63, 64, 65, 255, 256, 257, 1023, 1025, 4097])
def test_small_and_ragged_sizes(n):
    for name in ["c1_scalar_scan", "c3_star3", "c2_join_group"]:
        w = datagen.make_workload(name, n_fact=n, row_start=12_345)
        got, _ = run_gpu(w)
        assert_same(got.as_rows(), oracle_rows(w), f"{name} n={n}")


@pytest.mark.parametrize("offset", [1, 2, 3, 4])
def test_misaligned_columns(offset):
    w = datagen.make_workload("c3_star3", n_fact=300_007)
    want = oracle_rows(w)
    got, q = run_gpu(w, dev=upload(w, offset=offset))
    assert q.plan_obj.vector == (1 if offset % 4 == 0 else 0)
    assert_same(got.as_rows(), want, f"offset {offset}")


def test_repeat_runs_are_identical():
    w = workload("c4_star4_zipf")
    fact_dims = upload(w)
    from paper_2607_07632_amd import sdb
    tables = sdb.build_dims(fact_dims[1], w.dim_keys, w.query)
    first, q = run_gpu(w, dev=fact_dims, tables=tables)
    for _ in range(3):
        again = q.execute(replan=False)
        assert again.as_rows() == first.as_rows()


def test_two_host_threads_on_streams_of_their_own():
    """Builds, plans, runs and compactions from two host threads at once, each
    on a stream of its own: the library's per-thread state (error string,
    pinned staging) keeps them apart; every result against the oracle."""
    import threading
    import torch
    from paper_2607_07632_amd import sdb
    works = [datagen.make_workload("c3_star3", n_fact=400_003),
             datagen.make_workload("c5_hash_stress", n_fact=300_001)]
    wants = [oracle_rows(w) for w in works]
    devs = [upload(w) for w in works]
    torch.cuda.synchronize()
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            w = works[i]
            fact, dims = devs[i]
            with torch.cuda.stream(s):
                for it in range(4):
                    tables = sdb.build_dims(dims, w.dim_keys, w.query, stream=s)
                    got = sdb.StarQuery(fact, tables, w.query).execute(stream=s)
                    if got.as_rows() != wants[i]:
                        errors.append(f"thread {i}, iteration {it}: result differs from the oracle")
        except Exception as e:  # reported by the main thread
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=100)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors


def test_all_pass_and_all_fail():
    w = datagen.make_workload("c2_join_group", n_fact=200_000)
    q = dict(w.query)
    q["joins"] = [dict(w.query["joins"][0], preds=[{"col": "region", "op": "ge", "lo": -(2**40), "hi": None}]),
                  w.query["joins"][1]]
    w2 = datagen.Workload(w.name, w.n_fact, w.fact, w.dims, w.dim_keys, q)
    got, _ = run_gpu(w2)
    want = oracle_rows(w2)
    assert sum(c for _, _, c in want) == w.n_fact
    assert_same(got.as_rows(), want, "all pass")
    q["fact_preds"] = [{"col": "revenue", "op": "gt", "lo": 2**31, "hi": None}]
    w3 = datagen.Workload(w.name, w.n_fact, w.fact, w.dims, w.dim_keys, q)
    got, _ = run_gpu(w3)
    assert got.as_rows() == [] == oracle_rows(w3)


def test_extreme_literals_and_values():
    rng = np.random.default_rng(5)
    n = 70_001
    v = rng.integers(-(2**31), 2**31, size=n, dtype=np.int64).astype(np.int32)
    v[:6] = [-(2**31), 2**31 - 1, 0, -1, 1, 2**31 - 2]
    fact = {"v": v, "w": rng.integers(-(2**31), 2**31, size=n, dtype=np.int64).astype(np.int32)}
    for pred in [{"col": "v", "op": "lt", "lo": -(2**31)}, {"col": "v", "op": "le", "lo": -(2**31)},
                 {"col": "v", "op": "ge", "lo": 2**31 - 1}, {"col": "v", "op": "gt", "lo": 2**31 - 2},
                 {"col": "v", "op": "ne", "lo": 0}, {"col": "v", "op": "between", "lo": -5, "hi": 2**33},
                 {"col": "v", "op": "between", "lo": 10, "hi": -10}, {"col": "v", "op": "eq", "lo": 2**31 - 1},
                 {"col": "v", "op": "ne", "lo": -(2**35)}]:
        pred = dict(pred, hi=pred.get("hi"))
        for agg in [{"kind": "mul", "a": "v", "b": "w"}, {"kind": "sub", "a": "v", "b": "w"},
                    {"kind": "add", "a": "w", "b": "v"}]:
            q = {"fact_preds": [pred], "joins": [], "group_by": [], "agg": agg}
            w = datagen.Workload("extreme", n, fact, {}, {}, q)
            got, _ = run_gpu(w)
            assert_same(got.as_rows(), oracle_rows(w), f"{pred} {agg}")


def test_errors_are_reported():
    import torch
    from paper_2607_07632_amd import sdb
    key = torch.tensor([5, 6, 7, 6], dtype=torch.int32, device="cuda")
    a = torch.tensor([1, 2, 3, 4], dtype=torch.int32, device="cuda")
    for kind in ["dense", "hash", "auto"]:
        with pytest.raises(sdb.SdbError) as e:
            sdb.build_dim(key, {"a": a}, [], ["a"], kind)
        assert e.value.name == "SDB_DUP_KEY"
    sparse = torch.tensor([0, 10_000_000], dtype=torch.int32, device="cuda")
    b = torch.tensor([1, 2], dtype=torch.int32, device="cuda")
    with pytest.raises(sdb.SdbError) as e:
        sdb.build_dim(sparse, {"a": b}, [], [], "dense")
    assert e.value.name == "SDB_KEY_RANGE"
    t = sdb.build_dim(sparse, {"a": b}, [], [], "auto")
    assert t.kind == "hash"
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(sdb.SdbError) as e:
        sdb.build_dim(key[:3], {"a": a[:3]}, [], [], "auto", workspace=small)
    assert e.value.name == "SDB_WORKSPACE_TOO_SMALL"


def test_build_statistics_match_numpy():
    import torch
    from paper_2607_07632_amd import sdb
    w = datagen.make_workload("c4_star4_zipf", n_fact=10)
    part = w.dims["part"]
    dev = {k: torch.from_numpy(v).cuda() for k, v in part.items()}
    t = sdb.build_dim(dev["part_key"], {"category": dev["category"], "brand": dev["brand"]},
                      [{"col": "category", "op": "eq", "lo": 1, "hi": None}], ["brand"])
    ok = part["category"] == 1
    h = t.handle
    assert h.n_pass == int(ok.sum()) and h.kind == 1 and h.width == 2
    assert h.pass_key_min == part["part_key"][ok].min() and h.pass_key_max == part["part_key"][ok].max()
    assert h.payload_min[0] == part["brand"][ok].min()
    assert h.payload_radix[0] == part["brand"][ok].max() - part["brand"][ok].min() + 1
    # the map itself: the sentinel (0xFFFE) for filtered rows, brand - min otherwise
    assert h.sentinel == 0xFFFE
    torch.cuda.synchronize()
    ws = t.workspace.cpu().numpy()
    got = ws[256:256 + h.n_slots * 2].view(np.uint16)
    want = np.where(ok, part["brand"] - h.payload_min[0], 0xFFFE).astype(np.uint16)
    assert np.array_equal(got, want)
    # and its pass bitmap
    bits_off = h.bits - t.workspace.data_ptr()
    words = ws[bits_off:bits_off + (h.n_slots + 31) // 32 * 4].view(np.uint32)
    unpacked = np.unpackbits(words.view(np.uint8), bitorder="little")[:h.n_slots].astype(bool)
    assert np.array_equal(unpacked, ok)


@pytest.mark.parametrize("n,kind,npass", [(1, "dense", "some"), (4095, "dense", "some"), (4097, "hash", "some"),
                                           (10_000, "dense", "none"), (5_000_001, "dense", "some"),
                                           (5_000_001, "hash", "all")])
def test_build_statistics_over_many_blocks(n, kind, npass):
    """Key range, pass count and payload ranges from the per-block partials
    (one block per 4,096 rows, at most 1,024, so 5M rows loop) against numpy,
    with keys and payloads at the int32 extremes."""
    import torch
    from paper_2607_07632_amd import sdb
    rng = np.random.default_rng(n + len(kind))
    step = 1 if kind == "dense" else 3
    key = (rng.permutation(n).astype(np.int64) * step + np.iinfo(np.int32).min + 7).astype(np.int32)
    f = rng.integers(0, 10, n).astype(np.int32)
    a = rng.integers(-5, 41, n).astype(np.int32)
    b = rng.integers(1000, 1100, n).astype(np.int32)
    c = (np.iinfo(np.int32).min + rng.integers(0, 51, n)).astype(np.int32)
    bound = {"some": 3, "none": 0, "all": 10}[npass]
    ok = f < bound
    dev = lambda x: torch.from_numpy(x).cuda()
    t = sdb.build_dim(dev(key), {"f": dev(f), "a": dev(a), "b": dev(b), "c": dev(c)},
                      [{"col": "f", "op": "lt", "lo": bound, "hi": None}], ["a", "b", "c"], kind)
    info = sdb.dim_info(t)
    assert info["kind"] == kind
    assert info["n_rows"] == n and info["n_pass"] == int(ok.sum())
    assert (info["key_min"], info["key_max"]) == (int(key.min()), int(key.max()))
    if ok.any():
        assert (info["pass_key_min"], info["pass_key_max"]) == (int(key[ok].min()), int(key[ok].max()))
        for i, col in enumerate((a, b, c)):
            assert info["payload_min"][i] == int(col[ok].min())
            assert info["payload_max"][i] == int(col[ok].max())
            assert info["payload_radix"][i] == int(col[ok].max()) - int(col[ok].min()) + 1
    else:
        assert info["payload_radix"] == [1, 1, 1]


def _stage_masks(w, rows):
    """Pass mask of every stage (query order: predicates, then joins) on the
    given fact rows, by direct indexing (dimension keys are row numbers here)."""
    masks = []
    for p in w.query["fact_preds"]:
        masks.append(oracle.eval_pred(w.fact[p["col"]][rows], p))
    for jd in w.query["joins"]:
        t = w.dims[jd["dim"]]
        keys = t[w.dim_keys[jd["dim"]]].astype(np.int64)
        assert np.array_equal(keys, np.arange(keys.size))
        ok = np.ones(keys.size, dtype=bool)
        for p in jd["preds"]:
            ok &= oracle.eval_pred(t[p["col"]], p)
        fk = w.fact[jd["fact_key"]][rows].astype(np.int64)
        inr = (fk >= 0) & (fk < keys.size)
        masks.append(inr & ok[np.clip(fk, 0, keys.size - 1)])
    return masks


@pytest.mark.parametrize("name", ["c1_scalar_scan", "c3_star3", "c4_star4_zipf"])
def test_plan_pass_fractions_are_the_sampled_conditional_fractions(name):
    """Each stage's pass fraction in the plan is the fraction of sampled rows
    passing it among those passing every earlier stage, exactly as counted
    on the sampled rows."""
    w = workload(name)
    _, q = run_gpu(w)
    p = q.plan_obj
    n = w.n_fact
    step = (n + 65535) // 65536
    rows = np.arange(0, n, step)
    assert p.sampled_rows == rows.size
    masks = _stage_masks(w, rows)
    n_preds = len(w.query["fact_preds"])
    live = np.ones(rows.size, dtype=bool)
    for s in range(p.n_stages):
        m = masks[p.stage_index[s] + (n_preds if p.stage_kind[s] == 1 else 0)]
        assert abs(p.stage_pass_alone[s] - m.mean()) < 1e-12
        want = (live & m).sum() / live.sum() if live.sum() else None
        if want is not None:
            assert abs(p.stage_pass[s] - want) < 1e-12, (s, p.stage_pass[s], want)
        live &= m


def test_correlated_predicates_are_priced_jointly():
    """Two predicates on one column that each pass most rows but jointly few
    (qty < 30 and qty >= 28): the plan's second stage passes about 2/29 of the
    rows the first leaves, not the marginal product; results are exact."""
    w0 = workload("c1_scalar_scan")
    q = {**w0.query, "fact_preds": [{"col": "qty", "op": "lt", "lo": 30, "hi": None},
                                    {"col": "qty", "op": "ge", "lo": 28, "hi": None},
                                    {"col": "disc", "op": "between", "lo": 2, "hi": 4}]}
    w = datagen.Workload("c1 correlated", w0.n_fact, w0.fact, w0.dims, w0.dim_keys, q)
    got, sq = run_gpu(w)
    p = sq.plan_obj
    f = 1.0
    for s in range(p.n_stages):
        f *= p.stage_pass[s]
    qty = w.fact["qty"]
    live = ((qty < 30) & (qty >= 28) & (w.fact["disc"] >= 2) & (w.fact["disc"] <= 4) &
            (w.dims["date"]["year"][w.fact["date_key"]] == 1994))
    assert abs(f - live.mean()) < 0.002                   # joint estimate within sampling error
    alone = 1.0
    for s in range(p.n_stages):
        alone *= p.stage_pass_alone[s]
    assert alone > 3 * f                                  # the independence estimate would be far off
    assert_same(got.as_rows(), oracle_rows(w), "correlated predicates")


def _sparse_key_workload(seed=7, m=100_000, spread=7, n=400_003):
    """One dimension whose m keys spread over spread * m values (beyond the
    dense key-range limit of 2m), fact keys mostly hits, some misses."""
    rng = np.random.default_rng(seed)
    keys = (spread * rng.permutation(m) + 13).astype(np.int32)
    dim = {"k": keys, "region": rng.integers(0, 5, m).astype(np.int32),
           "attr": rng.integers(0, 200, m).astype(np.int32)}
    hit = keys[rng.integers(0, m, n)]
    miss = rng.integers(0, spread * m + 30, n).astype(np.int32)
    fact = {"fk": np.where(rng.random(n) < 0.9, hit, miss).astype(np.int32),
            "v": rng.integers(-1000, 1_000_000, n).astype(np.int32)}
    q = {"fact_preds": [], "joins": [{"fact_key": "fk", "dim": "d", "preds": [{"col": "region", "op": "eq",
                                                                               "lo": 2, "hi": None}],
                                      "payloads": ["attr"], "kind": "auto"}],
         "group_by": [["d", "attr"]], "agg": {"kind": "col", "a": "v", "b": None}}
    return datagen.Workload("sparse keys", n, fact, {"d": dim}, {"d": "k"}, q)


def test_dense_table_within_a_memory_budget():
    """Keys spread over 7x the rows: the key-range rule alone builds a hash
    table; a memory budget that holds the dense table (700,000 one-byte slots
    and the pass bitmap) builds it dense instead; a smaller budget does not;
    DENSE forced beyond both limits is refused. Every result equals the oracle."""
    from paper_2607_07632_amd import sdb
    w = _sparse_key_workload()
    want = oracle_rows(w)
    fact, dims = upload(w)
    for budget, kind in [(0, "hash"), (1 << 20, "dense"), (600_000, "hash")]:
        w.query["joins"][0]["dense_budget_bytes"] = budget
        tables = sdb.build_dims(dims, w.dim_keys, w.query)
        assert tables[0].kind == kind, (budget, tables[0].kind)
        info = sdb.dim_info(tables[0])
        if kind == "dense":
            assert info["n_slots"] == 7 * 99_999 + 1 and info["table_bytes"] <= budget
        got = sdb.StarQuery(fact, tables, w.query).execute()
        assert_same(got.as_rows(), want, f"budget {budget}")
    w.query["joins"][0]["kind"] = "dense"
    w.query["joins"][0]["dense_budget_bytes"] = 600_000
    with pytest.raises(sdb.SdbError) as e:
        sdb.build_dims(dims, w.dim_keys, w.query)
    assert e.value.name == "SDB_KEY_RANGE"


def _sorted_by(w, col):
    """The workload with its fact rows reordered by one column (the result of
    the query does not depend on row order)."""
    order = np.argsort(w.fact[col], kind="stable")
    fact = {k: np.ascontiguousarray(v[order]) for k, v in w.fact.items()}
    return datagen.Workload(f"{w.name} sorted by {col}", w.n_fact, fact, w.dims, w.dim_keys, w.query)


_SEGMENT_FORCES = [{"segments": 1}, {"segments": 1, "terminal": "global"}, {"segments": 1, "terminal": "part"},
                   {"segments": 1, "terminal": "part", "grid": 7}, {"segments": 1, "ipt": 1},
                   {"segments": 1, "vector": -1}, {"segments": 1, "terminal": "global", "xcd": 1},
                   {"segments": 1, "block": 1024}, {"segments": 1, "unroll": -1}, {"segments": 1, "lds": -1}]


@pytest.mark.parametrize("force", _SEGMENT_FORCES)
def test_segmented_plans_on_date_sorted_rows(force):
    """c3's rows sorted by date: the rows of 1998 and 1999 fail the date filter,
    so the planner gives their row range an order that tests the date first;
    each segment is its own launch into one terminal. The result equals c3's."""
    w = _sorted_by(workload("c3_star3"), "date_key")
    got, q = run_gpu(w, force=force)
    p = q.plan_obj
    assert p.n_segments >= 2, force
    assert p.segment_start[0] == 0 and p.segment_start[p.n_segments] == w.n_fact
    date = next(s for s in range(p.n_stages) if p.stage_kind[s] == 1 and w.query["joins"][p.stage_index[s]]["dim"]
                == "date")
    assert p.segment_order[p.n_segments - 1][0] == date          # the last rows test the date first
    assert_same(got.as_rows(), want_rows("c3_star3"), f"date-sorted {force}")


@pytest.mark.parametrize("name", ["c1_scalar_scan", "c2_join_group", "c4_star4_zipf"])
def test_segmented_plans_other_terminals(name):
    """Segments on date-sorted rows of the scalar (c1), LDS (c2) and global
    (c4) terminals, and no segments when they are turned off."""
    w = _sorted_by(workload(name), "date_key")
    got, q = run_gpu(w, force={"segments": 1})
    assert_same(got.as_rows(), want_rows(name), f"{name} date-sorted, segments")
    off, q2 = run_gpu(w, force={"segments": -1})
    assert q2.plan_obj.n_segments == 1
    assert_same(off.as_rows(), want_rows(name), f"{name} date-sorted, one order")


_WINDOW_FORCES = [{"window": 1}, {"window": 7}, {"window": 64, "terminal": "part"},
                  {"window": 1, "terminal": "global"}, {"window": 2, "ipt": 1}, {"window": 1, "vector": -1},
                  {"window": 300, "eager": 2}, {"window": 1, "lds": 3}, {"window": 1, "unroll": -1},
                  {"window": 1, "block": 512}, {"window": 9, "order": True}]


@pytest.mark.parametrize("name", ["c3_star3", "c4_star4_zipf"])
@pytest.mark.parametrize("force", _WINDOW_FORCES)
def test_lds_window_plans_agree(name, force):
    """LDS windows over the device-memory dense tables (c3's customer map, c4's
    part and customer maps): rows inside and outside the window, deferred
    codes, every terminal and item shape, against the oracle."""
    w = workload(name)
    got, q = run_gpu(w, force=force)
    windows = [s for s in range(q.plan_obj.n_stages) if q.plan_obj.stage_lds[s] == 5]
    assert len(windows) == 1, f"{name} {force}: no window placed"
    assert_same(got.as_rows(), want_rows(name), f"{name} {force}")


def test_lds_window_follows_the_sampled_keys():
    """Fact keys concentrated in the upper third of the customer key range:
    the sampled key histogram moves the window there; results stay exact."""
    w0 = workload("c3_star3")
    fact = dict(w0.fact)
    fact["cust_key"] = (2_000_000 + w0.fact["cust_key"] % 1_000_000).astype(np.int32)
    w = datagen.Workload("c3 keys in the upper third", w0.n_fact, fact, w0.dims, w0.dim_keys, w0.query)
    got, q = run_gpu(w, force={"window": 1})
    p = q.plan_obj
    s = next(s for s in range(p.n_stages) if p.stage_lds[s] == 5)
    lo, slots = p.stage_window_lo[s], p.stage_window_slots[s]
    assert lo < 3_000_000 and lo + slots > 2_000_000
    assert p.stage_window_cover[s] >= min(1.0, slots / 1_000_000) - 0.02
    assert_same(got.as_rows(), oracle_rows(w), "keys in the upper third")


@pytest.mark.parametrize("seed", range(8))
def test_lds_window_on_random_schemas(seed):
    """Random schemas with dimensions large enough that their pass bitmaps are
    not staged whole: windows of several sizes, against the oracle."""
    w = random_tiny_workload(seed + 5000, max_fact=60_000, max_dim_rows=400_000, n_fact=50_003)
    want = oracle_rows(w)
    for win in (1, 3, 40):
        got, _ = run_gpu(w, force={"window": win})
        assert_same(got.as_rows(), want, f"seed {seed} window {win}")


@pytest.mark.parametrize("name", ["c3_star3", "c4_star4_zipf", "c5_hash_stress", "c1_scalar_scan"])
def test_dim_info_of_built_tables(name):
    """sdb_dim_info through the ABI against numpy over the dimension columns."""
    import torch
    from paper_2607_07632_amd import sdb
    w = datagen.make_workload(name, n_fact=10)
    dev = {d: {c: torch.from_numpy(a).cuda() for c, a in t.items()} for d, t in w.dims.items()}
    tables = sdb.build_dims(dev, w.dim_keys, w.query)
    for jd, tab in zip(w.query["joins"], tables):
        t = w.dims[jd["dim"]]
        keys = t[w.dim_keys[jd["dim"]]].astype(np.int64)
        ok = np.ones(keys.size, dtype=bool)
        for p in jd["preds"]:
            ok &= oracle.eval_pred(t[p["col"]], p)
        info = sdb.dim_info(tab)
        assert info["n_rows"] == keys.size and info["n_pass"] == int(ok.sum())
        assert (info["key_min"], info["key_max"]) == (keys.min(), keys.max())
        assert (info["pass_key_min"], info["pass_key_max"]) == (keys[ok].min(), keys[ok].max())
        assert info["pass_keys_contiguous"] == (keys[ok].max() - keys[ok].min() + 1 == ok.sum())
        for i, col in enumerate(jd["payloads"]):
            assert info["payload_min"][i] == t[col][ok].min() and info["payload_max"][i] == t[col][ok].max()
        assert info["domain"] == int(np.prod([t[c][ok].max() - t[c][ok].min() + 1 for c in jd["payloads"]]))
        if jd.get("kind") == "hash":
            assert info["kind"] == "hash" and info["n_slots"] == 1 << 25 and info["table_bytes"] == 1 << 28
            assert info["occupancy"] == 0.5
        else:
            assert info["kind"] == "dense" and info["n_slots"] == keys.max() - keys.min() + 1
            assert info["table_bytes"] <= tab.workspace.numel() - 256
            assert info["width"] == (1 if info["domain"] <= 0xFE else 2 if info["domain"] <= 0xFFFE else 4)


def test_binding_rejects_unreadable_device_columns():
    """Device tensors the library cannot read as dense int32 arrays are refused
    by the binding with a ValueError before any launch."""
    import torch
    from paper_2607_07632_amd import sdb
    key = torch.arange(100, dtype=torch.int32, device="cuda")
    good = torch.zeros(100, dtype=torch.int32, device="cuda")
    for bad, msg in [(torch.zeros(200, dtype=torch.int32, device="cuda")[::2], "contiguous"),
                     (torch.zeros(100, 2, dtype=torch.int32, device="cuda")[:, 1], "contiguous"),
                     (torch.zeros(100, dtype=torch.int64, device="cuda"), "int32"),
                     (good.cpu(), "GPU"), (good[:99], "elements")]:
        with pytest.raises(ValueError, match=msg):
            sdb.build_dim(key, {"a": bad}, [], ["a"])
        q = {"fact_preds": [], "joins": [], "group_by": [], "agg": {"kind": "add", "a": "x", "b": "y"}}
        with pytest.raises(ValueError, match=msg):
            sdb.StarQuery({"x": good, "y": bad}, [], q)
    q = {"fact_preds": [], "joins": [], "group_by": [], "agg": {"kind": "col", "a": "x", "b": None}}
    sq = sdb.StarQuery({"x": good}, [], q)
    plan = sq.plan()
    sums, counts = sq.alloc_outputs(plan)
    with pytest.raises(ValueError, match="int64"):
        sq.run(sums.int(), counts, plan=plan)
    with pytest.raises(ValueError, match="elements"):
        sq.run(sums, torch.zeros(2, dtype=torch.int64, device="cuda"), plan=plan)


@pytest.mark.parametrize("name", ["c2_join_group", "c3_star3", "c4_star4_zipf", "c5_hash_stress", "c1_scalar_scan"])
def test_partitioned_terminal(name):
    w = workload(name)
    want = want_rows(name)
    got, q = run_gpu(w, force={"terminal": "part"})
    assert q.plan_obj.terminal == 4
    assert_same(got.as_rows(), want, f"{name} part")


@pytest.mark.parametrize("cap", [64, 1024])
def test_partitioned_terminal_region_overflow(cap):
    """Records that do not fit a block's region go straight to the group table."""
    from paper_2607_07632_amd import sdb
    w = workload("c3_star3")
    fact, dims = upload(w)
    tables = sdb.build_dims(dims, w.dim_keys, w.query)
    q = sdb.StarQuery(fact, tables, w.query, {"terminal": "part"})
    plan = q.plan()
    plan.part_cap = cap
    plan.run_scratch_bytes = 0          # recomputed below from the smaller regions
    sums, counts = q.alloc_outputs(plan)
    import torch
    scratch = torch.empty(1 << 26, dtype=torch.uint8, device="cuda")
    q.run(sums, counts, plan=plan, scratch=scratch)
    k, s, c, n, _ = q.finalize(sums, counts, plan=plan)
    torch.cuda.synchronize()
    m = int(n.item())
    rows = [(tuple(int(x) for x in kk), int(ss), int(cc))
            for kk, ss, cc in zip(k[:m].cpu().numpy(), s[:m].cpu().numpy(), c[:m].cpu().numpy())]
    assert_same(rows, want_rows("c3_star3"), f"overflow cap {cap}")


@pytest.mark.parametrize("groups", [1, 3])
@pytest.mark.parametrize("values", ["max", "min", "mixed"])
def test_partitioned_sums_at_the_int32_limits(values, groups):
    """All records in one group (or three), values at the int32 limits: each
    aggregation work item sums one group to about 2^47 in magnitude, and the
    partition's several work items are merged; the sums and counts stay
    exact."""
    rng = np.random.default_rng([2607, 7632, 83])
    n = 200_003
    vals = {"max": np.full(n, 2**31 - 1, np.int32), "min": np.full(n, -2**31, np.int32),
            "mixed": np.where(rng.random(n) < 0.5, 2**31 - 1, -2**31).astype(np.int32)}[values]
    g = np.zeros(4, np.int32) if groups == 1 else np.array([0, 0, 1, 2], np.int32)
    dims = {"d": {"k": np.arange(4, dtype=np.int32), "g": g}}
    fact = {"fk": rng.choice(np.array([0, 0, 0, 1, 2, 3], np.int32), n), "v": vals}
    query = {"fact_preds": [], "joins": [{"fact_key": "fk", "dim": "d", "preds": [], "payloads": ["g"]}],
             "group_by": [["d", "g"]], "agg": {"kind": "col", "a": "v", "b": None}}
    w = datagen.Workload(f"int32 limits {values}", n, fact, dims, {"d": "k"}, query)
    got, q = run_gpu(w, force={"terminal": "part"})
    assert q.plan_obj.terminal == 4
    assert_same(got.as_rows(), oracle_rows(w), f"int32 limits {values}, {groups} groups")


@pytest.mark.parametrize("seed", [3, 11, 29, 41])
def test_random_tiny_schemas_partitioned(seed):
    w = random_tiny_workload(seed + 2000, max_fact=6000, max_dim_rows=500, n_fact=5003)
    want = oracle_rows(w)
    got, _ = run_gpu(w, force={"terminal": "part"})
    assert_same(got.as_rows(), want, f"tiny {seed} part")


def test_batched_build_matches_single_builds():
    """sdb_build_dims gives every table exactly what sdb_build_dim gives it."""
    from paper_2607_07632_amd import sdb
    import torch
    w = workload("c4_star4_zipf")
    _, dims = upload(w)
    batch = sdb.build_dims(dims, w.dim_keys, w.query)
    torch.cuda.synchronize()
    for jd, b in zip(w.query["joins"], batch):
        args = sdb._join_inputs(dims, w.dim_keys, jd)
        one = sdb.build_dim(*args)
        torch.cuda.synchronize()
        for f, _ in sdb.SdbDim._fields_:
            if f in ("stats", "map", "bits"):
                continue
            a, c = getattr(b.handle, f), getattr(one.handle, f)
            if hasattr(a, "__len__"):
                a, c = list(a), list(c)
            assert a == c, (jd["dim"], f, a, c)
        n = min(b.workspace.numel(), one.workspace.numel())
        used = 256 + (b.handle.n_slots * b.handle.width + 255) // 256 * 256 + (b.handle.n_slots + 31) // 32 * 4
        n = min(n, used)
        assert torch.equal(b.workspace[256:n], one.workspace[256:n]), jd["dim"]


def test_batched_build_reports_failing_dimension():
    from paper_2607_07632_amd import sdb
    import torch
    w = workload("c3_star3")
    _, dims = upload(w)
    bad = {d: dict(t) for d, t in dims.items()}
    key = w.dim_keys["supplier"]
    k = bad["supplier"][key].clone()
    k[5] = k[6]
    bad["supplier"][key] = k
    with pytest.raises(sdb.SdbError) as e:
        sdb.build_dims(bad, w.dim_keys, w.query)
    idx = [j["dim"] for j in w.query["joins"]].index("supplier")
    assert "DUP_KEY" in str(e.value) and f"dimension {idx}" in str(e.value)


def test_fused_events_bracket_the_kernel():
    """The library's events time the fused kernel alone: within the run window."""
    from paper_2607_07632_amd import sdb
    import torch
    w = workload("c3_star3")
    fact, dims = upload(w)
    q = sdb.StarQuery(fact, sdb.build_dims(dims, w.dim_keys, w.query), w.query, {"terminal": "part"})
    plan = q.plan()
    sums, counts = q.alloc_outputs(plan)
    scratch = q.run_scratch(plan)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    sdb.set_fused_events(ev[0], ev[1])
    ev[2].record()
    q.run(sums, counts, plan=plan, scratch=scratch)
    ev[3].record()
    sdb.set_fused_events()
    torch.cuda.synchronize()
    fused, whole = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    assert 0.0 < fused < whole
    k, s, c, n, _ = q.finalize(sums, counts, plan=plan)
    m = int(n.item())
    rows = [(tuple(int(x) for x in kk), int(ss), int(cc))
            for kk, ss, cc in zip(k[:m].cpu().numpy(), s[:m].cpu().numpy(), c[:m].cpu().numpy())]
    assert_same(rows, want_rows("c3_star3"), "timed run")


def _range_workload(seed, n=50_003, empty_join=False):
    """Dimensions whose passing keys are one contiguous range (a day-to-year
    style attribute, a predicate on the key itself, on a dense and on a hash
    table, with fact keys partly outside the key set) next to a grouped one."""
    rng = np.random.default_rng([2607, 7632, 77, seed])
    dims, keys, joins, fact = {}, {}, [], {}
    m = 700
    off = int(rng.integers(-500, 500))
    r_key = (rng.permutation(m) + off).astype(np.int32)
    dims["r"] = {"k": r_key, "y": ((r_key - off) // 50).astype(np.int32)}
    joins.append({"fact_key": "fr", "dim": "r", "preds": [{"col": "y", "op": "eq", "lo": 3, "hi": None}],
                  "payloads": []})
    g_key = rng.permutation(300).astype(np.int32)
    dims["g"] = {"k": g_key, "a": rng.integers(0, 20, size=300, dtype=np.int32)}
    joins.append({"fact_key": "fg", "dim": "g", "preds": [], "payloads": ["a"]})
    h_key = (rng.permutation(900) * 3 + 11).astype(np.int32)      # keys 3 apart: hash table
    h_sorted = np.sort(h_key)
    dims["h"] = {"k": h_key}
    joins.append({"fact_key": "fh", "dim": "h", "kind": "hash",
                  "preds": [{"col": "k", "op": "between", "lo": int(h_sorted[100]), "hi": int(h_sorted[100])}],
                  "payloads": []})
    if empty_join:
        dims["e"] = {"k": np.arange(50, dtype=np.int32), "y": np.zeros(50, dtype=np.int32)}
        joins.append({"fact_key": "fe", "dim": "e", "preds": [{"col": "y", "op": "eq", "lo": 1, "hi": None}],
                      "payloads": []})
        fact["fe"] = rng.integers(0, 50, size=n, dtype=np.int32)
    fact["fr"] = rng.integers(off - 30, off + m + 30, size=n, dtype=np.int32)
    fact["fg"] = rng.integers(0, 300, size=n, dtype=np.int32)
    fact["fh"] = np.where(rng.random(n) < 0.5, h_sorted[100], h_key[rng.integers(0, 900, size=n)]).astype(np.int32)
    fact["v"] = rng.integers(-1000, 1000, size=n, dtype=np.int32)
    for name in dims:
        keys[name] = "k"
    query = {"fact_preds": [], "joins": joins, "group_by": [["g", "a"]], "agg": {"kind": "col", "a": "v", "b": None}}
    return datagen.Workload(f"range{seed}", n, fact, dims, keys, query)


@pytest.mark.parametrize("seed", [1, 2])
def test_key_range_probes(seed):
    from paper_2607_07632_amd import sdb
    w = _range_workload(seed)
    want = oracle_rows(w)
    assert want, "the workload should keep some groups"

    def tables_of(q, query):
        return {st["name"]: st["table"] for st in sdb.plan_summary(q.plan_obj, query)["stages"]}

    got, q = run_gpu(w)                      # automatic: only the device-memory probe
    t = tables_of(q, w.query)
    assert t["h"] == "key_range" and t["r"] == "lds_map" and t["g"] != "key_range"
    assert_same(got.as_rows(), want, f"range {seed}")
    for force in [{"range": 1}, {"range": -1}, {"range": 1, "terminal": "global"}, {"range": 1, "vector": -1},
                  {"range": 1, "order": True}, {"range": 1, "lds": -1}]:
        got, q = run_gpu(w, force=force)
        assert_same(got.as_rows(), want, f"range {seed} {force}")
        t = tables_of(q, w.query)
        if force["range"] == 1:
            assert t["r"] == "key_range" and t["h"] == "key_range"
        else:
            assert "key_range" not in t.values()
    w0 = _range_workload(seed, empty_join=True)
    got, q = run_gpu(w0, force={"range": 1})
    assert got.as_rows() == oracle_rows(w0) == []
    assert tables_of(q, w0.query)["e"] == "key_range"


def test_c1_date_join_as_key_range():
    from paper_2607_07632_amd import sdb
    w = workload("c1_scalar_scan")
    for force, table in [({}, "lds_map"), ({"range": 1}, "key_range")]:
        got, q = run_gpu(w, force=force)
        tables = {st["name"]: st.get("table") for st in sdb.plan_summary(q.plan_obj, w.query)["stages"]}
        assert tables["date"] == table
        assert_same(got.as_rows(), want_rows("c1_scalar_scan"), f"c1 {force}")


@pytest.mark.parametrize("n_cols", [1, 3, 4, 5, 9])
def test_read_columns_sums_every_value(n_cols):
    import torch
    from paper_2607_07632_amd import sdb
    rng = np.random.default_rng([2607, 7632, 88, n_cols])
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    for n in [0, 1, 5, 4097, 1_000_003]:
        host = [rng.integers(-2**31, 2**31, size=n, dtype=np.int64).astype(np.int32) for _ in range(n_cols)]
        dev = [torch.from_numpy(h).cuda() for h in host]
        want = sum(int(h.astype(np.int64).sum()) for h in host)
        want = (want + 2**63) % 2**64 - 2**63
        for per_cu in (0, 1, 4):
            sdb.read_columns(dev, out, blocks_per_cu=per_cu)
            torch.cuda.synchronize()
            assert int(out.item()) == want, (n_cols, n, per_cu)


@pytest.mark.parametrize("name,force", [(n, None) for n in SIZES] + [("c5_hash_stress", {"slice": 1})])
def test_graph_replay_of_run_and_finalize(name, force):
    """The run and the compaction enqueue only kernels (no memset, copy or
    synchronization), so they can be captured in a HIP graph: every replay,
    with eager work scribbling over the outputs in between, must give the
    eager result, which must equal the oracle's."""
    import torch
    from paper_2607_07632_amd import sdb
    w = workload(name)
    fact, dims = upload(w)
    q = sdb.StarQuery(fact, sdb.build_dims(dims, w.dim_keys, w.query), w.query, force)
    plan = q.plan()
    assert bool(plan.slice_bits) == bool(force)
    sums, counts = q.alloc_outputs(plan)
    scratch = q.run_scratch(plan)
    outs = q.finalize(sums, counts, plan=plan)
    q.run(sums, counts, plan=plan, scratch=scratch)
    q.finalize(sums, counts, plan=plan, outputs=outs)
    torch.cuda.synchronize()
    m = int(outs[3].item())
    want = [t[:m].clone() for t in outs[:3]]
    got_rows = sdb.QueryResult(want[0][:, :q.n_keys].long().cpu().numpy().reshape(m, q.n_keys),
                               want[1].cpu().numpy(), want[2].cpu().numpy()).as_rows()
    assert_same(got_rows, want_rows(name), f"{name} eager")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        q.run(sums, counts, plan=plan, scratch=scratch)
        q.finalize(sums, counts, plan=plan, outputs=outs)
    torch.cuda.synchronize()
    for rep in range(3):
        sums.fill_(-1)
        counts.fill_(7)
        outs[1].zero_()
        outs[3].fill_(-5)
        outs[4].fill_(0xCD)
        if scratch is not None:
            scratch.fill_(0xAB)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(outs[3].item()) == m, (name, rep)
        for a, b in zip(outs[:3], want):
            assert torch.equal(a[:m], b), (name, rep)


def test_concurrent_queries_on_two_streams():
    """Two different queries, and two copies of one, in flight at once on
    separate streams with their own outputs and scratch: the library keeps no
    device state between calls, so every result must equal the oracle's."""
    import torch
    from paper_2607_07632_amd import sdb
    runs = []
    for name in ["c2_join_group", "c3_star3", "c3_star3", "c4_star4_zipf"]:
        w = workload(name)
        fact, dims = upload(w)
        q = sdb.StarQuery(fact, sdb.build_dims(dims, w.dim_keys, w.query), w.query)
        plan = q.plan()
        sums, counts = q.alloc_outputs(plan)
        runs.append((name, w, q, plan, sums, counts, q.run_scratch(plan), torch.cuda.Stream()))
    torch.cuda.synchronize()
    outs = []
    for rep in range(3):                      # interleaved launches, no synchronization between
        for name, w, q, plan, sums, counts, scratch, st in runs:
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                q.run(sums, counts, plan=plan, scratch=scratch, stream=st)
    for name, w, q, plan, sums, counts, scratch, st in runs:
        with torch.cuda.stream(st):
            k, s, c, n, _ = q.finalize(sums, counts, plan=plan, stream=st)
        outs.append((name, w, q, k, s, c, n, st))
    torch.cuda.synchronize()
    for name, w, q, k, s, c, n, st in outs:
        m = int(n.item())
        rows = sdb.QueryResult(k[:m, :q.n_keys].long().cpu().numpy().reshape(m, q.n_keys),
                               s[:m].cpu().numpy(), c[:m].cpu().numpy()).as_rows()
        assert_same(rows, oracle_rows(w), f"{name} concurrent")


@pytest.mark.parametrize("shift", [1, 2, 3, 4, 5])
def test_coarse_prefilter_tables(shift):
    """Every dense table in device memory behind a coarse LDS bitmap of 2^shift
    slots per bit, on random tiny schemas with gapped, offset keys and on c3."""
    from paper_2607_07632_amd import sdb
    for seed in (3, 8, 13, 21):
        w = random_tiny_workload(seed + 2000, max_fact=6000, max_dim_rows=700, n_fact=5003)
        for jd in w.query["joins"]:
            jd["kind"] = "auto"                  # dense wherever the key range allows it
        got, q = run_gpu(w, force={"lds": -1, "coarse": shift})
        assert_same(got.as_rows(), oracle_rows(w), f"tiny {seed} coarse {shift}")
    w = workload("c3_star3")
    # supplier as a plain LDS bitmap (not rank tables), so that the customer
    # map's coarse bitmap fits LDS from 4 slots per bit on
    got, q = run_gpu(w, force={"coarse": shift, "block": 1024, "lds": 2})
    stages = sdb.plan_summary(q.plan_obj, w.query)["stages"]
    assert any(st.get("table") == "lds_coarse" for st in stages) or shift == 1
    assert_same(got.as_rows(), oracle_rows(w), f"c3 coarse {shift}")


@pytest.mark.parametrize("seed", range(6))
def test_random_override_combinations(seed):
    """Planner overrides drawn at random (seeded) in combination on random tiny
    schemas: every plan the planner accepts must give the oracle's result;
    combinations it refuses must be refused with a status, not run."""
    from paper_2607_07632_amd import sdb
    rng = np.random.default_rng([2607, 7632, 55, seed])
    choices = {
        "terminal": ["auto", "scalar", "lds", "global", "part"], "ipt": [0, 1, 2, 4], "vector": [0, 1, -1],
        "order": [False, True], "grid": [0, 0, 1, 3, 17], "lds": [-1, 0, 2, 3], "xcd": [-1, 0, 1],
        "eager": [-1, 0, 1, 2, 4], "block": [0, 64, 128, 256, 512, 1024], "range": [-1, 0, 1],
        "coarse": [-1, 0, 1, 2, 5], "slice": [-1, 0, 1], "prefilter": [-1, 0, 1], "segments": [-1, 0, 1],
        "unroll": [-1, 0], "window": [-1, 0, 1, 3],
    }
    refused = ran = 0
    for case in range(4):
        w = random_tiny_workload(int(rng.integers(0, 10**6)), max_fact=5000, max_dim_rows=600,
                                 n_fact=int(rng.integers(0, 5000)))
        want = oracle_rows(w)
        fact, dims = upload(w)
        tables = sdb.build_dims(dims, w.dim_keys, w.query)
        for _ in range(10):
            force = {k: v[int(rng.integers(0, len(v)))] for k, v in choices.items()}
            try:
                got, _ = run_gpu(w, force=force, dev=(fact, dims), tables=tables)
            except sdb.SdbError as e:
                assert e.name in ("SDB_INVALID_ARG", "SDB_CAPACITY", "SDB_UNSUPPORTED"), (force, str(e))
                refused += 1
                continue
            assert_same(got.as_rows(), want, f"seed {seed} case {case} {force}")
            ran += 1
    assert ran > 0
