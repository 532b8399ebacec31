"""GPU parity at the full workload sizes (60M and 600M fact rows), in the
launch configuration the benchmark times, against the oracle itself.

* Every group of the full-size result against the oracle run over the whole
  fact table: the unmodified oracle on row ranges of about 33M rows, on worker
  processes that regenerate their rows from the seeded generator, merged group
  by group modulo 2**64 (the row-range additivity the oracle pins check). The
  workers also return the 64-bit sum of every fact column of their rows, which
  must equal the sums of the device columns the GPU read.
* The oracle on a window of the same device columns starting at an unaligned
  row (the kernel's 1-row item path).
* Row-range additivity on the GPU: three unaligned slices of the full columns
  add up to the full result.
"""

import time

import numpy as np
import pytest

import datagen
from datagen.star import CHUNK
from gpu_util import assert_same, oracle_rows, require_gpu
from oracle import ranges

pytestmark = pytest.mark.gpu

TASK_ROWS = 8 * CHUNK


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


@pytest.fixture(scope="module")
def oracle_pool():
    # workers fork from the fork server the test session started before any GPU call
    with ranges.pool(ranges.worker_count()) as ex:
        yield ex


def _log(*a):
    print(*a, flush=True)


def _run(fact_dev, dims_dev, w, lo=None, hi=None):
    from paper_2607_07632_amd import sdb
    import torch
    cols = fact_dev if lo is None else {k: v[lo:hi] for k, v in fact_dev.items()}
    tables = sdb.build_dims(dims_dev, w.dim_keys, w.query)
    q = sdb.StarQuery(cols, tables, w.query)
    res = q.execute()
    torch.cuda.synchronize()
    return res, q


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name", ["c2_join_group", "c3_star3", "c4_star4_zipf", "c5_hash_stress"])
def test_full_size(name, oracle_pool):
    import torch
    t0 = time.time()
    w = datagen.make_workload(name)
    _log(f"{name}: generated {w.n_fact} rows in {time.time() - t0:.1f} s")
    fact_dev = {k: torch.from_numpy(v).cuda() for k, v in w.fact.items()}
    dims_dev = {d: {c: torch.from_numpy(a).cuda() for c, a in t.items()} for d, t in w.dims.items()}
    torch.cuda.synchronize()
    full, q = _run(fact_dev, dims_dev, w)
    from paper_2607_07632_amd import sdb
    _log(f"{name}: GPU {len(full.sums)} groups; plan {sdb.plan_summary(q.plan_obj, w.query)}")

    # 1. every group against the oracle over the whole fact table
    t0 = time.time()
    want, col_sums = ranges.run(name, w.n_fact, oracle_pool, TASK_ROWS, log=_log)
    _log(f"{name}: oracle over all {w.n_fact} rows in {time.time() - t0:.1f} s "
         f"({len(want.sums)} groups, {want.n_live} live rows)")
    dev_sums = {k: int(v.sum(dtype=torch.int64).item()) for k, v in fact_dev.items()}
    assert col_sums == dev_sums, "the oracle's workers saw other rows than the device holds"
    assert_same(full.as_rows(), want.as_rows(), f"{name} full size")
    _log(f"{name}: full-size result equals the oracle, group by group")

    # 2. the oracle on an unaligned window of the same device columns
    lo, hi = 123_457, 123_457 + 3_000_001
    part, _ = _run(fact_dev, dims_dev, w, lo, hi)
    sample = {k: v[lo:hi] for k, v in w.fact.items()}
    win = datagen.Workload(w.name, hi - lo, sample, w.dims, w.dim_keys, w.query)
    assert_same(part.as_rows(), oracle_rows(win), f"{name} oracle window")
    _log(f"{name}: oracle window of {hi - lo} rows agrees")

    # 3. unaligned row ranges add up to the full result
    cuts = [0, w.n_fact // 3 - 1, 2 * (w.n_fact // 3) + 2, w.n_fact]
    acc = {}
    for a, b in zip(cuts[:-1], cuts[1:]):
        r, _ = _run(fact_dev, dims_dev, w, a, b)
        for k, s, c in r.as_rows():
            s0, c0 = acc.get(k, (0, 0))
            acc[k] = ((s0 + s) % (1 << 64), c0 + c)
    merged = sorted((k, s - (1 << 64) if s >= 1 << 63 else s, c) for k, (s, c) in acc.items())
    assert merged == full.as_rows()
    _log(f"{name}: row ranges add up")
    del fact_dev
    torch.cuda.empty_cache()


@pytest.mark.timeout(1200)
def test_more_than_2g_rows(oracle_pool):
    """c3's query over 2^31 + 4,099 fact rows from the same seeded generator:
    64-bit row indexing end to end. Every group against the oracle over all
    rows (row ranges on the worker pool, merged), and two row ranges, the
    second starting at an unaligned row (1-row items), add up to the whole."""
    import torch
    from paper_2607_07632_amd import sdb
    n = 2**31 + 4099
    t0 = time.time()
    w = datagen.make_workload("c3_star3", n_fact=n)
    _log(f"2g rows: generated {n} rows in {time.time() - t0:.1f} s")
    fact = {}
    for k in list(w.fact):
        fact[k] = torch.from_numpy(w.fact[k]).cuda()
        del w.fact[k]                      # host copies are not needed past the upload
    dims = {d: {c: torch.from_numpy(a).cuda() for c, a in t.items()} for d, t in w.dims.items()}
    torch.cuda.synchronize()
    q = w.query
    tables = sdb.build_dims(dims, w.dim_keys, q)
    full = sdb.StarQuery(fact, tables, q).execute()
    _log(f"2g rows: GPU {len(full.sums)} groups")

    t0 = time.time()
    want, col_sums = ranges.run("c3_star3", n, oracle_pool, TASK_ROWS, log=_log)
    _log(f"2g rows: oracle over all rows in {time.time() - t0:.1f} s")
    dev_sums = {k: int(v.sum(dtype=torch.int64).item()) for k, v in fact.items()}
    assert col_sums == dev_sums, "the oracle's workers saw other rows than the device holds"
    assert_same(full.as_rows(), want.as_rows(), "2^31 + 4099 rows")
    _log("2g rows: full result equals the oracle")

    cut = 2**30 + 3
    acc = {}
    for a, b in [(0, cut), (cut, n)]:
        part = sdb.StarQuery({k: v[a:b] for k, v in fact.items()}, tables, q).execute()
        for k, s_, c in part.as_rows():
            s0, c0 = acc.get(k, (0, 0))
            acc[k] = (s0 + s_, c0 + c)
    assert sorted((k, s_, c) for k, (s_, c) in acc.items()) == full.as_rows()
    _log("2g rows: row ranges add up")
    del fact
    torch.cuda.empty_cache()
