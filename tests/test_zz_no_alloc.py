"""The allocation-free run (sdb_run_star_query_noalloc, through the C ABI)
against sdb_run_star_query with a caller-owned scratch buffer: the group
tables must be equal element by element, on two calls in a row, the second
over fewer rows (the fixed scratch keeps the first call's contents), with the
outputs scribbled over before every call."""

import numpy as np
import pytest

import datagen
from gpu_util import require_gpu, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _tables(sums, counts):
    import torch
    torch.cuda.synchronize()
    return sums.cpu().numpy().copy(), counts.cpu().numpy().copy()


# workload, rows of the first call, rows of the second, planner overrides,
# whether the plan keeps anything in the run scratch
CASES = [
    ("c4_star4_zipf", 4_000_002, 1_000_003, {"terminal": "global", "xcd": 1}, True),   # per-XCD copies
    ("c2_join_group", 4_000_003, 999_999, {"lds": 3}, True),                          # LDS rank tables
    ("c3_star3", 2_000_001, 700_001, {"terminal": "part"}, True),                      # partitioned terminal
    ("c5_hash_stress", 2_000_003, 600_001, {"slice": 1}, True),                        # sliced hash probe
    ("c3_star3", 4_000_001, 1_500_007, {"terminal": "global", "xcd": -1, "lds": 2}, False),   # LDS bitmaps, no rank tables
    ("c1_scalar_scan", None, 100_001, None, False),
]


@pytest.mark.parametrize("name,n1,n2,force,uses_scratch", CASES)
def test_noalloc_run_equals_the_scratch_run(name, n1, n2, force, uses_scratch):
    import torch
    from paper_2607_07632_amd import sdb
    w = datagen.make_workload(name, n_fact=n1)
    fact, dims = upload(w)
    tables = sdb.build_dims(dims, w.dim_keys, w.query)
    for n in (w.n_fact, n2):
        cols = {k: v[:n] for k, v in fact.items()}
        q = sdb.StarQuery(cols, tables, w.query, force)
        plan = q.plan()
        assert plan.run_scratch_bytes <= sdb.NOALLOC_SCRATCH_BYTES
        assert (plan.run_scratch_bytes > 0) == uses_scratch
        sums_a, counts_a = q.alloc_outputs(plan)
        sums_b, counts_b = q.alloc_outputs(plan)
        for t in (sums_a, counts_a, sums_b, counts_b):
            t.fill_(-7)
        q.run(sums_a, counts_a, plan=plan)
        q.run_noalloc(sums_b, counts_b, plan=plan)
        want, got = _tables(sums_a, counts_a), _tables(sums_b, counts_b)
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1]), f"{name} {n} rows"
        assert want[1].sum() > 0
        print(f"{name}: {n} rows, {plan.run_scratch_bytes} scratch bytes, {int((want[1] > 0).sum())} groups equal",
              flush=True)


def test_noalloc_run_refuses_a_plan_beyond_its_scratch():
    """A plan needing more than the fixed scratch is refused before any launch:
    the outputs keep what they held."""
    import torch
    from paper_2607_07632_amd import sdb
    n = (1 << 24) + 1_003
    w = datagen.make_workload("c5_hash_stress", n_fact=n)
    fact, dims = upload(w)
    tables = sdb.build_dims(dims, w.dim_keys, w.query)
    q = sdb.StarQuery(fact, tables, w.query, {"slice": 1})
    plan = q.plan()
    assert plan.slice_bits > 0 and plan.run_scratch_bytes > sdb.NOALLOC_SCRATCH_BYTES
    sums, counts = q.alloc_outputs(plan)
    sums.fill_(11)
    counts.fill_(13)
    with pytest.raises(sdb.SdbError) as e:
        q.run_noalloc(sums, counts, plan=plan)
    assert e.value.name == "SDB_WORKSPACE_TOO_SMALL"
    torch.cuda.synchronize()
    assert bool((sums == 11).all()) and bool((counts == 13).all())
