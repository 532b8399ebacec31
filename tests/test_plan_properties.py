"""Properties of the planner over random queries and every combination of
the planner overrides, on the CPU.

Dimension handles are filled in by hand (no table is built), the stage order
is the query's own (no sampling kernel) and the grid is given, so planning
makes no GPU call. For every query the planner accepts, the plan must be
internally consistent, and the run entry point's own validation must accept
it: without a GPU the run then stops at its first launch with SDB_HIP_ERROR,
never with SDB_INVALID_ARG.
"""

import ctypes as C

import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

from conftest import GPU_PRESENT
from paper_2607_07632_amd import sdb

OK, INVALID_ARG, UNSUPPORTED, CAPACITY, HIP_ERROR = 0, 1, 2, 3, 7
LDS_GLOBAL, LDS_MAP, LDS_BITS, LDS_RANK, LDS_COARSE, LDS_WINDOW = 0, 1, 2, 3, 4, 5


@st.composite
def dims(draw):
    kind = draw(st.sampled_from([1, 2]))                    # dense, hash
    n_rows = draw(st.one_of(st.integers(1, 3000), st.integers(1, 300_000), st.integers(1, 4_000_000)))
    n_pass = draw(st.integers(0, n_rows))
    n_pay = draw(st.integers(0, 2))
    radices = tuple(draw(st.integers(1, 300)) for _ in range(n_pay))
    h = sdb.SdbDim()
    h.kind = kind
    h.n_rows = n_rows
    h.n_pass = n_pass
    domain = 1
    for r in radices:
        domain *= r
    h.n_payloads = n_pay
    div = 1
    for p in range(n_pay - 1, -1, -1):
        h.payload_radix[p] = radices[p]
        h.payload_min[p] = draw(st.integers(-1000, 1000))
        h.payload_div[p] = div
        div *= radices[p]
    h.domain = domain
    if kind == 1:
        h.width = 1 if domain + 2 <= 0xFF else (2 if domain + 2 <= 0xFFFF else 4)
        h.n_slots = draw(st.integers(n_rows, 2 * n_rows))
        h.sentinel = (1 << (8 * h.width)) - 2
        h.bits = 0x200000 if draw(st.booleans()) else None
    else:
        h.width = 8
        bits = max(1, (2 * n_rows - 1).bit_length())
        h.hash_bits = bits
        h.n_slots = 1 << bits
        h.sentinel = 0xFFFFFFFE
    h.key_min = draw(st.integers(-5000, 5000))
    h.key_max = h.key_min + (h.n_slots - 1 if kind == 1 else n_rows * 2)
    if kind == 2:
        h.filter_kind = draw(st.sampled_from([0, 1, 2]))      # none, a bitmap over the key range, Bloom
        if h.filter_kind:
            h.filter = 0x800000
            h.filter_bits = (h.key_max - h.key_min + 1) if h.filter_kind == 1 else 32 << draw(st.integers(0, 20))
    if n_pass and draw(st.booleans()):                      # passing keys one contiguous range
        lo = draw(st.integers(h.key_min, h.key_min + 1000))
        h.pass_key_min, h.pass_key_max = lo, lo + n_pass - 1
    else:
        h.pass_key_min, h.pass_key_max = (h.key_min, h.key_min + n_pass) if n_pass else (0, -1)
    h.map = 0x400000
    return h


@st.composite
def queries(draw):
    ds = draw(st.lists(dims(), min_size=0, max_size=4))
    q = sdb.SdbQuery()
    q.n_fact = draw(st.sampled_from([0, 1, 1000, 5_000_003, 600_000_000]))
    q.n_cols = 4
    aligned = draw(st.booleans())
    for c in range(4):
        q.cols[c] = 0x1000000 + c * 0x100000 + (0 if aligned else 4)
    q.n_preds = draw(st.integers(0, 3))
    for i in range(q.n_preds):
        q.preds[i] = sdb.SdbPred(draw(st.integers(0, 3)), draw(st.integers(0, 6)),
                                 draw(st.integers(-100, 100)), draw(st.integers(-100, 100)))
    q.n_joins = len(ds)
    for j, d in enumerate(ds):
        q.joins[j] = sdb.SdbJoin(draw(st.integers(0, 3)), C.pointer(d))
    keys = [(j, p) for j, d in enumerate(ds) for p in range(d.n_payloads)]
    chosen = draw(st.lists(st.sampled_from(keys), unique=True, max_size=3)) if keys else []
    q.n_group_keys = len(chosen)
    for k, (j, p) in enumerate(chosen):
        q.group_keys[k] = sdb.SdbGroupKey(j, p)
    q.agg = sdb.SdbAgg(draw(st.integers(0, 3)), draw(st.integers(0, 3)), draw(st.integers(0, 3)))
    q.force_terminal = draw(st.integers(0, 4))
    q.force_ipt = draw(st.sampled_from([0, 1, 2, 4]))
    q.force_vector = draw(st.sampled_from([0, 1, -1]))
    q.force_order = 1
    q.grid_blocks = draw(st.integers(1, 3000))
    q.force_lds = draw(st.sampled_from([-1, 0, 2, 3]))
    q.force_xcd = draw(st.sampled_from([-1, 0, 1]))
    q.force_eager = draw(st.integers(-1, 4))
    q.force_block = draw(st.sampled_from([0, 64, 128, 256, 512, 1024]))
    q.force_range = draw(st.sampled_from([-1, 0, 1]))
    q.force_coarse = draw(st.integers(-1, 5))
    q.force_slice = draw(st.sampled_from([-1, 0, 1, 1]))
    q.force_unroll = draw(st.sampled_from([-1, 0, 0]))
    q.force_window = draw(st.sampled_from([-1, 0, 0, 1, 2, 7]))
    q.force_prefilter = draw(st.sampled_from([-1, 0, 1]))
    return q, ds


def check_plan(q, p):
    n = q.n_preds + q.n_joins
    assert p.n_stages == n
    seen = sorted((p.stage_kind[s], p.stage_index[s]) for s in range(n))
    assert seen == sorted([(0, i) for i in range(q.n_preds)] + [(1, j) for j in range(q.n_joins)])
    defers = 0
    for s in range(n):
        kind, idx, lds = p.stage_kind[s], p.stage_index[s], p.stage_lds[s]
        assert lds in (LDS_GLOBAL, LDS_MAP, LDS_BITS, LDS_RANK, LDS_COARSE, LDS_WINDOW)
        if lds != LDS_GLOBAL:
            d = q.joins[idx].dim.contents
            assert kind == 1 and d.kind == 1
            if lds in (LDS_BITS, LDS_RANK, LDS_COARSE, LDS_WINDOW):
                assert d.bits
        if lds == LDS_WINDOW:
            d = q.joins[idx].dim.contents
            lo, slots = p.stage_window_lo[s], p.stage_window_slots[s]
            assert lo % 128 == 0 and slots % 128 == 0 and slots > 0 and lo >= 0
            assert lo + slots <= (d.n_slots + 127) // 128 * 128
            assert q.force_window != -1 and q.force_lds != -1
            if q.force_window >= 2:
                assert slots <= 128 * q.force_window
            assert 0.0 <= p.stage_window_cover[s] <= 1.0
            assert p.stage_defer[s] == -1
        else:
            assert p.stage_window_lo[s] == 0 and p.stage_window_slots[s] == 0
        assert (lds == LDS_COARSE) == (p.stage_coarse[s] != 0)
        if lds == LDS_COARSE:
            assert 1 <= p.stage_coarse[s] <= 5
        if p.stage_range[s]:
            assert kind == 1 and lds == LDS_GLOBAL and p.stage_defer[s] == -1
            d = q.joins[idx].dim.contents
            assert d.n_pass == 0 or d.pass_key_max - d.pass_key_min + 1 == d.n_pass
            assert all(q.group_keys[k].join != idx for k in range(q.n_group_keys))
        assert p.stage_defer[s] in (-1, 0)
        if p.stage_defer[s] == 0:
            defers += 1
            assert lds == LDS_BITS
    assert defers <= 1
    assert sum(p.stage_lds[s] == LDS_WINDOW for s in range(n)) <= 1
    assert p.terminal in (1, 2, 3, 4)
    assert (p.terminal == 1) <= (q.n_group_keys == 0)
    assert p.ipt in (1, 2, 4) and p.block in (64, 128, 256, 512, 1024)
    if p.block == 1024:
        assert p.vector == 1 and p.ipt <= 2 and p.eager == 0
    assert 0 <= p.eager <= 4
    assert 0 <= p.lds_bytes <= 160 * 1024
    groups = 1
    for k in range(q.n_group_keys):
        groups *= p.radix[k]
    assert p.n_groups == groups
    assert p.run_scratch_bytes >= 0
    # the sliced hash probe: only the query shape it supports, and wherever
    # that shape is forced
    join_probe = [s for s in range(n) if p.stage_kind[s] == 1 and not p.stage_range[s]]
    read = ([q.joins[0].fact_key_col, q.agg.a] + ([q.agg.b] if q.agg.kind else []) +
            [q.preds[i].col for i in range(q.n_preds)]) if q.n_joins else []
    sliceable = (q.n_joins == 1 and len(join_probe) == 1 and q.joins[0].dim.contents.kind == 2 and
                 0 < q.n_fact <= 0xFFFFF000 and q.force_eager <= 0 and
                 all(q.cols[c] % 16 == 0 for c in read))
    if p.slice_bits:
        assert sliceable and q.force_slice != -1
        s = p.slice_stage
        d = q.joins[0].dim.contents
        assert s == join_probe[0] and 1 <= p.slice_bits <= min(10, d.hash_bits)
        assert 1 <= p.slice_grid <= 256 and p.eager == 0 and p.stage_lds[s] == LDS_GLOBAL
        # partition counts and offsets, and one key and value (two for a two-column aggregate) per fact row
        per_row = 12 if q.agg.kind else 8
        assert p.run_scratch_bytes >= per_row * q.n_fact + 4 * p.slice_grid * (1 << p.slice_bits)
        # the pre-filter: only into a table with a pass filter, always when forced, never when refused
        assert p.slice_prefilter in (0, 1)
        if d.filter_kind == 0 or q.force_prefilter == -1:
            assert p.slice_prefilter == 0
        elif q.force_prefilter == 1:
            assert p.slice_prefilter == 1
        if p.slice_prefilter:
            assert p.run_scratch_bytes >= per_row * q.n_fact + q.n_fact // 4
    else:
        assert not (sliceable and q.force_slice == 1)
        assert p.slice_prefilter == 0
    # the partitioned terminal: 1 to 4 record regions per block
    if p.terminal == 4:
        assert p.part_subs in (1, max(1, min(4, 1024 // p.grid))) and p.part_cap > 0 and p.n_parts > 0
    else:
        assert p.part_subs == 0
    # the unrolled stage loop: exactly where its instance exists and no hash
    # table is probed, unless turned off
    hash_probe = any(q.joins[p.stage_index[s]].dim.contents.kind == 2 for s in join_probe)
    can_unroll = (p.vector == 1 and p.ipt == 2 and p.eager == 0 and p.block in (512, 1024) and n <= 4 and
                  not p.slice_bits and not hash_probe)
    assert p.unroll == (1 if can_unroll and q.force_unroll != -1 else 0)


@settings(max_examples=400, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(queries())
def test_plans_are_consistent_and_pass_run_validation(qd):
    q, _dims = qd                                           # the handles must outlive the calls
    L = sdb.lib()
    p = sdb.SdbPlan()
    status = L.sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p))
    assert status in (OK, INVALID_ARG, UNSUPPORTED, CAPACITY), sdb.lib().sdb_last_error()
    if status != OK:
        return
    check_plan(q, p)
    if GPU_PRESENT:
        return
    scratch = 0x10000000 if p.run_scratch_bytes else None
    status = L.sdb_run_star_query(C.byref(q), C.byref(p), 0x20000000, 0x30000000, int(p.n_groups),
                                  scratch, int(p.run_scratch_bytes), None)
    assert status in (OK, HIP_ERROR), (status, sdb.lib().sdb_last_error())


@pytest.mark.parametrize("force_lds", [0, 2, 3])
@pytest.mark.parametrize("force_block", [0, 1024])
def test_rank_and_deferred_placements_pass_run_validation(force_lds, force_block):
    """A c2-like query (a 200,000-slot filtered dimension whose code is a group
    key, a small one beside it) reaches the deferred-bitmap and rank-table
    placements the random queries above rarely draw."""
    def dense(n, n_pass, radix, bits):
        h = sdb.SdbDim()
        h.kind, h.width, h.n_rows, h.n_pass, h.n_slots = 1, 1, n, n_pass, n
        h.key_min, h.key_max, h.sentinel = 0, n - 1, 0xFE
        h.n_payloads, h.payload_radix[0], h.payload_div[0], h.domain = 1, radix, 1, radix
        h.pass_key_min, h.pass_key_max = 0, n_pass      # not a contiguous range
        h.map, h.bits = 0x400000, bits
        return h
    sup, date = dense(200_000, 40_000, 25, 0x200000), dense(2556, 2556, 8, 0x300000)
    q = sdb.SdbQuery()
    q.n_fact, q.n_cols = 60_000_000, 3
    for c in range(3):
        q.cols[c] = 0x1000000 + c * 0x100000
    q.n_joins = 2
    q.joins[0], q.joins[1] = sdb.SdbJoin(0, C.pointer(sup)), sdb.SdbJoin(1, C.pointer(date))
    q.n_group_keys = 2
    q.group_keys[0], q.group_keys[1] = sdb.SdbGroupKey(0, 0), sdb.SdbGroupKey(1, 0)
    q.agg = sdb.SdbAgg(0, 2, 0)
    q.force_order, q.grid_blocks, q.force_lds, q.force_block = 1, 256, force_lds, force_block
    q.force_terminal = 3                                      # global: the deferred gather stays possible
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK
    check_plan(q, p)
    s_sup = next(s for s in range(p.n_stages) if p.stage_index[s] == 0)
    # no lookup goes to device memory, so the planner itself takes rank tables
    assert p.stage_lds[s_sup] == (LDS_BITS if force_lds == 2 else LDS_RANK)
    if p.stage_lds[s_sup] == LDS_BITS:
        assert p.stage_defer[s_sup] == 0
    else:
        assert p.block == 1024 and p.run_scratch_bytes > 0
    if GPU_PRESENT:
        return
    scratch = 0x10000000 if p.run_scratch_bytes else None
    status = sdb.lib().sdb_run_star_query(C.byref(q), C.byref(p), 0x20000000, 0x30000000, int(p.n_groups),
                                          scratch, int(p.run_scratch_bytes), None)
    assert status in (OK, HIP_ERROR), (status, sdb.lib().sdb_last_error())


def _c5_like(n_fact, hash_bits=25, n_preds=1, agg_kind=0, aligned=True, filt=None, pass_frac=0.5):
    """One hash join with its payload as the group key (a 2^hash_bits-slot
    table, `pass_frac` of its rows passing, with a pass filter `filt`: None,
    "bitmap" or "bloom"), an optional fact predicate, SUM of one column."""
    d = sdb.SdbDim()
    d.kind, d.width, d.n_rows = 2, 8, 1 << (hash_bits - 1)
    d.n_pass, d.hash_bits, d.n_slots, d.sentinel = int(pass_frac * d.n_rows), hash_bits, 1 << hash_bits, 0xFFFFFFFE
    d.key_min, d.key_max = 0, (1 << (hash_bits - 1)) - 1
    if filt:
        d.filter, d.filter_kind = 0x800000, {"bitmap": 1, "bloom": 2}[filt]
        d.filter_bits = d.key_max + 1 if filt == "bitmap" else min(8 * d.n_rows, sdb.MAX_FILTER_BYTES * 8)
    d.pass_key_min, d.pass_key_max = 0, 5                  # passing keys are not one range
    d.n_payloads, d.payload_radix[0], d.payload_div[0], d.domain = 1, 65536, 1, 65536
    d.map = 0x400000
    q = sdb.SdbQuery()
    q.n_fact, q.n_cols = n_fact, 3
    for c in range(3):
        q.cols[c] = 0x1000000 + c * 0x100000 + (0 if aligned else 4)
    q.n_preds = n_preds
    for i in range(n_preds):
        q.preds[i] = sdb.SdbPred(2, 5, 1, 100)               # col 2 BETWEEN 1 AND 100
    q.n_joins = 1
    q.joins[0] = sdb.SdbJoin(0, C.pointer(d))
    q.n_group_keys = 1
    q.group_keys[0] = sdb.SdbGroupKey(0, 0)
    q.agg = sdb.SdbAgg(agg_kind, 1, 2)
    q.force_order, q.grid_blocks = 1, 256
    return q, d


def _run_status(q, p):
    scratch = 0x10000000 if p.run_scratch_bytes else None
    return sdb.lib().sdb_run_star_query(C.byref(q), C.byref(p), 0x20000000, 0x30000000, int(p.n_groups),
                                        scratch, int(p.run_scratch_bytes), None)


@pytest.mark.parametrize("force_slice,n_fact,hash_bits,agg_kind,aligned,sliced", [
    (0, 600_000_000, 25, 0, True, True),      # c5's shape: a 256 MiB table, 600M rows
    (0, 600_000_000, 20, 0, True, False),     # an 8 MiB table: probes mostly hit L2 anyway
    (0, 1_000_000, 25, 0, True, False),       # too few rows to pay for the passes
    (1, 1_000_000, 12, 0, True, True),        # forced on a small case
    (1, 600_000_000, 25, 2, True, True),      # revenue - cost: both operands travel with the key
    (0, 600_000_000, 25, 1, True, True),      # a product, chosen by the planner
    (1, 600_000_000, 25, 0, False, False),    # the passes load 128 bits at a time
    (-1, 600_000_000, 25, 0, True, False),
])
def test_sliced_probe_choice(force_slice, n_fact, hash_bits, agg_kind, aligned, sliced):
    q, _d = _c5_like(n_fact, hash_bits, agg_kind=agg_kind, aligned=aligned)
    q.force_slice = force_slice
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK, sdb.lib().sdb_last_error()
    check_plan(q, p)
    assert bool(p.slice_bits) == sliced
    if sliced:
        assert p.stage_kind[p.slice_stage] == 1
        # 2 MiB slices of the table
        assert p.slice_bits == max(1, min(hash_bits + 3 - 21, hash_bits, 10))
        assert p.vector == 1
        assert p.slice_grid == min(256, -(-n_fact // 16384))
    if not GPU_PRESENT:
        assert _run_status(q, p) in (OK, HIP_ERROR), sdb.lib().sdb_last_error()


def test_sliced_plan_validation():
    q, _d = _c5_like(600_000_000)
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK
    assert p.slice_bits == 7
    good = bytes(p)
    for field, value in [("slice_bits", 11), ("slice_bits", -1), ("slice_stage", 0), ("slice_stage", 5),
                         ("slice_grid", 0), ("slice_grid", 257), ("unroll", 1), ("eager", 1)]:
        bad = sdb.SdbPlan.from_buffer_copy(good)
        setattr(bad, field, value)
        assert _run_status(q, bad) == INVALID_ARG, (field, value)
    # a plan for one query is not valid for one the slices cannot serve (unaligned columns)
    q2, _d2 = _c5_like(600_000_000, aligned=False)
    assert _run_status(q2, sdb.SdbPlan.from_buffer_copy(good)) == INVALID_ARG
    # nor, for want of scratch, for a two-column aggregate, whose second operands travel too
    q3, _d3 = _c5_like(600_000_000, agg_kind=2)
    assert _run_status(q3, sdb.SdbPlan.from_buffer_copy(good)) == 4
    # too little scratch for the partitioned records
    short = sdb.lib().sdb_run_star_query(C.byref(q), C.byref(p), 0x20000000, 0x30000000, int(p.n_groups),
                                         0x10000000, int(p.run_scratch_bytes) - 256, None)
    assert short == 4                                       # SDB_WORKSPACE_TOO_SMALL


def _bloom_false_positive(bits, n_keys):
    """Blocked Bloom filter, 3 bits of one 32-bit word per key: the chance
    that all 3 bits of a key not in the set are set, a word holding
    Poisson(n_keys / words) keys."""
    import math
    lam = n_keys / (bits // 32)
    fp, pmf = 0.0, math.exp(-lam)
    for j in range(int(lam + 12 * math.sqrt(lam + 1) + 24) + 1):
        fp += pmf * (1 - (31 / 32) ** (3 * j)) ** 3
        pmf *= lam / (j + 1)
    return fp


@pytest.mark.parametrize("filt,pass_frac,force,want", [
    ("bitmap", 0.5, 0, 1),       # c5: half the rows cannot pass the join
    ("bitmap", 0.9, 0, 0),       # too few rows dropped to pay for a filter read per row
    ("bitmap", 0.9, 1, 1),
    ("bitmap", 0.5, -1, 0),
    (None, 0.5, 1, 0),           # no filter to test against
    ("bloom", 0.05, 0, 1),       # few keys: few false positives
    ("bloom", 0.7, 0, 0),        # a crowded filter lets most of the rest through
])
def test_prefilter_choice(filt, pass_frac, force, want):
    q, _d = _c5_like(600_000_000, filt=filt, pass_frac=pass_frac)
    q.force_prefilter = force
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK, sdb.lib().sdb_last_error()
    check_plan(q, p)
    assert p.slice_bits and p.slice_prefilter == want
    if filt == "bloom" and force == 0:
        d = _d
        kept = pass_frac + (1 - pass_frac) * _bloom_false_positive(d.filter_bits, d.n_pass)
        assert (kept <= 0.7) == bool(want)
    if want:
        q0, _d0 = _c5_like(600_000_000, filt=filt, pass_frac=pass_frac)
        q0.force_prefilter = -1
        p0 = sdb.SdbPlan()
        assert sdb.lib().sdb_plan_star_query(C.byref(q0), None, 0, None, C.byref(p0)) == OK
        assert p.run_scratch_bytes - p0.run_scratch_bytes >= 600_000_000 // 4     # a byte per 4 rows
    if not GPU_PRESENT:
        assert _run_status(q, p) in (OK, HIP_ERROR), sdb.lib().sdb_last_error()


def test_prefilter_plan_validation():
    q, _d = _c5_like(600_000_000, filt="bitmap")
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK
    assert p.slice_prefilter == 1
    for value in (2, -1):
        bad = sdb.SdbPlan.from_buffer_copy(p)
        bad.slice_prefilter = value
        assert _run_status(q, bad) == INVALID_ARG
    # a table without a pass filter cannot serve the plan
    q2, _d2 = _c5_like(600_000_000)
    assert _run_status(q2, sdb.SdbPlan.from_buffer_copy(p)) == INVALID_ARG
    # nor a plan without the sliced probe
    unsliced = sdb.SdbPlan.from_buffer_copy(p)
    unsliced.slice_bits = 0
    assert _run_status(q, unsliced) == INVALID_ARG


@pytest.mark.parametrize("mutate", [
    lambda d: setattr(d, "filter_bits", d.filter_bits - 1),     # a bitmap covers exactly the key range
    lambda d: setattr(d, "filter", None),
    lambda d: setattr(d, "filter_kind", 3),
    lambda d: (setattr(d, "filter_kind", 2), setattr(d, "filter_bits", 96)),   # Bloom: 32 x a power of two
    lambda d: (setattr(d, "filter_kind", 2), setattr(d, "filter_bits", 64 << 20)),   # above 4 MiB
    lambda d: setattr(d, "reserved_", 1),
])
def test_filter_fields_are_checked(mutate):
    q, d = _c5_like(600_000_000, filt="bitmap")
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK
    mutate(d)
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(sdb.SdbPlan())) == INVALID_ARG
    msg = sdb.lib().sdb_last_error().decode()
    assert "filter" in msg or "reserved" in msg, msg


@pytest.mark.parametrize("n_fact,grid,subs", [(100_000_000, 256, 4), (100_000_000, 300, 3), (100_000_000, 512, 2),
                                              (100_000_000, 1024, 1), (100_000_000, 3000, 1),
                                              (600_000_000, 256, 1)])
def test_partitioned_record_regions(n_fact, grid, subs):
    """The partitioned terminal splits each block's records over part_subs
    regions (about 1024 regions per launch) when a block expects fewer than
    2^18 records; the run checks the field."""
    q, _d = _c5_like(n_fact)
    q.force_slice, q.force_terminal, q.grid_blocks = -1, 4, grid
    p = sdb.SdbPlan()
    assert sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p)) == OK, sdb.lib().sdb_last_error()
    check_plan(q, p)
    assert p.terminal == 4 and p.part_subs == subs
    # room for 1.5 x the estimated survivors (half the rows pass the join, about
    # half the predicate) over all the regions, in multiples of 64 records
    assert p.part_cap % 64 == 0 and p.part_cap * grid * subs >= 1.5 * n_fact * 0.25 * 0.98
    for value in (0, 5):
        bad = sdb.SdbPlan.from_buffer_copy(p)
        bad.part_subs = value
        assert _run_status(q, bad) == INVALID_ARG
