"""The C ABI on the CPU: the library loads, exports what include/sdb.h declares,
agrees with the binding's struct layout, and validates and plans on the host
(no GPU call is made by anything tested here)."""

import ctypes as C
import os
import re

import pytest

from conftest import GPU_PRESENT
from paper_2607_07632_amd import sdb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sdb.h")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SDB_API\s+[\w\s\*]+?\b(sdb_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    syms = declared_symbols()
    for name in ["sdb_build_dim", "sdb_run_star_query", "sdb_plan_star_query", "sdb_finalize_groups",
                 "sdb_dim_required_bytes", "sdb_last_error"]:
        assert name in syms


def test_library_exports_every_declared_symbol():
    L = sdb.lib()
    for name in declared_symbols():
        assert hasattr(L, name), name
    assert set(declared_symbols()) == set(sdb.SIGNATURES)


def test_struct_layout_matches_binding():
    L = sdb.lib()
    sizes = (C.c_int64 * 9)()
    assert L.sdb_struct_sizes(sizes, 9) == 0
    assert [C.sizeof(s) for s in sdb.STRUCTS] == list(sizes)
    assert L.sdb_struct_sizes(sizes, 10) == 1
    assert L.sdb_abi_version() == 10


def test_status_strings():
    L = sdb.lib()
    assert L.sdb_status_string(0) == b"SDB_OK"
    assert L.sdb_status_string(5) == b"SDB_DUP_KEY"
    assert L.sdb_status_string(99) == b"SDB_UNKNOWN_STATUS"


def _desc(n_rows=1000, kind="auto", n_cols=2, lf=0.0):
    d = sdb.SdbDimDesc()
    d.key = 0x10000
    d.n_rows = n_rows
    d.n_cols = n_cols
    for i in range(n_cols):
        d.cols[i] = 0x20000 + 0x1000 * i
    d.kind = sdb.TABLES[kind]
    d.load_factor = lf
    return d


def test_required_bytes_bounds():
    dense = sdb.dim_required_bytes(_desc(1000, "dense"))
    # stats + 2000 slots x 4 B + pass bitmap
    assert dense == 256 + 8192 + 256
    h = sdb.dim_required_bytes(_desc(1000, "hash"))
    assert h == 256 + 2048 * 8 + 1024            # slots, then a pass filter of 8 bits per row (1024 bytes)
    a = sdb.dim_required_bytes(_desc(1000, "auto"))
    assert a == max(dense, h)
    big = sdb.dim_required_bytes(_desc(1 << 24, "hash", lf=0.5))
    assert big == 256 + (1 << 25) * 8 + sdb.MAX_FILTER_BYTES   # 256 MiB table at load factor 0.5, 4 MiB filter
    assert sdb.dim_required_bytes(_desc(10, "hash")) == 256 + 256 + 256      # 32 slots padded, 256-byte filter
    budget = _desc(1000, "auto")
    budget.dense_budget_bytes = 1 << 20
    assert sdb.dim_required_bytes(budget) == 256 + (1 << 20) + 512      # room for a dense table of the budget
    budget.kind = sdb.TABLES["hash"]
    assert sdb.dim_required_bytes(budget) == h                          # a hash table ignores it
    for bad in (-1, 1 << 40):
        budget.dense_budget_bytes = bad
        with pytest.raises(sdb.SdbError) as e:
            sdb.dim_required_bytes(budget)
        assert e.value.name == "SDB_INVALID_ARG"


@pytest.mark.parametrize("mutate,status", [
    (lambda d: setattr(d, "n_rows", -1), "SDB_INVALID_ARG"),
    (lambda d: setattr(d, "n_cols", 9), "SDB_UNSUPPORTED"),
    (lambda d: setattr(d, "kind", 7), "SDB_INVALID_ARG"),
    (lambda d: (setattr(d, "kind", 2), setattr(d, "load_factor", 0.95)), "SDB_INVALID_ARG"),
    (lambda d: (setattr(d, "n_preds", 1), setattr(d.preds[0], "col", 5)), "SDB_INVALID_ARG"),
    (lambda d: (setattr(d, "n_preds", 1), setattr(d.preds[0], "op", 9)), "SDB_INVALID_ARG"),
    (lambda d: (setattr(d, "n_payloads", 1), setattr(d.payload_cols, "__setitem__", None)), None),
    (lambda d: (setattr(d, "n_payloads", 4)), "SDB_UNSUPPORTED"),
    (lambda d: setattr(d, "key", None), "SDB_INVALID_ARG"),
])
def test_dim_descriptor_validation(mutate, status):
    d = _desc()
    try:
        mutate(d)
    except (AttributeError, TypeError):
        pass
    if status is None:
        sdb.dim_required_bytes(d)
        return
    with pytest.raises(sdb.SdbError) as e:
        sdb.dim_required_bytes(d)
    assert e.value.name == status
    assert sdb.lib().sdb_last_error().decode().startswith(status)


def _fake_dim(kind=1, width=1, n_rows=200_000, n_pass=40_000, radices=(25,), mins=(0,),
              key_min=0, n_slots=200_000, bits=0, pass_range=(0, 0), with_bitmap=False):
    h = sdb.SdbDim()
    h.kind = kind
    h.width = width
    h.n_rows = n_rows
    h.n_pass = n_pass
    h.key_min = key_min
    h.key_max = key_min + n_slots - 1
    h.pass_key_min, h.pass_key_max = pass_range
    h.n_slots = n_slots if kind == 1 else (1 << bits)
    h.hash_bits = bits
    h.sentinel = 0xFF
    h.n_payloads = len(radices)
    div = 1
    for p in range(len(radices) - 1, -1, -1):
        h.payload_radix[p] = radices[p]
        h.payload_min[p] = mins[p]
        h.payload_div[p] = div
        div *= radices[p]
    h.domain = div
    h.map = 0x40000
    h.bits = 0x80000 if with_bitmap else None
    return h


def test_dim_info_reports_the_handle():
    """sdb_dim_info through the ABI, on handles filled on the host."""
    info = sdb.dim_info(_fake_dim(radices=(25, 7), mins=(3, -2), n_slots=200_000, pass_range=(10, 40_009),
                                  with_bitmap=True))
    assert info["kind"] == "dense" and info["width"] == 1 and info["n_slots"] == 200_000
    assert info["table_bytes"] == 200_192 + 25_088       # map and pass bitmap, each padded to 256 bytes
    assert info["payload_min"] == [3, -2] and info["payload_max"] == [27, 4]
    assert info["payload_radix"] == [25, 7] and info["domain"] == 175
    assert info["pass_keys_contiguous"] and info["occupancy"] == 1.0
    gap = sdb.dim_info(_fake_dim(pass_range=(0, 40_000), with_bitmap=True))   # 40,001 keys, 40,000 passing
    assert not gap["pass_keys_contiguous"]
    h = sdb.dim_info(_fake_dim(kind=2, width=8, n_rows=1 << 24, n_pass=1 << 23, bits=25, radices=(65536,)))
    assert h["kind"] == "hash" and h["n_slots"] == 1 << 25 and h["table_bytes"] == 1 << 28
    assert h["occupancy"] == 0.5 and h["payload_max"] == [65535]


def test_dim_info_reports_and_checks_the_pass_filter():
    """A hash table's pass filter through sdb_dim_info: its kind and bytes,
    and the handles whose filter fields contradict the table are refused."""
    h = _fake_dim(kind=2, width=8, n_rows=1 << 24, n_pass=1 << 23, bits=25, radices=(65536,),
                  n_slots=1 << 24)
    assert sdb.dim_info(h)["filter"] is None and sdb.dim_info(h)["filter_bytes"] == 0
    h.filter, h.filter_kind, h.filter_bits = 0x900000, 1, 1 << 24     # a bitmap over the 2^24 keys
    info = sdb.dim_info(h)
    assert info["filter"] == "bitmap" and info["filter_bytes"] == 2 << 20
    h.filter_kind, h.filter_bits = 2, 1 << 25                       # a 4 MiB Bloom filter
    assert sdb.dim_info(h)["filter"] == "bloom" and sdb.dim_info(h)["filter_bytes"] == 4 << 20
    for field, value in [("filter_bits", 3 << 20), ("filter_bits", 16), ("filter_bits", 1 << 26), ("filter", None),
                         ("filter_kind", 7), ("reserved_", 2)]:
        bad = sdb.SdbDim.from_buffer_copy(h)
        setattr(bad, field, value)
        with pytest.raises(sdb.SdbError) as e:
            sdb.dim_info(bad)
        assert e.value.name == "SDB_INVALID_ARG", (field, value)
    bad = sdb.SdbDim.from_buffer_copy(h)
    bad.filter_kind, bad.filter_bits = 1, (1 << 24) - 1               # a bitmap must cover the key range
    with pytest.raises(sdb.SdbError):
        sdb.dim_info(bad)
    dense = _fake_dim(with_bitmap=True)
    dense.filter, dense.filter_kind, dense.filter_bits = 0x900000, 1, 200_000
    with pytest.raises(sdb.SdbError):
        sdb.dim_info(dense)                                          # only hash tables carry one


@pytest.mark.parametrize("field,value", [("kind", 0), ("kind", 3), ("width", 3), ("n_pass", 200_001),
                                         ("n_rows", -1), ("n_payloads", 4), ("n_slots", 7), ("map", None),
                                         ("bits", None)])
def test_dim_info_rejects_inconsistent_handles(field, value):
    h = _fake_dim(with_bitmap=True)
    sdb.dim_info(h)
    setattr(h, field, value)
    with pytest.raises(sdb.SdbError) as e:
        sdb.dim_info(h)
    assert e.value.name == "SDB_INVALID_ARG"
    hh = _fake_dim(kind=2, width=8, n_rows=1000, n_pass=10, bits=11)
    hh.n_slots = 1000                                             # not 2^hash_bits
    with pytest.raises(sdb.SdbError):
        sdb.dim_info(hh)


def test_binding_rejects_unreadable_columns_before_any_library_call(monkeypatch):
    """int64, strided, two-dimensional and host tensors are refused with a
    ValueError by the binding; the library is never reached."""
    import torch

    def no_library():
        raise AssertionError("the binding called the library")

    monkeypatch.setattr(sdb, "lib", no_library)
    good = torch.arange(100, dtype=torch.int32)
    cases = [(torch.arange(100, dtype=torch.int64), "int32"),
             (torch.arange(200, dtype=torch.int32)[::2], "contiguous"),
             (torch.arange(200, dtype=torch.int32).reshape(100, 2)[:, 0], "contiguous"),
             (torch.arange(100, dtype=torch.int32).reshape(10, 10), "one-dimensional"),
             (good, "GPU")]
    for bad, msg in cases:
        with pytest.raises(ValueError, match=msg):
            sdb.dim_desc(bad, {"a": good}, [], [])
        with pytest.raises(ValueError, match=msg):
            sdb.build_dim(bad, {"a": good}, [], [])
        q = {"fact_preds": [], "joins": [], "group_by": [], "agg": {"kind": "col", "a": "v", "b": None}}
        with pytest.raises(ValueError, match=msg):
            sdb.StarQuery({"v": bad}, [], q)
    with pytest.raises(ValueError, match="must be a torch tensor"):
        sdb.dim_desc([1, 2, 3], {}, [], [])


def _query(dims, group_keys, n_fact=1000, n_preds=0, align=True):
    q = sdb.SdbQuery()
    q.n_fact = n_fact
    q.n_cols = 4
    base = 0x100000 if align else 0x100004
    for c in range(4):
        q.cols[c] = base + c * 0x10000
    q.n_preds = n_preds
    for i in range(n_preds):
        q.preds[i] = sdb.SdbPred(3, sdb.OPS["lt"], 30, 0)
    q.n_joins = len(dims)
    for j, d in enumerate(dims):
        q.joins[j] = sdb.SdbJoin(j % 3, C.pointer(d))
    q.n_group_keys = len(group_keys)
    for k, (j, p) in enumerate(group_keys):
        q.group_keys[k] = sdb.SdbGroupKey(j, p)
    q.agg = sdb.SdbAgg(sdb.AGGS["col"], 3, 0)
    q.force_order = 1
    return q


def _plan(q):
    p = sdb.SdbPlan()
    st = sdb.lib().sdb_plan_star_query(C.byref(q), None, 0, None, C.byref(p))
    if st != 0:
        raise sdb.SdbError(st, sdb.lib().sdb_last_error().decode())
    return p


def test_plan_group_layout_and_terminals():
    sup = _fake_dim(radices=(25,), mins=(0,))
    date = _fake_dim(n_rows=2556, n_pass=2556, radices=(8,), mins=(1992,), n_slots=2556)
    p = _plan(_query([sup, date], [(0, 0), (1, 0)]))
    assert p.n_groups == 200 and list(p.radix[:2]) == [25, 8] and list(p.stride[:2]) == [8, 1]
    assert list(p.key_min[:2]) == [0, 1992]
    assert sdb.TERMINAL_NAMES[p.terminal] == "lds" and p.ipt == 2 and p.vector == 1
    assert [p.stage_kind[i] for i in range(2)] == [1, 1]
    cust = _fake_dim(n_rows=3_000_000, radices=(250,), n_slots=3_000_000)
    sup2 = _fake_dim(radices=(250,))
    date2 = _fake_dim(n_rows=2556, radices=(6,), mins=(1992,), n_slots=2556)
    p3 = _plan(_query([cust, sup2, date2], [(0, 0), (1, 0), (2, 0)]))
    assert p3.n_groups == 375_000 and sdb.TERMINAL_NAMES[p3.terminal] == "global"
    assert list(p3.stride[:3]) == [1500, 6, 1]
    p1 = _plan(_query([date2], [], n_preds=2))
    assert p1.n_groups == 1 and sdb.TERMINAL_NAMES[p1.terminal] == "scalar" and p1.ipt == 2
    assert [p1.stage_kind[i] for i in range(3)] == [0, 0, 1]


def test_plan_multi_payload_layout():
    d = _fake_dim(radices=(5, 7, 3), mins=(10, -2, 0))
    p = _plan(_query([d], [(0, 2), (0, 0)]))
    assert p.n_groups == 15 and list(p.radix[:2]) == [3, 5] and list(p.stride[:2]) == [5, 1]
    assert list(p.key_min[:2]) == [0, 10]


def test_plan_capacity_and_validation_errors():
    big = _fake_dim(radices=(60_000,))
    with pytest.raises(sdb.SdbError) as e:
        _plan(_query([big, big], [(0, 0), (1, 0)]))
    assert e.value.name == "SDB_CAPACITY"
    d = _fake_dim()
    q = _query([d], [(0, 1)])
    with pytest.raises(sdb.SdbError) as e:
        _plan(q)
    assert e.value.name == "SDB_INVALID_ARG"
    q = _query([d], [(0, 0)])
    q.force_terminal = sdb.TERMINALS["scalar"]
    with pytest.raises(sdb.SdbError) as e:
        _plan(q)
    assert e.value.name == "SDB_INVALID_ARG"
    q = _query([d], [(0, 0)])
    q.force_ipt = 8
    with pytest.raises(sdb.SdbError) as e:
        _plan(q)
    assert e.value.name == "SDB_UNSUPPORTED"
    q = _query([d], [(0, 0)], align=False)
    assert _plan(q).vector == 0
    q.force_vector = 1
    with pytest.raises(sdb.SdbError) as e:
        _plan(q)
    assert e.value.name == "SDB_INVALID_ARG"
    q = _query([d], [(0, 0)])
    q.n_fact = -5
    with pytest.raises(sdb.SdbError):
        _plan(q)
    q = _query([d, d], [(0, 0)], n_fact=1000)
    q.force_order = 0
    with pytest.raises(sdb.SdbError) as e:          # sampling two stages needs scratch
        _plan(q)
    assert e.value.name == "SDB_INVALID_ARG"


def test_run_rejects_mismatched_plan_before_any_launch():
    d = _fake_dim()
    q = _query([d], [(0, 0)])
    p = _plan(q)
    L = sdb.lib()
    assert L.sdb_run_star_query(C.byref(q), C.byref(p), 0x1000, 0x2000, 10, None, 0, None) == 3   # CAPACITY
    p2 = sdb.SdbPlan.from_buffer_copy(p)
    p2.n_stages = 0
    assert L.sdb_run_star_query(C.byref(q), C.byref(p2), 0x1000, 0x2000, 100, None, 0, None) == 1
    p3 = sdb.SdbPlan.from_buffer_copy(p)
    p3.stage_index[0] = 4
    assert L.sdb_run_star_query(C.byref(q), C.byref(p3), 0x1000, 0x2000, 100, None, 0, None) == 1
    assert L.sdb_run_star_query(C.byref(q), C.byref(p), None, 0x2000, 100, None, 0, None) == 1
    p4 = sdb.SdbPlan.from_buffer_copy(p)
    p4.stage_lds[0] = 1                                   # LDS map on a table with width 1: allowed
    p4.stage_defer[0] = 0                                 # but a deferred gather needs the bitmap mode
    assert L.sdb_run_star_query(C.byref(q), C.byref(p4), 0x1000, 0x2000, 100, None, 0, None) == 1
    p5 = sdb.SdbPlan.from_buffer_copy(p)
    p5.xcd_copies = 8                                     # copies need the global terminal
    assert L.sdb_run_star_query(C.byref(q), C.byref(p5), 0x1000, 0x2000, 100, None, 0, None) == 1
    # the unrolled stage loop: only for the instance it exists for
    p6 = sdb.SdbPlan.from_buffer_copy(p)
    p6.unroll = 2
    assert L.sdb_run_star_query(C.byref(q), C.byref(p6), 0x1000, 0x2000, 100, None, 0, None) == 1
    if p.unroll:
        p7 = sdb.SdbPlan.from_buffer_copy(p)
        p7.ipt = 1                                        # no unrolled instance with one item per lane
        assert L.sdb_run_star_query(C.byref(q), C.byref(p7), 0x1000, 0x2000, 100, None, 0, None) == 1


def test_unroll_choice_and_validation():
    d = _fake_dim()
    q = _query([d], [(0, 0)])
    assert _plan(q).unroll == 1                            # one dense probe, 4-row items, ipt 2, blocks of 512
    q.force_unroll = -1
    assert _plan(q).unroll == 0
    q.force_ipt = 1
    q.force_unroll = 0
    assert _plan(q).unroll == 0                            # no unrolled instance for ipt 1
    L = sdb.lib()
    p = sdb.SdbPlan()
    for field, bad in [("force_unroll", 1), ("force_unroll", -2), ("force_window", -2)]:
        qb = _query([d], [(0, 0)])
        setattr(qb, field, bad)
        assert L.sdb_plan_star_query(C.byref(qb), None, 0, None, C.byref(p)) == 1, (field, bad)


def test_probe_as_key_range():
    d_gk = _fake_dim(pass_range=(100, 40_099))              # contiguous, but it feeds a group key
    d_f = _fake_dim(pass_range=(5, 40_004))                 # contiguous, filter only: a key range
    d_gap = _fake_dim(pass_range=(5, 40_005))               # 40,001 values for 40,000 keys: a gap
    d_none = _fake_dim(n_pass=0, pass_range=(0, -1))        # nothing passes: the empty range
    q = _query([d_gk, d_f, d_gap, d_none], [(0, 0)])
    q.force_range = 1
    p = _plan(q)
    got = {p.stage_index[s]: p.stage_range[s] for s in range(p.n_stages) if p.stage_kind[s] == 1}
    assert got == {0: 0, 1: 1, 2: 0, 3: 1}
    for s in range(p.n_stages):
        if p.stage_range[s]:
            assert p.stage_lds[s] == 0 and p.stage_defer[s] == -1
    assert sdb.plan_summary(p)["stages"][1]["table"] == "key_range"
    # automatic: only probes that would look up device memory; a small table staged in LDS stays a lookup
    d_small = _fake_dim(n_rows=1000, n_pass=200, n_slots=1000, pass_range=(300, 499))
    d_big = _fake_dim(n_rows=4_000_000, n_pass=800_000, n_slots=4_000_000, pass_range=(7, 800_006))
    qa = _query([d_small, d_big, d_gk], [(2, 0)])
    pa = _plan(qa)
    table = {st["index"]: st["table"] for st in sdb.plan_summary(pa)["stages"]}
    assert table[0] == "lds_map" and table[1] == "key_range" and table[2] != "key_range"
    # the cost-model order (no sample without fact rows) moves the flags with their stages
    q.n_fact = 0
    q.force_order = 0
    p2 = _plan(q)
    order = [p2.stage_index[s] for s in range(p2.n_stages)]
    assert order != [0, 1, 2, 3]
    assert {p2.stage_index[s]: p2.stage_range[s] for s in range(p2.n_stages)} == {0: 0, 1: 1, 2: 0, 3: 1}
    q.n_fact = 1000
    q.force_order = 1
    q.force_range = -1
    p_off = _plan(q)
    assert all(p_off.stage_range[s] == 0 for s in range(p_off.n_stages))
    q.force_range = 2
    with pytest.raises(sdb.SdbError) as e:
        _plan(q)
    assert e.value.name == "SDB_INVALID_ARG"
    q.force_range = 1
    # a plan that marks a probe with a gap in its passing keys is refused before any launch
    bad = sdb.SdbPlan.from_buffer_copy(p)
    s_gap = next(s for s in range(p.n_stages) if p.stage_kind[s] == 1 and p.stage_index[s] == 2)
    bad.stage_lds[s_gap] = 0
    bad.stage_range[s_gap] = 1
    L = sdb.lib()
    assert L.sdb_run_star_query(C.byref(q), C.byref(bad), 0x1000, 0x2000, 100, None, 0, None) == 1
    assert "key range" in L.sdb_last_error().decode()


def test_read_columns_validation():
    L = sdb.lib()
    cols = (C.c_void_p * 2)(0x10000, 0x20000)
    assert L.sdb_read_columns(None, 1, 10, 0, 0x3000, None) == 1
    assert L.sdb_read_columns(cols, 2, 10, 0, None, None) == 1
    assert L.sdb_read_columns(cols, 17, 10, 0, 0x3000, None) == 1
    assert L.sdb_read_columns(cols, 2, -1, 0, 0x3000, None) == 1
    assert L.sdb_read_columns(cols, 2, 10, 5, 0x3000, None) == 1
    bad = (C.c_void_p * 2)(0x10000, 0x20004)
    assert L.sdb_read_columns(bad, 2, 10, 0, 0x3000, None) == 1
    assert "aligned" in L.sdb_last_error().decode()


def test_coarse_placement_and_validation():
    big = _fake_dim(n_rows=4_000_000, n_pass=800_000, n_slots=4_000_000)
    big.bits = 0x80000
    q = _query([big], [(0, 0)])
    q.force_coarse = 2
    p = _plan(q)
    assert p.stage_lds[0] == 4 and p.stage_coarse[0] == 2        # 4M slots / 4 per bit = 125,000 bytes
    st = sdb.plan_summary(p)["stages"][0]
    assert st["table"] == "lds_coarse" and st["coarse_slots_per_bit"] == 4
    assert p.lds_bytes >= 125_000 and p.run_scratch_bytes >= 125_000
    q.force_coarse = 1                                          # 250,000 bytes do not fit LDS
    p1 = _plan(q)
    assert p1.stage_lds[0] == 0 and p1.stage_coarse[0] == 0
    q.force_coarse = -1
    assert _plan(q).stage_lds[0] == 0
    for bad in (6, -2):
        q.force_coarse = bad
        with pytest.raises(sdb.SdbError) as e:
            _plan(q)
        assert e.value.name == "SDB_INVALID_ARG"
    nobits = _fake_dim(n_rows=4_000_000, n_pass=800_000, n_slots=4_000_000)
    qn = _query([nobits], [(0, 0)])
    qn.force_coarse = 2
    assert _plan(qn).stage_lds[0] == 0                          # no pass bitmap, no coarse filter
    # plans whose coarse fields disagree are refused before any launch
    q.force_coarse = 2
    L = sdb.lib()
    for lds, shift in ((0, 2), (4, 0), (4, 6)):
        bad = sdb.SdbPlan.from_buffer_copy(p)
        bad.stage_lds[0] = lds
        bad.stage_coarse[0] = shift
        assert L.sdb_run_star_query(C.byref(q), C.byref(bad), 0x1000, 0x2000, 100, None, 0, None) == 1


def test_baseline_scratch_and_validation():
    L = sdb.lib()
    nb = C.c_int64(0)
    assert L.sdb_baseline_scratch_bytes(1000, C.byref(nb)) == 0
    assert nb.value == 1024 + 4096                        # flags, then 256-aligned group ids
    assert L.sdb_baseline_scratch_bytes(0, C.byref(nb)) == 0 and nb.value == 0
    assert L.sdb_baseline_scratch_bytes(-1, C.byref(nb)) == 1
    d = _fake_dim()
    q = _query([d], [(0, 0)])
    p = _plan(q)
    run = L.sdb_run_star_query_baseline
    assert run(C.byref(q), C.byref(p), 0, 0x1000, 0x2000, 10, None, 0, None) == 3           # CAPACITY
    assert run(C.byref(q), C.byref(p), 2, 0x1000, 0x2000, 100, 0x100, 1 << 20, None) == 1   # mode
    assert run(C.byref(q), C.byref(p), 1, 0x1000, 0x2000, 100, None, 0, None) == 1
    assert run(C.byref(q), C.byref(p), 0, 0x1000, 0x2000, 100, 0x180, 1 << 20, None) == 1   # alignment
    assert run(C.byref(q), C.byref(p), 1, 0x1000, 0x2000, 100, 0x100, 16, None) == 4        # too small


def test_finalize_scratch_and_validation():
    d = _fake_dim(radices=(250,))
    q = _query([d, d], [(0, 0), (1, 0)])
    p = _plan(q)
    nb = C.c_int64(0)
    assert sdb.lib().sdb_finalize_scratch_bytes(C.byref(p), C.byref(nb)) == 0
    assert nb.value == ((62_500 + 1023) // 1024) * 8
    L = sdb.lib()
    st = L.sdb_finalize_groups(C.byref(p), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 10, 0x6000, 0x7000,
                               nb.value, None)
    assert st == 3
    st = L.sdb_finalize_groups(C.byref(p), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 62_500, 0x6000,
                               0x7000, 8, None)
    assert st == 4


def test_batched_build_validates_every_table_before_any_launch():
    L = sdb.lib()
    descs = (sdb.SdbDimDesc * 2)(_desc(1000, "dense"), _desc(1000, "hash"))
    need = [sdb.dim_required_bytes(descs[0]), sdb.dim_required_bytes(descs[1])]
    ws = (C.c_void_p * 2)(0x100000, 0x40000000)          # never dereferenced: validation fails first
    outs = (sdb.SdbDim * 2)()

    def status(n, wsb, w=ws, d=descs):
        return sdb.STATUS[L.sdb_build_dims(n, d, w, (C.c_int64 * 2)(*wsb), None, outs)]

    assert status(-1, need) == "SDB_INVALID_ARG"
    assert status(7, need) == "SDB_INVALID_ARG"
    assert status(0, need) == "SDB_OK"                   # nothing to build
    # the second table's workspace is one byte short: nothing may launch
    assert status(2, [need[0], need[1] - 1]) == "SDB_WORKSPACE_TOO_SMALL"
    assert "dimension 1" in L.sdb_last_error().decode()
    bad = (C.c_void_p * 2)(0x100000, 0x40000010)          # not 256-byte aligned
    assert status(2, need, w=bad) == "SDB_INVALID_ARG"
    assert "dimension 1" in L.sdb_last_error().decode()
    d2 = (sdb.SdbDimDesc * 2)(_desc(1000, "dense"), _desc(1000, "dense"))
    d2[0].n_rows = -1
    assert status(2, need, d=d2) == "SDB_INVALID_ARG"
    assert "dimension 0" in L.sdb_last_error().decode()


def test_fused_events_hook_validation():
    L = sdb.lib()
    assert sdb.STATUS[L.sdb_set_fused_events(C.c_void_p(0x1000), None)] == "SDB_INVALID_ARG"
    assert sdb.STATUS[L.sdb_set_fused_events(None, C.c_void_p(0x1000))] == "SDB_INVALID_ARG"
    assert sdb.STATUS[L.sdb_set_fused_events(None, None)] == "SDB_OK"


def test_plan_block_and_items_per_lane():
    """Block size and items per lane: the planner's choice and the forcing rules."""
    d = _fake_dim()                                   # dense, too large for LDS: a device-memory lookup
    q = _query([d], [(0, 0)])
    p = _plan(q)
    assert (p.ipt, p.block) == (2, 512)
    q2 = _query([d, _fake_dim()], [(0, 0)])          # two device-memory lookups
    p2 = _plan(q2)
    assert (p2.ipt, p2.block) == (1, 1024)
    q3 = _query([d], [(0, 0)], align=False)          # 1-row items keep blocks of 256
    assert _plan(q3).block == 256
    for block, ipt, status in [(300, 0, "SDB_INVALID_ARG"), (1024, 4, "SDB_INVALID_ARG"), (128, 0, None)]:
        qq = _query([d], [(0, 0)])
        qq.force_block = block
        qq.force_ipt = ipt
        if status is None:
            assert _plan(qq).block == block
            continue
        with pytest.raises(sdb.SdbError) as e:
            _plan(qq)
        assert e.value.name == status
    qq = _query([d], [(0, 0)], align=False)
    qq.force_block = 1024
    with pytest.raises(sdb.SdbError) as e:
        _plan(qq)
    assert e.value.name == "SDB_INVALID_ARG"


def test_window_placement_and_validation():
    """LDS windows (SDB_LDS_WINDOW) on the host: the planner's choice under the
    overrides, its LDS and block size, and the run's refusal of inconsistent
    window fields before any launch."""
    big = _fake_dim(n_rows=3_000_000, n_pass=600_000, n_slots=3_000_000, with_bitmap=True)
    q = _query([big], [(0, 0)])
    q.force_window = 1
    p = _plan(q)
    assert p.stage_lds[0] == 5 and p.stage_defer[0] == -1 and p.block == 1024
    lo, slots = p.stage_window_lo[0], p.stage_window_slots[0]
    assert lo == 0 and slots % 128 == 0 and 500_000 < slots < 1_300_000
    assert abs(p.stage_window_cover[0] - slots / 3_000_000) < 1e-9     # no sample: the share of the key range
    assert p.terminal == 2 and p.lds_bytes == 16 * p.n_groups + slots // 8 <= 152 * 1024   # LDS group table first
    assert sdb.plan_summary(p)["stages"][0]["window"] == [0, slots]
    q.force_window = 4
    p4 = _plan(q)
    assert p4.stage_window_slots[0] == 512 and p4.lds_bytes == 16 * p4.n_groups + 64
    q.force_window = -1
    assert _plan(q).stage_lds[0] == 0
    q.force_window = 0                                   # 1,000 fact rows: too few for the staging copy
    assert _plan(q).stage_lds[0] == 0
    mid = _fake_dim(n_rows=300_000, n_pass=60_000, n_slots=300_000, with_bitmap=True)   # bitmap over 32 KB
    qm = _query([mid], [(0, 0)])
    qm.force_window = 1
    pm = _plan(qm)
    assert pm.stage_lds[0] == 5 and pm.stage_window_slots[0] == 300_032 and pm.stage_window_lo[0] == 0
    assert pm.stage_window_cover[0] == 1.0
    qm.force_lds = -1                                    # no LDS staging at all: no window either
    assert _plan(qm).stage_lds[0] == 0
    small = _fake_dim(n_rows=1000, n_pass=500, n_slots=1000, with_bitmap=True)
    qs = _query([small], [(0, 0)])
    qs.force_window = 1
    assert _plan(qs).stage_lds[0] == 1                   # a small map sits in LDS whole
    nobits = _fake_dim(n_rows=3_000_000, n_pass=600_000, n_slots=3_000_000)
    qn = _query([nobits], [(0, 0)])
    qn.force_window = 1
    assert _plan(qn).stage_lds[0] == 0                   # no pass bitmap, no window
    L = sdb.lib()
    q.force_window = 4
    for field, value in [("stage_window_lo", 64), ("stage_window_lo", -128), ("stage_window_slots", 100),
                         ("stage_window_slots", 0), ("stage_window_lo", 3_000_064), ("stage_defer", 1),
                         ("stage_defer", 0), ("stage_lds", 0)]:
        pb = sdb.SdbPlan.from_buffer_copy(p4)
        getattr(pb, field)[0] = value
        assert L.sdb_run_star_query(C.byref(q), C.byref(pb), 0x1000, 0x2000, 1 << 20, None, 0, None) == 1, \
            (field, value)
    filt = _query([big], [])                             # a filter-only table gets its window too
    filt.force_window = 4
    pf = _plan(filt)
    assert pf.stage_lds[0] == 5 and pf.stage_defer[0] == -1


def test_segment_validation():
    """A plan with stage orders per row range: the run checks the segments
    (cover the rows, start at multiples of 4096, each order a permutation,
    no eager loads) before any launch."""
    a = _fake_dim(n_rows=200_000, n_pass=40_000, n_slots=200_000)
    b = _fake_dim(n_rows=200_000, n_pass=100_000, n_slots=200_000)
    q = _query([a, b], [(0, 0)], n_fact=100_000)
    q.force_order = 1
    p = _plan(q)
    assert p.n_segments == 1 and p.segment_start[0] == 0 and p.segment_start[1] == 100_000
    assert list(p.segment_order[0][:2]) == [0, 1]
    L = sdb.lib()

    def status(pl):
        return L.sdb_run_star_query(C.byref(q), C.byref(pl), 0x1000, 0x2000, 1 << 20, 0x100000,
                                    1 << 30, None)

    good = sdb.SdbPlan.from_buffer_copy(p)
    good.n_segments = 2
    good.segment_start[1], good.segment_start[2] = 8192, 100_000
    good.segment_order[1][0], good.segment_order[1][1] = 1, 0
    if not GPU_PRESENT:
        assert status(good) != 1, sdb.lib().sdb_last_error()    # valid: the launch itself fails without a GPU
    assert sdb.plan_summary(good)["segments"][1] == {"rows": [8192, 100_000], "order": [1, 0]}
    for mutate in [lambda x: x.segment_start.__setitem__(1, 8000),        # not a multiple of 4096
                   lambda x: x.segment_start.__setitem__(2, 99_999),      # does not reach n_fact
                   lambda x: x.segment_start.__setitem__(1, 0),           # empty segment
                   lambda x: x.segment_order[1].__setitem__(0, 0),        # not a permutation
                   lambda x: x.segment_order[1].__setitem__(1, 5),
                   lambda x: setattr(x, "n_segments", 9),
                   lambda x: setattr(x, "eager", 1)]:
        bad = sdb.SdbPlan.from_buffer_copy(good)
        mutate(bad)
        assert status(bad) == 1
    for field, value in [("force_segments", 2), ("force_segments", -2), ("force_prefilter", 2), ("force_prefilter", -2)]:
        qb = sdb.SdbQuery.from_buffer_copy(q)
        setattr(qb, field, value)
        assert L.sdb_plan_star_query(C.byref(qb), None, 0, None, C.byref(sdb.SdbPlan())) == 1
