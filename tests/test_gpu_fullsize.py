"""GPU parity at the full workload sizes (600M fact rows), in the launch
configuration the benchmark times.

The oracle cannot scan 600M rows in seconds, so three checks stand in:

* every group of the full-size result against an independent numpy
  computation by direct indexing (dimension keys are row numbers, or a
  permutation for c5): group counts with ``np.bincount``, sums as two
  float64 ``np.bincount``s of the 16-bit halves of each value (every partial
  sum stays below 2^53, so both are exact), in chunks on a thread pool;
* the oracle itself on a window of the same device columns starting at an
  unaligned row (the kernel's 1-row item path);
* row-range additivity: three unaligned slices of the full columns add up to
  the full result.
"""

import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import datagen
from gpu_util import assert_same, oracle_rows, require_gpu

pytestmark = pytest.mark.gpu

CHUNK = 20_000_000


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _log(*a):
    print(*a, flush=True)


def _pass_mask(table, preds):
    ok = np.ones(next(iter(table.values())).size, dtype=bool)
    for p in preds:
        x = table[p["col"]].astype(np.int64)
        if p["op"] == "eq":
            ok &= x == p["lo"]
        elif p["op"] == "between":
            ok &= (x >= p["lo"]) & (x <= p["hi"])
        else:
            raise AssertionError(f"unexpected op {p['op']}")
    return ok


def independent_groups(w):
    """(keys, sums, counts) by direct indexing, for the full-size workloads."""
    q = w.query
    joins = q["joins"]
    # per join: slot of each key, pass flag per slot, payload values per slot
    info = []
    for jd in joins:
        t = w.dims[jd["dim"]]
        keys = t[w.dim_keys[jd["dim"]]].astype(np.int64)
        kmin, kmax = int(keys.min()), int(keys.max())
        slot_row = np.full(kmax - kmin + 1, -1, dtype=np.int64)
        slot_row[keys - kmin] = np.arange(keys.size)
        ok = _pass_mask(t, jd["preds"])
        info.append((jd, t, kmin, slot_row, ok))
    gkeys = q["group_by"]
    radix, kmins, stride = [], [], []
    for dim, col in gkeys:
        jd, t, kmin, slot_row, ok = next(x for x in info if x[0]["dim"] == dim)
        vals = t[col][ok]
        radix.append(int(vals.max() - vals.min() + 1))
        kmins.append(int(vals.min()))
    g = 1
    for rdx in reversed(radix):
        stride.insert(0, g)
        g *= rdx
    agg = q["agg"]

    def chunk(lo):
        hi = min(w.n_fact, lo + CHUNK)
        live = np.ones(hi - lo, dtype=bool)
        gid = np.zeros(hi - lo, dtype=np.int64)
        for jd, t, kmin, slot_row, ok in info:
            fk = w.fact[jd["fact_key"]][lo:hi].astype(np.int64) - kmin
            inr = (fk >= 0) & (fk < slot_row.size)
            row = np.where(inr, slot_row[np.clip(fk, 0, slot_row.size - 1)], -1)
            hit = row >= 0
            live &= hit & ok[np.where(hit, row, 0)]
            for k, (dim, col) in enumerate(gkeys):
                if dim == jd["dim"]:
                    gid += (t[col][np.where(hit, row, 0)].astype(np.int64) - kmins[k]) * stride[k]
        a = w.fact[agg["a"]][lo:hi].astype(np.int64)
        if agg["kind"] == "col":
            v = a
        elif agg["kind"] == "sub":
            v = a - w.fact[agg["b"]][lo:hi].astype(np.int64)
        else:
            raise AssertionError(agg["kind"])
        gl = gid[live]
        vl = v[live]
        counts = np.bincount(gl, minlength=g)
        # exact sums from float64 bincounts of 16-bit halves (every partial sum < 2^53)
        lo16 = (vl & 0xFFFF).astype(np.float64)
        hi16 = (vl >> 16).astype(np.float64)
        s_lo = np.bincount(gl, weights=lo16, minlength=g)
        s_hi = np.bincount(gl, weights=hi16, minlength=g)
        assert np.abs(s_lo).max(initial=0) < 2.0**53 and np.abs(s_hi).max(initial=0) < 2.0**53
        return counts, s_hi.astype(np.int64) * 65536 + s_lo.astype(np.int64)

    sums = np.zeros(g, dtype=np.int64)
    counts = np.zeros(g, dtype=np.int64)
    with ThreadPoolExecutor(max_workers=8) as ex:
        for c, s in ex.map(chunk, range(0, w.n_fact, CHUNK)):
            counts += c
            sums += s
    present = np.flatnonzero(counts)
    keys = np.stack([(present // stride[k]) % radix[k] + kmins[k] for k in range(len(gkeys))], axis=1)
    return [(tuple(int(x) for x in kk), int(s), int(c))
            for kk, s, c in zip(keys, sums[present], counts[present])]


def _run(fact_dev, dims_dev, w, lo=None, hi=None):
    from paper_2607_07632_amd import sdb
    import torch
    cols = fact_dev if lo is None else {k: v[lo:hi] for k, v in fact_dev.items()}
    tables = sdb.build_dims(dims_dev, w.dim_keys, w.query)
    q = sdb.StarQuery(cols, tables, w.query)
    res = q.execute()
    torch.cuda.synchronize()
    return res, q


@pytest.mark.parametrize("name", ["c2_join_group", "c3_star3", "c4_star4_zipf", "c5_hash_stress"])
def test_full_size(name):
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

    # 1. every group against the direct-indexing computation
    t0 = time.time()
    want = independent_groups(w)
    _log(f"{name}: independent full-size groups in {time.time() - t0:.1f} s")
    assert_same(full.as_rows(), want, f"{name} full size")

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


def test_more_than_2g_rows():
    """c3's query over 2^31 + 4,099 fact rows drawn on the device: 64-bit row
    indexing end to end. Every group's count and sum against torch (gathers,
    masks and bincount, in chunks; every partial sum stays below 2^53, so the
    float64 weights are exact), and two row ranges, the second starting at an
    unaligned row (1-row items), add up to the whole."""
    import torch
    from paper_2607_07632_amd import sdb
    w = datagen.make_workload("c3_star3", n_fact=0)
    q = w.query
    n = 2**31 + 4099
    g = torch.Generator(device="cuda")
    g.manual_seed(26077632)
    spans = {"cust_key": (0, 3_000_000), "supp_key": (0, 200_000), "date_key": (0, 2556), "revenue": (1, 1_000_001)}
    fact = {c: torch.randint(lo, hi, (n,), generator=g, device="cuda", dtype=torch.int32)
            for c, (lo, hi) in spans.items()}
    dims = {d: {c: torch.from_numpy(a).cuda() for c, a in t.items()} for d, t in w.dims.items()}
    _log(f"2g rows: {n} rows drawn on the device")

    # per join: pass flag and payload value by key (keys are 0 .. rows-1 here)
    per_join = []
    for jd in q["joins"]:
        t = w.dims[jd["dim"]]
        keys = t[w.dim_keys[jd["dim"]]]
        assert np.array_equal(keys, np.arange(keys.size))
        ok = _pass_mask(t, jd["preds"])
        per_join.append((jd, torch.from_numpy(ok).cuda()))
    radix, kmin, vals = [], [], []
    for dim, col in q["group_by"]:
        jd, ok = next(x for x in per_join if x[0]["dim"] == dim)
        v = w.dims[dim][col][ok.cpu().numpy()]
        kmin.append(int(v.min()))
        radix.append(int(v.max()) - int(v.min()) + 1)
        vals.append((dim, jd["fact_key"], torch.from_numpy(w.dims[dim][col].astype(np.int64)).cuda()))
    stride = [int(np.prod(radix[k + 1:])) for k in range(len(radix))]
    G = int(np.prod(radix))
    counts = torch.zeros(G, dtype=torch.int64, device="cuda")
    sums = torch.zeros(G, dtype=torch.float64, device="cuda")
    chunk = 1 << 28
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        live = torch.ones(hi - lo, dtype=torch.bool, device="cuda")
        for jd, ok in per_join:
            live &= ok[fact[jd["fact_key"]][lo:hi].long()]
        gid = torch.zeros(hi - lo, dtype=torch.int64, device="cuda")
        for k, (dim, fk, v) in enumerate(vals):
            gid += (v[fact[fk][lo:hi].long()] - kmin[k]) * stride[k]
        gl = gid[live]
        counts += torch.bincount(gl, minlength=G)
        sums += torch.bincount(gl, weights=fact["revenue"][lo:hi][live].double(), minlength=G)
    assert float(sums.max()) < 2.0**53
    present = torch.nonzero(counts).flatten().cpu().numpy()
    c_h, s_h = counts.cpu().numpy(), sums.cpu().numpy().astype(np.int64)
    want = [(tuple(int((p // stride[k]) % radix[k] + kmin[k]) for k in range(len(radix))), int(s_h[p]), int(c_h[p]))
            for p in present]
    _log(f"2g rows: torch reference has {len(want)} groups")

    tables = sdb.build_dims(dims, w.dim_keys, q)
    full = sdb.StarQuery(fact, tables, q).execute()
    assert_same(full.as_rows(), want, "2^31 + 4099 rows")
    _log("2g rows: full result agrees")

    cut = 2**30 + 3
    acc = {}
    for a, b in [(0, cut), (cut, n)]:
        part = sdb.StarQuery({k: v[a:b] for k, v in fact.items()}, tables, q).execute()
        for k, s, c in part.as_rows():
            s0, c0 = acc.get(k, (0, 0))
            acc[k] = (s0 + s, c0 + c)
    assert sorted((k, s, c) for k, (s, c) in acc.items()) == full.as_rows()
    _log("2g rows: row ranges add up")
    del fact
    torch.cuda.empty_cache()
