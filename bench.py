#!/usr/bin/env python3
"""Benchmark of the fused star-schema query on one MI355X.

One step is one pass of the whole hot path over the resident fact table:
build every dimension lookup table, plan (a sampling kernel orders the
stages), the fused probe-filter-aggregate kernel, and the device compaction of
the group table (its size read back to the host). Fact columns are generated
once, uploaded, and stay in HBM; the timed region starts with them resident.

Default workload: c3_star3, 600M fact rows (int32 cust_key, supp_key,
date_key, revenue), customer 3M / supplier 200k / date 2556 rows, SUM(revenue)
GROUP BY (customer city, supplier city, year).

Prints one JSON line. `value` = fact rows per second of the whole step.
`roofline` rates the fused kernel on B_alg, the fact-column bytes the method
must move at 128-byte line granularity (4 bytes per column times the fraction
of lines holding a row still live where the plan first reads that column,
measured on the first rows of the same data), over its mean duration timed
with HIP events that the library records on the kernel's stream right around
its launch; `frac_b_dense` rates it on all fact-column bytes, and
`frac_run_window` rates the whole run (output fill, fused kernel, terminal
passes). `cpu_baseline` times the CPU oracle over the whole fact table on one
worker process per host core (at most 16), and the full GPU result is compared
with it group by group; `cpu_oracle_one_core` times it in one process on the
first rows (c1 whole, c2 and c3 8M rows). `configs` holds a compact record of
each other workload (run and kernel times, roofline fractions, oracle parity
over its first 2^27 fact rows, the whole table for c1 and c2).
"""

from __future__ import annotations

import argparse
import copy
import functools
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# The paper's own measurements of the fused star-query path, on SSB at scale
# factor 100 and on other GPUs: context only, not a target (the workloads
# here are synthetic stand-ins for the SSB query shapes).
PAPER_CONTEXT = {
    "note": "the paper's measurements on SSB SF100 (600,043,265 fact rows) on other GPUs; context only",
    "nvidia_l40s": {
        "dram_peak_GBps": 864,
        "q3_1_three_dimension_star_warm_ms": {"SHADB-Opt": 8.49, "SYCLDB-Opt": 8.41, "Crystal": 14.07},
        "q4_1_four_dimension_star_warm_ms": {"SHADB-Opt": 10.24, "SYCLDB-Opt": 13.32, "Crystal": 22.23},
        "suite_total_warm_ms": {"SHADB-Opt": 77.94},
        "source": "Table 1 (section 2.2) and the SF100 L40S figure of section 5.2",
    },
    "amd_mi210": {
        "hbm_peak_GBps": 1600,
        "fused_kernel_TBps": {"Q1.1 scan": 0.85, "Q1.3 scan": 1.13, "Q4.1 join, group terminal": 0.65,
                              "Q4.3 join, group terminal": 0.35},
        "synthesized_scan_kernels_TBps": 0.95,
        "source": "section 5.3 and its MI210 counter table",
    },
}
ONE_CORE_ROWS = 8_000_000        # rows of the one-core oracle timings (c1 whole, c2 and c3 a head)
# the fused kernel's source: its template and the device helpers it uses
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2607_07632_amd", "csrc", f) for f in ("sdb_fused.h", "sdb_device.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        h.update(open(path, "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload: str):
    """HBM bytes per fused-kernel launch from a committed counter summary, or None
    when the summary is missing or was taken from a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"star_fused_{workload}_pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_source_hash():
        return None
    return float(m_bytes.group(1))


def _in_range(x, p) -> "np.ndarray":
    """Predicate dict {op, lo, hi} on an int64 array (measurement helper)."""
    op, lo, hi = p["op"], p["lo"], p.get("hi")
    if op == "between":
        return (x >= lo) & (x <= hi)
    return {"eq": x == lo, "ne": x != lo, "lt": x < lo, "le": x <= lo, "gt": x > lo, "ge": x >= lo}[op]


def b_alg_per_row(sample: dict, dims: dict, dim_keys: dict, query: dict, plan_info: dict) -> float:
    """B_alg: 4 bytes per fact column times the fraction of 128-byte lines (32
    rows) holding a row that is still live where the plan first reads that
    column, on the sample rows."""
    import numpy as np
    m = next(iter(sample.values())).size
    m32 = m // 32 * 32
    live = np.ones(m, dtype=bool)
    seen, total = set(), 0.0

    def read(col):
        nonlocal total
        if col not in seen:
            seen.add(col)
            total += 4.0 * float(live[:m32].reshape(-1, 32).any(axis=1).mean())

    for st in plan_info["stages"]:
        if st["kind"] == "pred":
            p = query["fact_preds"][st["index"]]
            read(p["col"])
            live &= _in_range(sample[p["col"]].astype(np.int64), p)
        else:
            j = query["joins"][st["index"]]
            read(j["fact_key"])
            t = dims[j["dim"]]
            keys = t[dim_keys[j["dim"]]].astype(np.int64)
            ok = np.ones(keys.size, dtype=bool)
            for p in j.get("preds", []):
                ok &= _in_range(t[p["col"]].astype(np.int64), p)
            order = np.argsort(keys, kind="stable")
            fk = sample[j["fact_key"]].astype(np.int64)
            pos = np.clip(np.searchsorted(keys[order], fk), 0, keys.size - 1)
            live &= (keys[order][pos] == fk) & ok[order][pos]
    agg = query["agg"]
    read(agg["a"])
    if agg["kind"] != "col":
        read(agg["b"])
    return total


# The plan features of the fused pass added one at a time, each rung a set of
# planner overrides (the last rung is the planner's own choice).
# the rungs before the key-range rewrite keep every probe a lookup, unsliced, without LDS windows
_NR = {"range": -1, "slice": -1, "window": -1}
ABLATION_RUNGS = [
    ("kernel at a time: flags and group ids through HBM; hash tables; query order",
     {"order": True, "baseline": "per_operator", "tables": "hash", "slice": -1}),
    ("one kernel; operators hand off through HBM", {"order": True, "baseline": "global_handoff", "tables": "hash",
                                                    "slice": -1}),
    ("+ register table; 1-row items", {"order": True, "lds": -1, "vector": -1, "ipt": 1, "terminal": "global",
                                       "xcd": -1, "block": 256, "tables": "hash"} | _NR),
    ("+ packed direct-mapped maps", {"order": True, "lds": -1, "vector": -1, "ipt": 1,
                                     "terminal": "global", "xcd": -1, "block": 256} | _NR),
    ("+ 4-row items (128-bit loads)", {"order": True, "lds": -1, "ipt": 1, "terminal": "global", "xcd": -1,
                                       "block": 256} | _NR),
    ("+ two items per lane", {"order": True, "lds": -1, "ipt": 2, "terminal": "global", "xcd": -1,
                              "block": 256} | _NR),
    ("+ LDS-staged maps and bitmaps", {"order": True, "lds": 2, "ipt": 2, "terminal": "global", "xcd": -1,
                                      "block": 256} | _NR),
    ("+ sampled stage order", {"lds": 2, "ipt": 2, "terminal": "global", "xcd": -1, "block": 256} | _NR),
    ("+ per-XCD group tables", {"lds": 2, "ipt": 2, "terminal": "global", "block": 256} | _NR),
    ("+ probes of one contiguous passing key range run as BETWEEN", {"lds": 2, "ipt": 2, "terminal": "global",
                                                                     "block": 256, "range": 1, "slice": -1,
                                                                     "window": -1}),
    ("planner's choice (terminal, block size, rank tables)", {"slice": -1, "unroll": -1, "window": -1}),
    ("+ stage loop written out (plans without a hash probe)", {"slice": -1, "window": -1}),
    ("+ LDS window over the busiest device-memory map", {"slice": -1}),
    ("+ a hash probe over 2 MiB table slices", {"prefilter": -1}),
    ("+ rows the table's pass filter rejects dropped before the slicing (planner's choice)", {}),
]


def ablation_ladder(sdb, fact, dims, wdims, query, stream, base_force) -> list:
    """Run-window time (fill, fused kernel, terminal passes) of every rung;
    every rung's group table must equal the planner's own."""
    import numpy as np
    import torch
    out, ref = [], None
    for name, f in list(ABLATION_RUNGS)[::-1]:
        force = dict(base_force)
        force.update(f)
        baseline = force.pop("baseline", None)
        rq = query
        if force.pop("tables", None) == "hash":
            rq = copy.deepcopy(query)
            for jd in rq["joins"]:
                jd["kind"] = "hash"
        if rq.get("group_by") == [] and force.get("terminal") == "global":
            force.pop("terminal")
        tabs = sdb.build_dims(dims, wdims.dim_keys, rq)
        try:
            q = sdb.StarQuery(fact, tabs, rq, force)
            plan = q.plan()
        except sdb.SdbError as e:
            out.append({"rung": name, "force": f, "run_ms": float("nan"), "error": str(e), "plan": None})
            continue
        sums, counts = q.alloc_outputs(plan)
        if baseline:
            scratch = q.baseline_scratch(sums.device)
            run = functools.partial(q.run_baseline, baseline)
        else:
            scratch = q.run_scratch(plan)
            run = q.run
        for _ in range(2):
            run(sums, counts, plan=plan, scratch=scratch)
        torch.cuda.synchronize()
        ts = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            run(sums, counts, plan=plan, scratch=scratch)
            b.record(stream)
            b.synchronize()
            ts.append(a.elapsed_time(b))
        tab = (sums.cpu().numpy(), counts.cpu().numpy())
        if ref is None:
            ref = tab
        same = bool(np.array_equal(tab[0], ref[0]) and np.array_equal(tab[1], ref[1]))
        info = sdb.plan_summary(plan, rq)
        shape = {k: info[k] for k in ("terminal", "ipt", "vector", "block", "xcd_copies")}
        stages = [(s["name"], s.get("table", "pred")) for s in info["stages"]]
        if baseline:
            shape = {"terminal": baseline}
            stages = [(nm, "pred" if t == "pred" else "device") for nm, t in stages]
        out.append({"rung": name, "force": f, "run_ms": float(np.mean(ts)), "same_result": same,
                    "plan": shape | {"stages": stages}})
        if not same:
            raise AssertionError(f"ablation rung {name!r} changed the result")
    return out[::-1]


def query_columns(query: dict) -> list:
    """Fact columns the query reads, in first-use order."""
    cols = [p["col"] for p in query.get("fact_preds", [])] + [j["fact_key"] for j in query.get("joins", [])]
    cols += [query["agg"]["a"]] + ([query["agg"]["b"]] if query["agg"].get("b") else [])
    return list(dict.fromkeys(cols))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def upload_fact(cfg_name: str, n: int, device) -> dict:
    """Generate each fact column into one pinned host buffer and copy it to HBM."""
    import torch
    import datagen
    from datagen.star import CONFIGS
    cfg = CONFIGS[cfg_name]
    staging = torch.empty(n, dtype=torch.int32, pin_memory=True)
    out = {}
    for col in cfg.fact_cols:
        t0 = time.perf_counter()
        datagen.fact_column(cfg_name, col.name, 0, n, out=staging.numpy())
        d = torch.empty(n, dtype=torch.int32, device=device)
        d.copy_(staging, non_blocking=True)
        torch.cuda.synchronize()
        out[col.name] = d
        log(f"  fact column {col.name}: {n} rows in {time.perf_counter() - t0:.1f} s")
    del staging
    return out


def stream_read_reference(sdb, cols: list, n: int, stream, achieved: float) -> dict:
    """A plain streaming read of the query's fact columns (sdb_read_columns),
    best of 1-4 blocks of 512 per CU: the practical ceiling of the stream."""
    import numpy as np
    import torch
    acc = torch.zeros(1, dtype=torch.int64, device=cols[0].device)
    best = None
    for per_cu in (1, 2, 3, 4):
        sdb.read_columns(cols, acc, blocks_per_cu=per_cu)
        torch.cuda.synchronize()
        rd = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            sdb.read_columns(cols, acc, blocks_per_cu=per_cu)
            b.record(stream)
            b.synchronize()
            rd.append(a.elapsed_time(b))
        if best is None or np.mean(rd) < best[1]:
            best = (per_cu, float(np.mean(rd)))
    gbps = n * 4 * len(cols) / (best[1] * 1e-3) / 1e9
    log(f"[bench] streaming read of {len(cols)} columns: {best[1]:.4f} ms, {gbps:.0f} GB/s "
        f"({best[0]} blocks per CU)")
    return {"ms": best[1], "GBps": gbps, "frac_of_peak": gbps / HBM_PEAK_GBPS,
            "fused_frac_of_stream_read": achieved / gbps,
            "what": f"sdb_read_columns over the query's {len(cols)} fact columns (128-bit loads), "
                    f"best of 1-4 blocks of 512 per CU ({best[0]})"}


def graph_replay_ms(q, sums, counts, plan, fin_out, stream, n_groups: int) -> float:
    """The run and the compaction captured in one HIP graph and replayed (no
    host launch gaps); the replay must reproduce the group count."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    graph = torch.cuda.CUDAGraph()
    scratch = q.run_scratch(plan)
    with torch.cuda.graph(graph, stream=side):
        q.run(sums, counts, plan=plan, scratch=scratch)
        q.finalize(sums, counts, plan=plan, outputs=fin_out)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    if int(fin_out[3].item()) != n_groups:
        raise AssertionError("graph replay changed the number of groups")
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(10):
        graph.replay()
    b.record(stream)
    b.synchronize()
    ms = a.elapsed_time(b) / 10
    log(f"[bench] run + finalize replayed from a HIP graph: {ms:.4f} ms")
    return ms


def end_to_end(sdb, build_tables, fact, query, force, sums, counts, fin_out) -> dict:
    """One query end to end (builds, plan, run, compaction, copy of the groups
    to the host), and an MD5 digest of the whole result (keys, sums, counts as
    little-endian bytes) for comparing runs across machines, the way the paper
    compares its outputs."""
    import numpy as np
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    q = sdb.StarQuery(fact, build_tables(), query, force)
    q.plan()
    q.run(sums, counts)
    k, s, c, nout, _ = q.finalize(sums, counts, outputs=fin_out)
    m = int(nout.item())
    host = (k[:m].cpu(), s[:m].cpu(), c[:m].cpu())
    ms = 1000.0 * (time.perf_counter() - t0)
    digest = hashlib.md5()
    for t in host:
        digest.update(np.ascontiguousarray(t.numpy()).tobytes())
    return {"e2e_ms": ms, "e2e_includes": f"build + plan + run + finalize + copy of {m} groups to the host",
            "result_md5": digest.hexdigest()}


def mall_cold_ms(q, sums, counts, plan, stream, dev) -> float:
    """Run time with a 1 GiB write before every run, which evicts the columns
    from the 256 MB cache."""
    import numpy as np
    import torch
    flush = torch.empty(1 << 28, dtype=torch.int32, device=dev)
    scratch = q.run_scratch(plan)
    cold = []
    for _ in range(5):
        flush.fill_(7)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        q.run(sums, counts, plan=plan, scratch=scratch)
        b.record(stream)
        b.synchronize()
        cold.append(a.elapsed_time(b))
    return float(np.mean(cold))


def copy_calibration(dev) -> None:
    """Three device copies of exactly 1 GiB: the reference launches that scale
    the HBM byte counters in the profiles."""
    import torch
    src = torch.empty(1 << 28, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("[bench] copy calibration: 3 x 1 GiB device-to-device copies done")


def host_sample(fact: dict, rows: int) -> dict:
    """The first ``rows`` rows of every device column, on the host."""
    return {k: v[:rows].cpu().numpy() for k, v in fact.items()}


def device_column_sums(fact: dict) -> dict:
    import torch
    return {k: int(v.sum(dtype=torch.int64).item()) for k, v in fact.items()}


def one_core_oracle(cfg_name: str, rows: int) -> dict:
    """The oracle in this process, on one core, over the first ``rows`` fact
    rows (generation excluded from the time)."""
    from oracle import ranges
    _, _, secs = ranges.range_task(cfg_name, 0, rows)
    log(f"[bench] {cfg_name}: oracle on one core over the first {rows} rows: {secs:.1f} s")
    return {"value": rows / secs, "unit": "fact rows/s", "cores": 1, "kind": "oracle", "rows": rows,
            "secs": secs, "sample": f"the first {rows} fact rows of {cfg_name}, one process, generation excluded"}


def cpu_baseline_leg(cfg_name: str, n: int, gpu_rows: list, fact: dict) -> dict:
    """The oracle over all n fact rows, one row range per worker process (one
    per host core, at most 16), the oracle phases started together once every
    worker has generated its rows; the full GPU result compared with it group
    by group, and the workers' column sums with the device columns'."""
    from oracle import ranges
    workers = ranges.worker_count()
    res, col_sums, info = ranges.run_timed(cfg_name, n, workers)
    same_rows = col_sums == device_column_sums(fact)
    parity = same_rows and gpu_rows == res.as_rows()
    per_core = n / sum(info["worker_oracle_s"])
    log(f"[bench] oracle over all {n} rows on {info['workers']} processes: {info['wall_s']:.1f} s "
        f"(merge {info['merge_s']:.1f} s); the full GPU result {'equals' if parity else 'DIFFERS FROM'} it")
    return {
        "cpu_baseline": {
            "value": n / info["wall_s"],
            "unit": "fact rows/s",
            "cores": info["workers"],
            "kind": "oracle",
            "sample": f"all {n} fact rows of {cfg_name} and its full dimension tables: the numpy oracle "
                      f"on {info['workers']} row ranges, one worker process each, merged group by group; "
                      f"{info['wall_s']:.1f} s wall clock from the first range's start to the merge's end "
                      f"(generation excluded)",
            "cpu": cpu_model(),
            "host_cores_in_affinity": len(os.sched_getaffinity(0)),
            "rows_per_s_per_core": per_core,
        },
        "cpu_oracle_one_core": one_core_oracle(cfg_name, min(n, ONE_CORE_ROWS)),
        "parity_full_table": parity,
        "parity_detail": {"groups": len(gpu_rows), "oracle_groups": len(res.sums),
                          "oracle_live_rows": int(res.n_live), "oracle_saw_device_rows": same_rows},
    }


def config_record(sdb, name: str, ex, dev, runs: int = 10, balg_rows: int = 16_000_000,
                  parity_rows: int = 1 << 27, compare: dict | None = None) -> dict:
    """One workload measured compactly: table builds, the run window and the
    fused kernel (HIP events), roofline fractions on B_alg and B_dense, and the
    GPU result against the oracle over the first min(N, parity_rows) fact rows
    (the whole table for c1 and c2; the full-size tests compare all 600M rows
    of c4 and c5)."""
    import numpy as np
    import torch
    import datagen
    from datagen.star import CHUNK, CONFIGS
    cfg = CONFIGS[name]
    n = cfg.n_fact
    log(f"[bench] {name}: {n} fact rows")
    fact = upload_fact(name, n, dev)
    w = datagen.make_workload(name, n_fact=0)
    dims = {d: {c: torch.from_numpy(a).to(dev) for c, a in t.items()} for d, t in w.dims.items()}
    query = w.query
    stream = torch.cuda.current_stream()
    build_ms = []
    for _ in range(4):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        tabs = sdb.build_dims(dims, w.dim_keys, query)
        torch.cuda.synchronize()
        build_ms.append(1000.0 * (time.perf_counter() - t0))
    q = sdb.StarQuery(fact, tabs, query)
    plan = q.plan()
    sums, counts = q.alloc_outputs(plan)
    scratch = q.run_scratch(plan)
    for _ in range(2):
        q.run(sums, counts, plan=plan, scratch=scratch)
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(runs)]
    torch.cuda.synchronize()
    for ev in evs:
        sdb.set_fused_events(ev[0], ev[1])
        ev[2].record(stream)
        q.run(sums, counts, plan=plan, scratch=scratch)
        ev[3].record(stream)
    sdb.set_fused_events()
    torch.cuda.synchronize()
    kernel_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    run_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    got = q.execute(replan=False).as_rows()
    versus = None
    if compare:
        # the same query under planner overrides, timed the same way (context)
        qc = sdb.StarQuery(fact, tabs, query, compare)
        pc = qc.plan()
        sc, cc = qc.alloc_outputs(pc)
        scr = qc.run_scratch(pc)
        qc.run(sc, cc, plan=pc, scratch=scr)
        evc = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(runs)]
        torch.cuda.synchronize()
        for ev in evc:
            sdb.set_fused_events(ev[0], ev[1])
            ev[2].record(stream)
            qc.run(sc, cc, plan=pc, scratch=scr)
            ev[3].record(stream)
        sdb.set_fused_events()
        torch.cuda.synchronize()
        same = qc.execute(replan=False).as_rows() == got
        versus = {"force": compare, "fused_kernel_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evc])),
                  "run_ms": float(np.mean([e[2].elapsed_time(e[3]) for e in evc])), "same_result": same,
                  "plan": sdb.plan_summary(pc, query)}
        del qc, sc, cc, scr
    info = sdb.plan_summary(plan, query)
    b_dense = 4 * int(q.q.n_cols)
    b_alg = b_alg_per_row(host_sample(fact, min(n, balg_rows)), w.dims, w.dim_keys, query, info)
    parity = same_rows = None
    m = min(n, parity_rows)
    if ex is not None:
        from oracle import ranges
        t0 = time.perf_counter()
        head = {k: v[:m] for k, v in fact.items()}
        got_m = got if m == n else sdb.StarQuery(head, tabs, query).execute().as_rows()
        want, col_sums = ranges.run(name, m, ex, 2 * CHUNK)
        same_rows = col_sums == device_column_sums(head)
        parity = same_rows and got_m == want.as_rows()
        log(f"[bench] {name}: oracle over the first {m} rows in {time.perf_counter() - t0:.1f} s: "
            f"{'equal' if parity else 'DIFFERENT'}")
    log(f"[bench] {name}: fused {kernel_ms:.4f} ms, run {run_ms:.4f} ms, builds {min(build_ms):.3f} ms")
    rec = {
        "workload": f"{name}: {cfg.describe}",
        "fact_rows": n,
        "plan": info,
        "runs": runs,
        "fused_kernel_ms": kernel_ms,
        "run_ms": run_ms,
        "build_ms_min": min(build_ms),
        "run_rows_per_s": n / (run_ms * 1e-3),
        "b_dense_bytes_per_row": b_dense,
        "b_alg_bytes_per_row": b_alg,
        "frac_b_alg_fused": n * b_alg / (kernel_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "frac_b_alg_run_window": n * b_alg / (run_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "frac_b_dense_fused": n * b_dense / (kernel_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "groups": len(got),
        "oracle_parity": parity,
        "oracle_parity_rows": m if ex is not None else 0,
        "oracle_saw_device_rows": same_rows,
    }
    if versus:
        rec["versus"] = versus
    if ex is not None and name in ("c1_scalar_scan", "c2_join_group"):
        rec["cpu_oracle_one_core"] = one_core_oracle(name, min(n, ONE_CORE_ROWS))
    if plan.slice_bits:
        rec["fused_window_covers"] = "count pass + scatter pass + fused kernel (hash probe over table slices)"
    if any(sdb.dim_info(t)["kind"] == "hash" for t in tabs):
        rec["probes_per_s_run"] = n / (run_ms * 1e-3)
        rec["build_reported_separately"] = True
    del fact, q, sums, counts, scratch, tabs
    torch.cuda.empty_cache()
    return rec


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c3_star3")
    ap.add_argument("--rows", type=int, default=None, help="fact rows (default: the workload's size)")
    ap.add_argument("--balg-rows", type=int, default=40_000_000,
                    help="first fact rows on which B_alg (line-granular algorithmic bytes) is measured")
    ap.add_argument("--no-cpu", action="store_true",
                    help="skip the oracle leg (CPU baseline and every comparison with the oracle)")
    ap.add_argument("--no-configs", action="store_true", help="skip the compact records of the other workloads")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (scale for HBM byte counters)")
    ap.add_argument("--force", default="", help="planner overrides, e.g. ipt=4,vector=1,terminal=global")
    ap.add_argument("--ablation", default=None, metavar="PATH",
                    help="also time the fused-plan ablation ladder and write it as JSON to PATH")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported (sharding the fact rows "
              "over GPUs would need one all-reduce of the group table per query, which is not built)",
              file=sys.stderr)
        return 2

    if not args.no_cpu:
        # the oracle's worker processes fork from a server started before any GPU call
        from oracle import ranges
        ranges.start_forkserver()

    import numpy as np
    import torch

    import datagen
    from datagen.star import CONFIGS
    from paper_2607_07632_amd import sdb

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        return 1
    sdb.lib()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.config]
    n = cfg.n_fact if args.rows is None else int(args.rows)
    force = {}
    for kv in filter(None, args.force.split(",")):
        k, v = kv.split("=")
        force[k] = v if k == "terminal" else (v == "1" if k == "order" else int(v))

    log(f"[bench] {args.config}: {n} fact rows; generating and uploading")
    t0 = time.perf_counter()
    fact = upload_fact(args.config, n, dev)
    wdims = datagen.make_workload(args.config, n_fact=0)
    dims = {d: {c: torch.from_numpy(a).to(dev) for c, a in t.items()} for d, t in wdims.dims.items()}
    query = wdims.query
    log(f"[bench] data resident after {time.perf_counter() - t0:.1f} s")

    # Two slots of buffers (dimension workspaces, group tables, compaction
    # outputs) so that step i builds and plans on its slot's own stream as
    # soon as step i-1's fused kernel is done, while that step's terminal
    # passes and compaction still run: the host synchronizations of the
    # builds and of the planner's sample overlap the previous run instead of
    # idling the GPU, and no build kernel shares the GPU with a fused kernel,
    # whose HIP-event time therefore stays its own. Runs and compactions all
    # go to one stream, in step order. The library allocates nothing itself.
    # Each slot marshals its build arguments and its query once (PreparedDims,
    # StarQuery): a step reruns every build, the plan with its sampling, the
    # run and the compaction, and only the host-side argument structs persist.
    stream = torch.cuda.current_stream()
    slots = []
    for _ in range(2):
        pd = sdb.PreparedDims(dims, wdims.dim_keys, query)
        tabs = pd.build()
        qs = sdb.StarQuery(fact, tabs, query, force)
        pl = qs.plan()
        sm, ct = qs.alloc_outputs(pl)
        slots.append({"ws": [t.workspace for t in tabs], "dims": pd, "sums": sm, "counts": ct,
                      "fin": qs.finalize(sm, ct, plan=pl), "bstream": torch.cuda.Stream(),
                      "done": torch.cuda.Event(), "q": qs})
    q0, plan0 = slots[0]["q"], slots[0]["q"].plan_obj
    sums, counts, fin_out = slots[0]["sums"], slots[0]["counts"], slots[0]["fin"]
    workspaces = slots[0]["ws"]
    torch.cuda.synchronize()
    for sl in slots:
        sl["done"].record(stream)

    def build_tables():
        return sdb.build_dims(dims, wdims.dim_keys, query, workspaces=workspaces)

    build_ms = []

    last_fused = [None]                    # event after the previous step's fused kernel

    def step(i, ev=None, n_out=None):
        sl = slots[i % 2]
        bs = sl["bstream"]
        bs.wait_event(sl["done"])          # step i-2, the slot's last user, has finished
        if last_fused[0] is not None:      # and the builds never share the GPU with a fused kernel
            bs.wait_event(last_fused[0])
        if ev is None:
            ev = tuple(torch.cuda.Event(enable_timing=True) for _ in range(4))
        t0 = time.perf_counter()
        q = sl["q"]
        with torch.cuda.stream(bs):
            sl["dims"].build(stream=bs)        # refills the handles q's joins point to
            build_ms.append(1000.0 * (time.perf_counter() - t0))
            plan = q.plan(stream=bs)
        # no event from the build stream to the run stream: sdb_build_dims ends
        # with a synchronization of the build stream and sdb_plan_star_query
        # either synchronizes it or makes no GPU call, so the tables and the
        # plan are complete here (an event record and wait cost about 25 us of
        # the critical path from one fused kernel to the next)
        # ev[0..1]: the fused kernel alone (recorded by the library around its
        # launch); ev[2..3]: the whole run (fill, fused kernel, terminal passes)
        sdb.set_fused_events(ev[0], ev[1])
        ev[2].record(stream)
        q.run(sl["sums"], sl["counts"], plan=plan, stream=stream)
        ev[3].record(stream)
        sdb.set_fused_events()
        last_fused[0] = ev[1]
        nout = q.finalize(sl["sums"], sl["counts"], plan=plan, outputs=sl["fin"], stream=stream)[3]
        if n_out is not None:
            n_out[i].copy_(nout[0], non_blocking=True)
        sl["done"].record(stream)
        return plan

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    build_ms.clear()

    events = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(args.steps)]
    for ev in events:                      # create the HIP events before the timed region
        for e in ev:
            e.record(stream)
    n_out = torch.zeros(max(args.steps, 1), dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    plan = plan0
    for i in range(args.steps):
        plan = step(i, events[i], n_out)
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    groups_per_step = n_out[:args.steps].cpu().numpy()
    n_groups_out = int(groups_per_step[-1]) if args.steps else 0
    if args.steps and not (groups_per_step == n_groups_out).all():
        raise AssertionError(f"steps disagree on the number of groups: {sorted(set(groups_per_step.tolist()))}")
    kernel_ms = [ev[0].elapsed_time(ev[1]) for ev in events]
    kernel_ms_mean = float(np.mean(kernel_ms))
    run_ms = [ev[2].elapsed_time(ev[3]) for ev in events]
    run_ms_mean = float(np.mean(run_ms))

    # the same steps one after another, each waiting for the last (context);
    # their build times are the builds alone (in the overlapped loop a build
    # call also waits for the previous step's fused kernel)
    last_fused[0] = None
    build_ms.clear()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(2 * i)                        # always slot 0: no overlap between steps
        torch.cuda.synchronize()
    ms_per_step_serial = 1000.0 * (time.perf_counter() - t0) / max(args.steps, 1)

    ms_per_step = 1000.0 * t_total / max(args.steps, 1)
    rows_per_s = n / (t_total / max(args.steps, 1))
    fact_cols = int(q0.q.n_cols)
    b_dense_per_row = 4 * fact_cols
    traffic = traffic_from_profile(args.config)
    plan_info = sdb.plan_summary(plan, query)
    balg_rows = min(n, args.balg_rows)
    b_alg = b_alg_per_row(host_sample(fact, balg_rows), wdims.dims, wdims.dim_keys, query, plan_info)
    achieved = n * b_alg / (kernel_ms_mean * 1e-3) / 1e9
    achieved_dense = n * b_dense_per_row / (kernel_ms_mean * 1e-3) / 1e9
    log(f"[bench] plan {json.dumps(plan_info)}")
    log(f"[bench] fused kernel mean {kernel_ms_mean:.4f} ms (min {min(kernel_ms):.4f}, "
        f"max {max(kernel_ms):.4f}); run {run_ms_mean:.4f} ms; step {ms_per_step:.4f} ms; groups {n_groups_out}")

    result = {
        "metric": "fact rows/sec and effective GB/s per star query; % of HBM peak (1 GPU)",
        "value": rows_per_s,
        "unit": "fact rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_serial": ms_per_step_serial,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": f"{args.config}: {cfg.describe}",
            "fact_rows": n,
            "fact_columns": fact_cols,
            "dimensions": {d: int(next(iter(t.values())).numel()) for d, t in dims.items()},
            "n_groups_domain": int(plan.n_groups),
            "n_groups_nonempty": n_groups_out,
            "plan": plan_info,
            "step": "build dims + sampled plan + fused kernel + device compaction; a step's builds and "
                    "plan overlap the previous step's terminal passes and compaction (second stream, "
                    "double-buffered)",
        },
        "effective_GBps_step": rows_per_s * b_dense_per_row / 1e9,
        "fused_kernel_ms": kernel_ms_mean,
        "fused_kernel_ms_median_min": [float(np.median(kernel_ms)), float(np.min(kernel_ms))],
        "run_ms": run_ms_mean,
        "run_ms_median_min": [float(np.median(run_ms)), float(np.min(run_ms))],
        "build_ms": float(np.mean(build_ms)) if build_ms else None,
        "build_ms_is": "host time of sdb_build_dims (every table, both synchronizations) in the serial steps",
        "fused_kernel_rows_per_s": n / (kernel_ms_mean * 1e-3),
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "bytes_basis": f"B_alg {b_alg:.4f} B/row (4 B per fact column x fraction of 128-byte lines holding "
                           f"a row live where the plan first reads the column, measured on the first "
                           f"{balg_rows} rows) x {n} rows per launch",
            "frac_b_dense": achieved_dense / HBM_PEAK_GBPS,
            "b_dense_basis": f"{b_dense_per_row} B/row: every byte of the {fact_cols} fact columns",
            "frac_run_window": n * b_alg / (run_ms_mean * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "run_window": "output fill + fused kernel + terminal passes (t_query), B_alg basis",
        },
        "cpu_baseline": None,
        "paper_context": PAPER_CONTEXT,
        "b_alg_bytes_per_row": b_alg,
    }
    if traffic:
        # measured HBM bytes per launch (profiles/) over the kernel's time: the
        # rate the memory actually delivered, gathers and probe lines included
        result["hbm_traffic_GBps_fused"] = traffic / (kernel_ms_mean * 1e-3) / 1e9
        result["hbm_traffic_frac_fused"] = result["hbm_traffic_GBps_fused"] / HBM_PEAK_GBPS

    result["stream_read"] = stream_read_reference(sdb, [fact[c] for c in query_columns(query)], n, stream,
                                                  achieved)

    result["run_finalize_ms_graph"] = graph_replay_ms(q0, sums, counts, plan, fin_out, stream, n_groups_out)

    result.update(end_to_end(sdb, build_tables, fact, query, force, sums, counts, fin_out))

    if cfg.n_fact <= 100_000_000:
        result["run_ms_mall_cold"] = mall_cold_ms(q0, sums, counts, plan, stream, dev)
        log(f"[bench] MALL-cold run {result['run_ms_mall_cold']:.4f} ms (warm {run_ms_mean:.4f} ms)")

    if args.ablation:
        ladder = ablation_ladder(sdb, fact, dims, wdims, query, stream, force)
        with open(args.ablation, "w") as f:
            json.dump({"workload": args.config, "fact_rows": n, "rungs": ladder}, f, indent=1)
        for r in ladder:
            log(f"[ablation] {r['rung']:58s} {r['run_ms']:8.3f} ms  {r['plan']}")

    if args.copy_calibration:
        copy_calibration(dev)

    if not args.no_cpu:
        q0.run(sums, counts, plan=plan)
        k, s_, c, nout, _ = q0.finalize(sums, counts, plan=plan, outputs=fin_out)
        torch.cuda.synchronize()
        m = int(nout.item())
        keys = k[:m, :q0.n_keys].to(torch.int64).cpu().numpy()
        gpu_rows = sdb.QueryResult(keys.reshape(m, q0.n_keys), s_[:m].cpu().numpy(), c[:m].cpu().numpy()).as_rows()
        result.update(cpu_baseline_leg(args.config, n, gpu_rows, fact))

    if not args.no_configs and args.rows is None and args.config == "c3_star3":
        del fact, slots, sums, counts, fin_out, q0
        torch.cuda.empty_cache()
        ex = None
        if not args.no_cpu:
            from oracle import ranges
            ex = ranges.pool(ranges.worker_count())
        try:
            result["configs"] = [config_record(sdb, name, ex, dev)
                                 for name in ("c1_scalar_scan", "c2_join_group", "c4_star4_zipf", "c5_hash_stress")]
            # c3's query over date-sorted rows: the planner's per-range stage
            # orders against one order for the whole table
            result["configs"].append(config_record(sdb, "c3d_star3_date_sorted", ex, dev,
                                                   compare={"segments": -1}))
        finally:
            if ex is not None:
                ex.shutdown()

    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
