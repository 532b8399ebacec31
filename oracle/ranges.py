"""The oracle over row ranges, on worker processes (test infrastructure only).

A SUM and a COUNT over a set of rows are the sums of the SUMs and COUNTs over
any partition of that set into disjoint parts; with 64-bit wrapping integers
this holds modulo 2**64 for every group separately. So the result over fact
rows [0, N) equals the group-by-group merge of the results over row ranges
[r_0, r_1), [r_1, r_2), ... that cover [0, N). ``merge`` performs exactly that
merge; ``star_query`` itself is run unchanged on each range. The pins check
``merge`` against the whole-table oracle and against a pure-Python dict merge.

The workers regenerate their own rows from the seeded generator (every column
is drawn in counter-addressed chunks, so a row range regenerates alone), and
return, besides their partial result, the 64-bit sum of every fact column of
their range, so a caller can check that the rows they saw are the rows it holds.

Worker processes come from a ``forkserver`` started by ``start_forkserver``:
the server is started while the calling process has not yet touched the GPU,
and every worker is forked from the server, never from the caller.

Only the test suite and the benchmark's CPU-baseline leg use this module.
"""

from __future__ import annotations

import multiprocessing as mp
import os
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

from .star import OracleResult, star_query

_PRELOAD = ["numpy", "oracle.star", "datagen.star"]


def merge(results: list) -> OracleResult:
    """Group-by-group sum (mod 2**64) and count of partial results over
    disjoint row ranges of one query."""
    results = list(results)
    if not results:
        raise ValueError("merge needs at least one partial result")
    n_live = sum(int(r.n_live) for r in results)
    n_keys = results[0].keys.shape[1]
    if n_keys == 0:                      # scalar query: one (sum, count) row per part
        s = np.array([sum(int(r.sums[0]) for r in results) % (1 << 64)], dtype=np.uint64)
        c = np.array([sum(int(r.counts[0]) for r in results)], dtype=np.int64)
        return OracleResult(np.zeros((1, 0), dtype=np.int64), s.view(np.int64), c, n_live)
    keys = np.concatenate([r.keys for r in results], axis=0)
    sums = np.concatenate([r.sums.view(np.uint64) for r in results])
    counts = np.concatenate([r.counts for r in results])
    uniq, inverse = np.unique(keys, axis=0, return_inverse=True)
    inverse = inverse.reshape(-1)
    out_s = np.zeros(uniq.shape[0], dtype=np.uint64)
    np.add.at(out_s, inverse, sums)
    out_c = np.zeros(uniq.shape[0], dtype=np.int64)
    np.add.at(out_c, inverse, counts)
    return OracleResult(uniq.astype(np.int64), out_s.view(np.int64), out_c, n_live)


def row_ranges(n: int, parts: int, align: int) -> list:
    """At most ``parts`` contiguous ranges covering [0, n), cut at multiples of ``align``."""
    if n <= 0:
        return [(0, 0)]
    units = -(-n // align)
    per = -(-units // max(1, parts))
    out = []
    for u in range(0, units, per):
        out.append((u * align, min(n, (u + per) * align)))
    return out


def worker_count(cap: int = 16) -> int:
    """Host cores this process may use, at most ``cap``."""
    return max(1, min(cap, len(os.sched_getaffinity(0))))


def start_forkserver() -> None:
    """Starts the fork server the worker pools fork from. Call it before the
    process makes its first GPU call."""
    mp.set_forkserver_preload(_PRELOAD)
    from multiprocessing import forkserver
    forkserver.ensure_running()


def pool(workers: int, initializer=None, initargs=()) -> ProcessPoolExecutor:
    return ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("forkserver"),
                               initializer=initializer, initargs=initargs)


# ---------------------------------------------------------------- worker side

_DIMS = {}
_BARRIER = None


def _set_barrier(barrier) -> None:
    global _BARRIER
    _BARRIER = barrier


def _workload_rows(name: str, lo: int, hi: int):
    import datagen
    w = datagen.make_workload(name, n_fact=0, threads=1) if name not in _DIMS else None
    if w is not None:
        _DIMS[name] = (w.dims, w.dim_keys, w.query)
    dims, dim_keys, query = _DIMS[name]
    fact = datagen.fact_rows(name, lo, hi, threads=1)
    return fact, dims, dim_keys, query


def _column_sums(fact: dict) -> dict:
    return {k: int(v.astype(np.int64).sum()) for k, v in fact.items()}


def range_task(name: str, lo: int, hi: int):
    """Rows [lo, hi) of workload ``name``: (partial result, column sums, oracle seconds)."""
    fact, dims, dim_keys, query = _workload_rows(name, lo, hi)
    t0 = time.perf_counter()
    r = star_query(fact, dims, dim_keys, query)
    return r, _column_sums(fact), time.perf_counter() - t0


def timed_range_task(name: str, lo: int, hi: int, timeout: float):
    """As ``range_task``, but every worker first generates its rows, then waits
    at a barrier shared by all workers, so the oracle phase of all workers
    starts together; returns wall-clock start and end of the oracle phase."""
    fact, dims, dim_keys, query = _workload_rows(name, lo, hi)
    _BARRIER.wait(timeout)
    t0 = time.time()
    r = star_query(fact, dims, dim_keys, query)
    t1 = time.time()
    return r, _column_sums(fact), t0, t1


# ---------------------------------------------------------------- caller side

def run(name: str, n: int, ex: ProcessPoolExecutor, task_rows: int, log=None):
    """The oracle over rows [0, n) of workload ``name`` in ranges of about
    ``task_rows`` rows on ``ex``: (merged result, column sums of [0, n))."""
    import datagen.star as ds
    ranges = row_ranges(n, -(-n // max(1, task_rows)), ds.CHUNK)
    futs = [ex.submit(range_task, name, lo, hi) for lo, hi in ranges]
    parts, sums = [], {}
    for i, f in enumerate(futs):
        r, cs, secs = f.result()
        parts.append(r)
        for k, v in cs.items():
            sums[k] = sums.get(k, 0) + v
        if log:
            log(f"oracle range {i + 1}/{len(ranges)} {ranges[i]}: {secs:.1f} s")
    return merge(parts), sums


def run_timed(name: str, n: int, workers: int, timeout: float = 600.0):
    """The oracle over rows [0, n) of workload ``name`` split into one range per
    worker process, the oracle phases started together after every worker has
    generated its rows. Returns (merged result, column sums, info) with info
    holding the wall-clock time from the first start to the last end plus the
    merge, and the summed per-worker oracle seconds."""
    import datagen.star as ds
    ranges = row_ranges(n, workers, ds.CHUNK)
    ctx = mp.get_context("forkserver")
    barrier = ctx.Barrier(len(ranges))
    with ProcessPoolExecutor(max_workers=len(ranges), mp_context=ctx, initializer=_set_barrier,
                             initargs=(barrier,)) as ex:
        futs = [ex.submit(timed_range_task, name, lo, hi, timeout) for lo, hi in ranges]
        out = [f.result(timeout=timeout) for f in futs]
    t_merge = time.perf_counter()
    res = merge([o[0] for o in out])
    t_merge = time.perf_counter() - t_merge
    sums = {}
    for _, cs, _, _ in out:
        for k, v in cs.items():
            sums[k] = sums.get(k, 0) + v
    starts, ends = [o[2] for o in out], [o[3] for o in out]
    wall = max(ends) - min(starts) + t_merge
    return res, sums, {"wall_s": wall, "merge_s": t_merge, "workers": len(ranges),
                       "worker_oracle_s": [e - s for s, e in zip(starts, ends)], "ranges": ranges}
