"""Seeded synthetic star schemas shaped like the paper's query flights.

The paper measures the Star Schema Benchmark at SF100 (about 600M fact rows of
int32 columns, Section 5.1). Its data and generator are not used here: five
synthetic workloads stand in for its query shapes (a date-filtered scalar scan,
one join with a small group-by, a three-dimension star, a four-dimension star
with a Zipf-skewed key, and an open-addressing stress), plus small random
schemas for exhaustive checking.

Generation recipe (stated once, used everywhere):

* Every random column is cut into chunks of ``CHUNK`` rows. Chunk ``c`` of the
  column with stream id ``s`` in workload ``w`` draws from
  ``numpy.random.Generator(PCG64(SeedSequence([2607, 7632, w, s, c])))``. A row
  range can therefore be regenerated without generating the rows before it,
  and the result does not depend on how many threads generate it.
* ``uniform lo hi`` draws ``integers(lo, hi, endpoint=True, dtype=int32)``.
* ``zipf n s`` draws ``u = random()`` (float64 in [0, 1)) and returns the
  0-based rank ``r`` with ``cdf[r-1] <= u < cdf[r]`` where ``cdf`` is the
  normalised cumulative sum of ``k**-s`` for ``k = 1..n``; rank 0 is the most
  frequent key.
* ``index`` is the row number (dense primary keys, as in the benchmark the
  paper uses); ``perm n`` is one seeded permutation of ``0..n-1``.
* ``ramp lo hi n`` gives row ``i`` of an ``n``-row column the value
  ``lo + i * (hi - lo + 1) // n``: rows sorted by that column, each value
  holding an equal run of rows (a fact table clustered by date).
* The date dimension has one row per day ``d`` in ``0..2555`` with
  ``year = 1992 + d // 365`` (integer floor). That formula gives eight years,
  the last (1999) holding day 2555 only.

Nothing in this module evaluates a predicate, probes a key or sums a value.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from functools import lru_cache

import numpy as np

CHUNK = 1 << 22
SEED_ROOT = (2607, 7632)
FULL_ROWS = 600_000_000
N_DAYS = 2556


# --------------------------------------------------------------------------
# column recipes
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Col:
    name: str
    dist: tuple          # ("uniform", lo, hi) | ("zipf", n, s) | ("index",) | ("perm", n) | ("year_of_day",)
                         # | ("ramp", lo, hi, n)
    stream: int = 0


@dataclass(frozen=True)
class Dim:
    name: str
    n_rows: int
    key: str
    cols: tuple          # tuple[Col, ...]; the key column is one of them


@dataclass(frozen=True)
class Config:
    config_id: int
    name: str
    n_fact: int
    fact_cols: tuple     # tuple[Col, ...]
    dims: tuple          # tuple[Dim, ...]
    query: dict
    describe: str = ""


def _date_dim() -> Dim:
    return Dim("date", N_DAYS, "date_key",
               (Col("date_key", ("index",)), Col("year", ("year_of_day",))))


def _pred(col, op, lo, hi=None):
    return {"col": col, "op": op, "lo": int(lo), "hi": None if hi is None else int(hi)}


CONFIGS: dict[str, Config] = {}


def _register(cfg: Config) -> None:
    CONFIGS[cfg.name] = cfg


_register(Config(
    1, "c1_scalar_scan", 1_048_576,
    (Col("date_key", ("uniform", 0, N_DAYS - 1), 1),
     Col("qty", ("uniform", 1, 50), 2),
     Col("disc", ("uniform", 0, 10), 3),
     Col("price", ("uniform", 90_000, 10_000_000), 4)),
    (_date_dim(),),
    {
        "fact_preds": [_pred("disc", "between", 2, 4), _pred("qty", "lt", 30)],
        "joins": [{"fact_key": "date_key", "dim": "date",
                   "preds": [_pred("year", "eq", 1994)], "payloads": [], "kind": "auto"}],
        "group_by": [],
        "agg": {"kind": "mul", "a": "price", "b": "disc"},
    },
    "scalar SUM(price*disc) over a date-filtered scan with two fact predicates",
))

_register(Config(
    2, "c2_join_group", 60_000_000,
    (Col("supp_key", ("uniform", 0, 199_999), 1),
     Col("date_key", ("uniform", 0, N_DAYS - 1), 2),
     Col("revenue", ("uniform", 1, 1_000_000), 3)),
    (Dim("supplier", 200_000, "supp_key",
         (Col("supp_key", ("index",)),
          Col("region", ("uniform", 0, 4), 101),
          Col("nation", ("uniform", 0, 24), 102))),
     _date_dim()),
    {
        "fact_preds": [],
        "joins": [{"fact_key": "supp_key", "dim": "supplier",
                   "preds": [_pred("region", "eq", 2)], "payloads": ["nation"], "kind": "auto"},
                  {"fact_key": "date_key", "dim": "date",
                   "preds": [], "payloads": ["year"], "kind": "auto"}],
        "group_by": [["supplier", "nation"], ["date", "year"]],
        "agg": {"kind": "col", "a": "revenue", "b": None},
    },
    "SUM(revenue) GROUP BY (supplier nation, year) over one filtered join",
))

_register(Config(
    3, "c3_star3", FULL_ROWS,
    (Col("cust_key", ("uniform", 0, 2_999_999), 1),
     Col("supp_key", ("uniform", 0, 199_999), 2),
     Col("date_key", ("uniform", 0, N_DAYS - 1), 3),
     Col("revenue", ("uniform", 1, 1_000_000), 4)),
    (Dim("customer", 3_000_000, "cust_key",
         (Col("cust_key", ("index",)),
          Col("region", ("uniform", 0, 4), 201),
          Col("city", ("uniform", 0, 249), 202))),
     Dim("supplier", 200_000, "supp_key",
         (Col("supp_key", ("index",)),
          Col("region", ("uniform", 0, 4), 101),
          Col("city", ("uniform", 0, 249), 103))),
     _date_dim()),
    {
        "fact_preds": [],
        "joins": [{"fact_key": "cust_key", "dim": "customer",
                   "preds": [_pred("region", "eq", 2)], "payloads": ["city"], "kind": "auto"},
                  {"fact_key": "supp_key", "dim": "supplier",
                   "preds": [_pred("region", "eq", 2)], "payloads": ["city"], "kind": "auto"},
                  {"fact_key": "date_key", "dim": "date",
                   "preds": [_pred("year", "between", 1992, 1997)], "payloads": ["year"],
                   "kind": "auto"}],
        "group_by": [["customer", "city"], ["supplier", "city"], ["date", "year"]],
        "agg": {"kind": "col", "a": "revenue", "b": None},
    },
    "SUM(revenue) GROUP BY (customer city, supplier city, year) over a three-dimension star",
))

_register(Config(
    4, "c4_star4_zipf", FULL_ROWS,
    (Col("cust_key", ("uniform", 0, 2_999_999), 1),
     Col("supp_key", ("uniform", 0, 199_999), 2),
     Col("part_key", ("zipf", 1_400_000, 1.1), 3),
     Col("date_key", ("uniform", 0, N_DAYS - 1), 4),
     Col("revenue", ("uniform", 1, 1_000_000), 5),
     Col("supplycost", ("uniform", 1, 100_000), 6)),
    (Dim("part", 1_400_000, "part_key",
         (Col("part_key", ("index",)),
          Col("category", ("uniform", 0, 24), 301),
          Col("brand", ("uniform", 0, 999), 302))),
     Dim("customer", 3_000_000, "cust_key",
         (Col("cust_key", ("index",)),
          Col("region", ("uniform", 0, 4), 201))),
     Dim("supplier", 200_000, "supp_key",
         (Col("supp_key", ("index",)),
          Col("region", ("uniform", 0, 4), 101),
          Col("nation", ("uniform", 0, 24), 102))),
     _date_dim()),
    {
        "fact_preds": [],
        "joins": [{"fact_key": "part_key", "dim": "part",
                   "preds": [_pred("category", "eq", 1)], "payloads": ["brand"], "kind": "auto"},
                  {"fact_key": "cust_key", "dim": "customer",
                   "preds": [_pred("region", "eq", 2)], "payloads": [], "kind": "auto"},
                  {"fact_key": "supp_key", "dim": "supplier",
                   "preds": [_pred("region", "eq", 2)], "payloads": ["nation"], "kind": "auto"},
                  {"fact_key": "date_key", "dim": "date",
                   "preds": [_pred("year", "between", 1992, 1997)], "payloads": ["year"],
                   "kind": "auto"}],
        "group_by": [["date", "year"], ["part", "brand"], ["supplier", "nation"]],
        "agg": {"kind": "sub", "a": "revenue", "b": "supplycost"},
    },
    "SUM(revenue - supplycost) GROUP BY (year, brand, supplier nation), Zipf part keys",
))

_register(Config(
    5, "c5_hash_stress", FULL_ROWS,
    (Col("key", ("uniform", 0, (1 << 24) - 1), 1),
     Col("value", ("uniform", 1, 1_000_000), 2)),
    (Dim("big", 1 << 24, "key",
         (Col("key", ("perm", 1 << 24), 401),
          Col("flag", ("uniform", 0, 1), 402),
          Col("attr", ("uniform", 0, 65_535), 403))),),
    {
        "fact_preds": [],
        "joins": [{"fact_key": "key", "dim": "big",
                   "preds": [_pred("flag", "eq", 1)], "payloads": ["attr"],
                   "kind": "hash", "load_factor": 0.5}],
        "group_by": [["big", "attr"]],
        "agg": {"kind": "col", "a": "value", "b": None},
    },
    "SUM(value) GROUP BY attr through a 2^25-slot open-addressing table",
))

_c3 = CONFIGS["c3_star3"]
_register(Config(
    6, "c3d_star3_date_sorted", FULL_ROWS,
    tuple(Col("date_key", ("ramp", 0, N_DAYS - 1, FULL_ROWS)) if c.name == "date_key" else c for c in _c3.fact_cols),
    _c3.dims,
    _c3.query,
    "c3's query over fact rows sorted by date (each day an equal run of rows): the date filter's pass "
    "fraction changes along the table",
))

CONFIG_ORDER = ["c1_scalar_scan", "c2_join_group", "c3_star3", "c4_star4_zipf", "c5_hash_stress"]


# --------------------------------------------------------------------------
# generation
# --------------------------------------------------------------------------

def _rng(config_id: int, stream: int, chunk: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], config_id, stream, chunk])))


@lru_cache(maxsize=8)
def zipf_cdf(n: int, s: float) -> np.ndarray:
    """Normalised cumulative weights of ranks 1..n under P(k) proportional to k**-s."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-float(s))
    c = np.cumsum(w)
    c /= c[-1]
    c[-1] = 1.0
    return c


def _chunk_values(config_id: int, col: Col, chunk: int, lo_row: int, hi_row: int) -> np.ndarray:
    """Rows [lo_row, hi_row) of chunk ``chunk`` (offsets inside the chunk)."""
    kind = col.dist[0]
    n_in_chunk = hi_row - lo_row
    if kind == "index":
        base = chunk * CHUNK
        return np.arange(base + lo_row, base + hi_row, dtype=np.int64).astype(np.int32)
    if kind == "year_of_day":
        base = chunk * CHUNK
        d = np.arange(base + lo_row, base + hi_row, dtype=np.int64)
        return (1992 + d // 365).astype(np.int32)
    if kind == "ramp":
        _, lo, hi, n_total = col.dist
        base = chunk * CHUNK
        i = np.arange(base + lo_row, base + hi_row, dtype=np.int64)
        return (lo + i * (hi - lo + 1) // n_total).astype(np.int32)
    rng = _rng(config_id, col.stream, chunk)
    if kind == "uniform":
        _, lo, hi = col.dist
        # Always draw the whole chunk prefix so a sub-range equals the same rows
        # of a full-chunk draw.
        v = rng.integers(lo, hi, size=hi_row, endpoint=True, dtype=np.int32)
        return v[lo_row:hi_row]
    if kind == "zipf":
        _, n, s = col.dist
        u = rng.random(size=hi_row)[lo_row:hi_row]
        r = np.searchsorted(zipf_cdf(n, s), u, side="right")
        np.minimum(r, n - 1, out=r)
        return r.astype(np.int32)
    raise ValueError(f"unsupported chunked distribution {kind!r} ({n_in_chunk} rows)")


def _fill_column(config_id: int, col: Col, start: int, stop: int, out: np.ndarray,
                 threads: int | None) -> np.ndarray:
    assert out.shape == (stop - start,) and out.dtype == np.int32
    if stop <= start:
        return out
    if col.dist[0] == "perm":
        n = col.dist[1]
        p = _rng(config_id, col.stream, 0).permutation(n).astype(np.int32)
        out[:] = p[start:stop]
        return out
    jobs = []
    c0, c1 = start // CHUNK, (stop - 1) // CHUNK
    for c in range(c0, c1 + 1):
        lo = max(start, c * CHUNK) - c * CHUNK
        hi = min(stop, (c + 1) * CHUNK) - c * CHUNK
        dst = c * CHUNK + lo - start
        jobs.append((c, lo, hi, dst))

    def run(job):
        c, lo, hi, dst = job
        out[dst:dst + (hi - lo)] = _chunk_values(config_id, col, c, lo, hi)

    nthreads = threads if threads is not None else min(16, os.cpu_count() or 1)
    if nthreads <= 1 or len(jobs) == 1:
        for j in jobs:
            run(j)
    else:
        with ThreadPoolExecutor(max_workers=nthreads) as ex:
            list(ex.map(run, jobs))
    return out


def _config(cfg) -> Config:
    if isinstance(cfg, Config):
        return cfg
    if isinstance(cfg, int):
        return CONFIGS[CONFIG_ORDER[cfg - 1]]
    return CONFIGS[cfg]


def fact_column(cfg, name: str, start: int, stop: int, out: np.ndarray | None = None,
                threads: int | None = None) -> np.ndarray:
    """Rows [start, stop) of one fact column of a workload, as int32."""
    c = _config(cfg)
    col = next(x for x in c.fact_cols if x.name == name)
    if out is None:
        out = np.empty(stop - start, dtype=np.int32)
    return _fill_column(c.config_id, col, start, stop, out, threads)


def fact_rows(cfg, start: int, stop: int, threads: int | None = None) -> dict:
    """All fact columns of rows [start, stop)."""
    c = _config(cfg)
    return {col.name: fact_column(c, col.name, start, stop, threads=threads) for col in c.fact_cols}


def dim_table(cfg, dim_name: str, threads: int | None = None) -> dict:
    c = _config(cfg)
    d = next(x for x in c.dims if x.name == dim_name)
    out = {}
    for col in d.cols:
        arr = np.empty(d.n_rows, dtype=np.int32)
        out[col.name] = _fill_column(c.config_id, col, 0, d.n_rows, arr, threads)
    return out


@dataclass
class Workload:
    """One star schema plus the query to run over it.

    ``fact`` maps column name to an int32 array of ``n_fact`` rows, ``dims``
    maps dimension name to ``{column name: int32 array}``, ``dim_keys`` names
    each dimension's primary-key column, and ``query`` is the plain-data query
    description (predicates, joins, group keys, aggregate) shared by the oracle
    and the GPU library binding.
    """
    name: str
    n_fact: int
    fact: dict
    dims: dict
    dim_keys: dict
    query: dict
    row_start: int = 0
    meta: dict = field(default_factory=dict)


def make_workload(cfg, n_fact: int | None = None, row_start: int = 0,
                  threads: int | None = None, fact: dict | None = None) -> Workload:
    """Generate workload ``cfg`` (name, 1-based index or Config).

    ``n_fact`` rows starting at fact row ``row_start`` are generated (default:
    the workload's full size); the dimension tables are always complete.
    ``fact`` may supply preallocated int32 output arrays per column.
    """
    c = _config(cfg)
    n = c.n_fact if n_fact is None else int(n_fact)
    fcols = {}
    for col in c.fact_cols:
        out = None if fact is None else fact[col.name]
        fcols[col.name] = fact_column(c, col.name, row_start, row_start + n, out=out,
                                      threads=threads)
    dims = {d.name: dim_table(c, d.name, threads) for d in c.dims}
    keys = {d.name: d.key for d in c.dims}
    return Workload(c.name, n, fcols, dims, keys, _copy_query(c.query), row_start,
                    {"config_id": c.config_id, "describe": c.describe})


def _copy_query(q: dict) -> dict:
    import copy
    return copy.deepcopy(q)


# --------------------------------------------------------------------------
# small random schemas (for brute-force checking and edge cases)
# --------------------------------------------------------------------------

_OPS = ["eq", "ne", "lt", "le", "gt", "ge", "between"]
_I32_MIN, _I32_MAX = -(1 << 31), (1 << 31) - 1


def _random_literal(rng, values: np.ndarray) -> int:
    r = rng.random()
    if r < 0.05:
        return int(rng.choice([_I32_MIN, _I32_MAX, _I32_MIN - 5, _I32_MAX + 7, 0]))
    if len(values) == 0 or r < 0.15:
        return int(rng.integers(-50, 50))
    return int(values[rng.integers(0, len(values))]) + int(rng.integers(-1, 2))


def _random_pred(rng, name: str, values: np.ndarray) -> dict:
    op = _OPS[rng.integers(0, len(_OPS))]
    a = _random_literal(rng, values)
    if op == "between":
        b = _random_literal(rng, values)
        if rng.random() < 0.8 and b < a:
            a, b = b, a
        return _pred(name, op, a, b)
    return _pred(name, op, a)


def random_tiny_workload(seed: int, max_fact: int = 2000, max_dim_rows: int = 300,
                         max_dims: int = 3, allow_hash: bool = True,
                         n_fact: int | None = None) -> Workload:
    """A small random star schema with random predicates, joins and group keys.

    Dimension keys are distinct, shuffled and offset (so ``kmin`` is not 0 and
    key ranges may have gaps); fact keys fall partly outside the dimension's
    key set; values may be negative; literals sometimes sit at or beyond the
    int32 limits. Every draw comes from ``SeedSequence([2607, 7632, 99, seed])``.
    """
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], 99, int(seed)])))
    n = int(rng.integers(0, max_fact + 1)) if n_fact is None else int(n_fact)
    n_dims = int(rng.integers(0, max_dims + 1))
    dims, dim_keys, joins = {}, {}, []
    fact = {}
    for j in range(n_dims):
        dn = f"d{j}"
        m = int(rng.integers(1, max_dim_rows + 1))
        span = m + int(rng.integers(0, 2 * m + 1))          # gaps in the key set
        offset = int(rng.integers(-1000, 1000))
        keys = (rng.permutation(span)[:m] + offset).astype(np.int32)
        cols = {"k": keys}
        n_attr = int(rng.integers(1, 4))
        for a in range(n_attr):
            hi = int(rng.choice([1, 4, 30, 300]))
            lo = int(rng.choice([0, -3, 5]))
            cols[f"a{a}"] = rng.integers(lo, lo + hi, size=m, endpoint=True, dtype=np.int32)
        dims[dn] = cols
        dim_keys[dn] = "k"
        preds = [_random_pred(rng, f"a{int(rng.integers(0, n_attr))}", cols[f"a{0}"])
                 for _ in range(int(rng.integers(0, 3)))]
        n_pay = int(rng.integers(0, min(n_attr, 3) + 1))
        payloads = [f"a{x}" for x in rng.permutation(n_attr)[:n_pay]]
        kind = "auto"
        if allow_hash and rng.random() < 0.35:
            kind = "hash"
        elif rng.random() < 0.2 and span <= 2 * m:      # a forced dense map needs a key range within 2m
            kind = "dense"
        jd = {"fact_key": f"fk{j}", "dim": dn, "preds": preds, "payloads": payloads, "kind": kind}
        if kind == "hash":
            jd["load_factor"] = float(rng.choice([0.5, 0.25, 0.9]))
        joins.append(jd)
        # fact keys: mostly hits, some misses just outside / far outside the key range
        hit = keys[rng.integers(0, m, size=n)] if n else np.empty(0, np.int32)
        miss = rng.integers(offset - 50, offset + span + 50, size=n, dtype=np.int64)
        pick = rng.random(n) < 0.8
        fact[f"fk{j}"] = np.where(pick, hit, miss).astype(np.int32)
    n_val = int(rng.integers(1, 4))
    for v in range(n_val):
        scale = int(rng.choice([10, 1000, 1_000_000, _I32_MAX]))
        fact[f"v{v}"] = rng.integers(-scale, scale, size=n, endpoint=False, dtype=np.int64).astype(np.int32)
    fact_preds = [_random_pred(rng, f"v{int(rng.integers(0, n_val))}", fact["v0"])
                  for _ in range(int(rng.integers(0, 3)))]
    group_by = []
    for jd in joins:
        for p in jd["payloads"]:
            group_by.append([jd["dim"], p])
    rng.shuffle(group_by)
    group_by = [list(g) for g in group_by[:3]]
    # payloads that are not group keys are dropped again so the description stays minimal
    used = {(g[0], g[1]) for g in group_by}
    for jd in joins:
        jd["payloads"] = [p for p in jd["payloads"] if (jd["dim"], p) in used]
    kind = ["col", "mul", "sub", "add"][int(rng.integers(0, 4))]
    a = f"v{int(rng.integers(0, n_val))}"
    b = None if kind == "col" else f"v{int(rng.integers(0, n_val))}"
    query = {"fact_preds": fact_preds, "joins": joins, "group_by": group_by,
             "agg": {"kind": kind, "a": a, "b": b}}
    return Workload(f"tiny{seed}", n, fact, dims, dim_keys, query, 0, {"seed": seed})
