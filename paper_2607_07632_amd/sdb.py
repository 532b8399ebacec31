"""ctypes binding of libsdb (include/sdb.h): argument marshalling only.

Every step of the query runs in the library's HIP kernels; this module only
lays out the C structs, passes torch device pointers and the current HIP
stream, allocates the caller-owned buffers with torch, and copies results back.
It fails loudly when the built library is missing: there is no fallback.

The high-level helpers (``build_dims``, ``StarQuery``) translate the plain-data
query description used by the test suite and the benchmark (column names,
predicate ops, joins, group keys, aggregate) into the C descriptors.
"""

from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass, field

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsdb.so")

MAX_DIM_COLS = 8
MAX_DIM_PREDS = 4
MAX_PAYLOADS = 3
MAX_FACT_COLS = 16
MAX_FACT_PREDS = 8
MAX_JOINS = 6
MAX_GROUP_KEYS = 4
MAX_STAGES = MAX_FACT_PREDS + MAX_JOINS
MAX_SEGMENTS = 8
PLAN_SCRATCH_BYTES = 81920
NOALLOC_SCRATCH_BYTES = 64 << 20

OPS = {"eq": 0, "ne": 1, "lt": 2, "le": 3, "gt": 4, "ge": 5, "between": 6}
TABLES = {"auto": 0, "dense": 1, "hash": 2}
AGGS = {"col": 0, "mul": 1, "sub": 2, "add": 3}
TERMINALS = {"auto": 0, "scalar": 1, "lds": 2, "global": 3, "part": 4}
BASELINES = {"per_operator": 0, "global_handoff": 1}
TERMINAL_NAMES = {1: "scalar", 2: "lds", 3: "global", 4: "part"}
LDS_NAMES = {0: "global", 1: "lds_map", 2: "lds_bits", 3: "lds_rank", 4: "lds_coarse", 5: "lds_window"}
FILTER_NAMES = {0: None, 1: "bitmap", 2: "bloom"}
MAX_FILTER_BYTES = 4 << 20
STATUS = {0: "SDB_OK", 1: "SDB_INVALID_ARG", 2: "SDB_UNSUPPORTED", 3: "SDB_CAPACITY",
          4: "SDB_WORKSPACE_TOO_SMALL", 5: "SDB_DUP_KEY", 6: "SDB_KEY_RANGE", 7: "SDB_HIP_ERROR"}

i32, u32, i64, u64, vp = C.c_int32, C.c_uint32, C.c_int64, C.c_uint64, C.c_void_p


class SdbPred(C.Structure):
    _fields_ = [("col", i32), ("op", i32), ("lo", i64), ("hi", i64)]


class SdbDimDesc(C.Structure):
    _fields_ = [("key", vp), ("n_rows", i64), ("n_cols", i32), ("cols", vp * MAX_DIM_COLS),
                ("n_preds", i32), ("preds", SdbPred * MAX_DIM_PREDS), ("n_payloads", i32),
                ("payload_cols", i32 * MAX_PAYLOADS), ("kind", i32), ("load_factor", C.c_double),
                ("dense_budget_bytes", i64)]


class SdbDim(C.Structure):
    _fields_ = [("kind", i32), ("width", i32), ("n_rows", i64), ("n_pass", i64),
                ("key_min", i32), ("key_max", i32), ("pass_key_min", i32), ("pass_key_max", i32),
                ("n_slots", u64), ("hash_bits", i32),
                ("sentinel", u32), ("domain", u64), ("n_payloads", i32),
                ("payload_min", i32 * MAX_PAYLOADS), ("payload_radix", u32 * MAX_PAYLOADS),
                ("payload_div", u64 * MAX_PAYLOADS), ("map", vp), ("stats", vp), ("bits", vp),
                ("filter", vp), ("filter_bits", u64), ("filter_kind", i32), ("reserved_", i32)]


class SdbDimSummary(C.Structure):
    _fields_ = [("kind", i32), ("width", i32), ("n_rows", i64), ("n_pass", i64),
                ("key_min", i32), ("key_max", i32), ("pass_key_min", i32), ("pass_key_max", i32),
                ("pass_keys_contiguous", i32), ("n_payloads", i32), ("n_slots", u64), ("table_bytes", u64),
                ("occupancy", C.c_double), ("payload_min", i32 * MAX_PAYLOADS),
                ("payload_max", i32 * MAX_PAYLOADS), ("payload_radix", u32 * MAX_PAYLOADS),
                ("filter_kind", i32), ("domain", u64), ("filter_bytes", u64)]


class SdbJoin(C.Structure):
    _fields_ = [("fact_key_col", i32), ("dim", C.POINTER(SdbDim))]


class SdbGroupKey(C.Structure):
    _fields_ = [("join", i32), ("payload", i32)]


class SdbAgg(C.Structure):
    _fields_ = [("kind", i32), ("a", i32), ("b", i32)]


class SdbQuery(C.Structure):
    _fields_ = [("n_fact", i64), ("n_cols", i32), ("cols", vp * MAX_FACT_COLS),
                ("n_preds", i32), ("preds", SdbPred * MAX_FACT_PREDS),
                ("n_joins", i32), ("joins", SdbJoin * MAX_JOINS),
                ("n_group_keys", i32), ("group_keys", SdbGroupKey * MAX_GROUP_KEYS),
                ("agg", SdbAgg), ("force_terminal", i32), ("force_ipt", i32),
                ("force_vector", i32), ("force_order", i32), ("grid_blocks", i32),
                ("force_lds", i32), ("force_xcd", i32), ("force_eager", i32),
                ("force_block", i32), ("force_range", i32), ("force_coarse", i32),
                ("force_slice", i32), ("force_unroll", i32), ("force_window", i32), ("force_segments", i32),
                ("force_prefilter", i32)]


class SdbPlan(C.Structure):
    _fields_ = [("n_stages", i32), ("stage_kind", i32 * MAX_STAGES),
                ("stage_index", i32 * MAX_STAGES), ("stage_pass", C.c_double * MAX_STAGES),
                ("stage_pass_alone", C.c_double * MAX_STAGES),
                ("stage_lds", i32 * MAX_STAGES), ("stage_defer", i32 * MAX_STAGES),
                ("stage_range", i32 * MAX_STAGES), ("stage_coarse", i32 * MAX_STAGES),
                ("stage_window_lo", i32 * MAX_STAGES), ("stage_window_slots", i32 * MAX_STAGES),
                ("stage_window_cover", C.c_double * MAX_STAGES),
                ("sampled_rows", i64), ("est_cost", C.c_double), ("terminal", i32), ("ipt", i32),
                ("vector", i32), ("eager", i32), ("block", i32), ("grid", i32), ("xcd_copies", i32),
                ("lds_bytes", i32), ("part_shift", i32), ("n_parts", i32), ("part_subs", i32), ("part_cap", i64),
                ("n_group_keys", i32),
                ("key_min", i32 * MAX_GROUP_KEYS), ("radix", u32 * MAX_GROUP_KEYS),
                ("stride", u64 * MAX_GROUP_KEYS), ("n_groups", u64), ("run_scratch_bytes", i64),
                ("slice_bits", i32), ("slice_stage", i32), ("slice_grid", i32), ("slice_prefilter", i32),
                ("unroll", i32),
                ("n_segments", i32), ("segment_order", (i32 * MAX_STAGES) * MAX_SEGMENTS),
                ("segment_start", i64 * (MAX_SEGMENTS + 1))]


STRUCTS = [SdbPred, SdbDimDesc, SdbDim, SdbJoin, SdbGroupKey, SdbAgg, SdbQuery, SdbPlan, SdbDimSummary]

# exported symbol -> (restype, argtypes)
SIGNATURES = {
    "sdb_last_error": (C.c_char_p, []),
    "sdb_status_string": (C.c_char_p, [i32]),
    "sdb_abi_version": (i32, []),
    "sdb_struct_sizes": (i32, [C.POINTER(i64), i32]),
    "sdb_dim_required_bytes": (i32, [C.POINTER(SdbDimDesc), C.POINTER(i64)]),
    "sdb_build_dim": (i32, [C.POINTER(SdbDimDesc), vp, i64, vp, C.POINTER(SdbDim)]),
    "sdb_build_dims": (i32, [i32, C.POINTER(SdbDimDesc), C.POINTER(vp), C.POINTER(i64), vp, C.POINTER(SdbDim)]),
    "sdb_dim_info": (i32, [C.POINTER(SdbDim), C.POINTER(SdbDimSummary)]),
    "sdb_set_fused_events": (i32, [vp, vp]),
    "sdb_read_columns": (i32, [C.POINTER(vp), i32, i64, i32, vp, vp]),
    "sdb_baseline_scratch_bytes": (i32, [i64, C.POINTER(i64)]),
    "sdb_run_star_query_baseline": (i32, [C.POINTER(SdbQuery), C.POINTER(SdbPlan), i32, vp, vp, i64, vp, i64,
                                          vp]),
    "sdb_plan_star_query": (i32, [C.POINTER(SdbQuery), vp, i64, vp, C.POINTER(SdbPlan)]),
    "sdb_run_star_query": (i32, [C.POINTER(SdbQuery), C.POINTER(SdbPlan), vp, vp, i64, vp, i64, vp]),
    "sdb_run_star_query_noalloc": (i32, [C.POINTER(SdbQuery), C.POINTER(SdbPlan), vp, vp, i64, vp]),
    "sdb_finalize_scratch_bytes": (i32, [C.POINTER(SdbPlan), C.POINTER(i64)]),
    "sdb_finalize_groups": (i32, [C.POINTER(SdbPlan), vp, vp, vp, vp, vp, i64, vp, vp, i64, vp]),
}


class SdbError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


_lib = None


def lib():
    """The loaded libsdb (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_07632_amd.build` (there is no fallback)")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        sizes = (i64 * len(STRUCTS))()
        if L.sdb_struct_sizes(sizes, len(STRUCTS)) != 0:
            raise RuntimeError("sdb_struct_sizes failed")
        for s, n in zip(STRUCTS, sizes):
            if C.sizeof(s) != n:
                raise RuntimeError(f"struct {s.__name__}: binding has {C.sizeof(s)} bytes, library {n}")
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        msg = lib().sdb_last_error().decode()
        raise SdbError(status, msg)


def _stream_handle(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _ptr(t) -> int | None:
    return None if t is None else (t.data_ptr() or None)


def check_column(t, what: str, n: int | None = None, device=None, dtype: str = "int32") -> None:
    """Raises ValueError unless ``t`` is a one-dimensional contiguous torch
    tensor of ``dtype`` on the GPU (on ``device`` and of ``n`` elements when
    given): the library reads it through a raw device pointer as a dense array."""
    import torch
    want = {"int32": torch.int32, "int64": torch.int64, "uint8": torch.uint8}[dtype]
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what} must be a torch tensor, not {type(t).__name__}")
    if t.dtype != want:
        raise ValueError(f"{what} must be {dtype}, not {t.dtype}")
    if t.dim() != 1 or not t.is_contiguous():
        raise ValueError(f"{what} must be a one-dimensional contiguous tensor "
                         f"(shape {tuple(t.shape)}, strides {t.stride()})")
    if not t.is_cuda:
        raise ValueError(f"{what} must be on the GPU, not {t.device}")
    if device is not None and t.device != device:
        raise ValueError(f"{what} is on {t.device}, the other inputs on {device}")
    if n is not None and t.numel() != n:
        raise ValueError(f"{what} has {t.numel()} elements, {n} expected")


def _pred(p: dict, col_index: dict) -> SdbPred:
    if p["op"] not in OPS:
        raise ValueError(f"unknown predicate op {p['op']!r}")
    hi = p.get("hi")
    return SdbPred(col_index[p["col"]], OPS[p["op"]], int(p["lo"]), int(hi if hi is not None else 0))


# ---------------------------------------------------------------------------
# dimension tables
# ---------------------------------------------------------------------------

@dataclass
class DimTable:
    """A built lookup table and the device memory it lives in."""
    handle: SdbDim
    desc: SdbDimDesc
    workspace: object                      # torch uint8 tensor (device)
    keep: list = field(default_factory=list)

    @property
    def kind(self) -> str:
        return {1: "dense", 2: "hash"}[self.handle.kind]


def dim_required_bytes(desc: SdbDimDesc) -> int:
    out = i64(0)
    _check(lib().sdb_dim_required_bytes(C.byref(desc), C.byref(out)))
    return out.value


def dim_desc(key, cols: dict, preds: list, payloads: list, kind: str = "auto",
             load_factor: float = 0.0, dense_budget_bytes: int = 0) -> SdbDimDesc:
    """The C descriptor of one dimension: ``key`` and the values of ``cols``
    are int32 device tensors of equal length; ``preds`` are predicate dicts
    naming columns of ``cols``; ``payloads`` name the columns to gather;
    ``dense_budget_bytes`` lets a dense table of that size be built whatever
    its key range."""
    names = list(cols)
    if len(names) > MAX_DIM_COLS:
        raise ValueError("too many dimension columns")
    check_column(key, "dimension key")
    idx = {n: i for i, n in enumerate(names)}
    d = SdbDimDesc()
    d.key = _ptr(key)
    d.n_rows = int(key.numel())
    d.n_cols = len(names)
    for i, n in enumerate(names):
        t = cols[n]
        check_column(t, f"dimension column {n!r}", key.numel(), key.device)
        d.cols[i] = _ptr(t)
    if len(preds) > MAX_DIM_PREDS or len(payloads) > MAX_PAYLOADS:
        raise ValueError("too many dimension predicates or payloads")
    d.n_preds = len(preds)
    for i, p in enumerate(preds):
        d.preds[i] = _pred(p, idx)
    d.n_payloads = len(payloads)
    for i, p in enumerate(payloads):
        d.payload_cols[i] = idx[p]
    d.kind = TABLES[kind]
    d.load_factor = float(load_factor or 0.0)
    d.dense_budget_bytes = int(dense_budget_bytes or 0)
    return d


def build_dim(key, cols: dict, preds: list, payloads: list, kind: str = "auto",
              load_factor: float = 0.0, dense_budget_bytes: int = 0, stream=None, workspace=None) -> DimTable:
    """Builds the lookup table of one dimension (arguments as dim_desc)."""
    import torch
    d = dim_desc(key, cols, preds, payloads, kind, load_factor, dense_budget_bytes)
    need = dim_required_bytes(d)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=key.device)
    check_column(workspace, "dimension workspace", device=key.device, dtype="uint8")
    h = SdbDim()
    _check(lib().sdb_build_dim(C.byref(d), _ptr(workspace), workspace.numel(),
                               _stream_handle(stream), C.byref(h)))
    return DimTable(h, d, workspace, [key] + list(cols.values()))


def dim_info(table) -> dict:
    """sdb_dim_info of a built table (a DimTable or an SdbDim handle), as a dict."""
    h = table.handle if isinstance(table, DimTable) else table
    o = SdbDimSummary()
    _check(lib().sdb_dim_info(C.byref(h), C.byref(o)))
    k = o.n_payloads
    return {"kind": {1: "dense", 2: "hash"}[o.kind], "width": o.width, "n_rows": o.n_rows, "n_pass": o.n_pass,
            "key_min": o.key_min, "key_max": o.key_max, "pass_key_min": o.pass_key_min,
            "pass_key_max": o.pass_key_max, "pass_keys_contiguous": bool(o.pass_keys_contiguous),
            "n_slots": int(o.n_slots), "table_bytes": int(o.table_bytes), "occupancy": o.occupancy,
            "payload_min": list(o.payload_min[:k]), "payload_max": list(o.payload_max[:k]),
            "payload_radix": [int(x) for x in o.payload_radix[:k]], "domain": int(o.domain),
            "filter": FILTER_NAMES.get(o.filter_kind, o.filter_kind), "filter_bytes": int(o.filter_bytes)}


def _join_inputs(dims: dict, dim_keys: dict, jd: dict):
    t = dims[jd["dim"]]
    cols = {}
    for n in [p["col"] for p in jd.get("preds", [])] + list(jd.get("payloads", [])):
        cols.setdefault(n, t[n])
    return (t[dim_keys[jd["dim"]]], cols, jd.get("preds", []), list(jd.get("payloads", [])),
            jd.get("kind", "auto"), jd.get("load_factor", 0.0), jd.get("dense_budget_bytes", 0))


class PreparedDims:
    """The batched build of a query's dimension tables with its arguments
    marshalled once. Every :meth:`build` runs sdb_build_dims again (all of its
    work and both stream synchronizations) on the same descriptors and
    workspaces and refills the same handles in place, so a StarQuery made
    from :attr:`tables` stays valid from one build to the next."""

    def __init__(self, dims: dict, dim_keys: dict, query: dict, workspaces=None):
        import torch
        joins = query.get("joins", [])
        self.n = len(joins)
        inputs = [_join_inputs(dims, dim_keys, jd) for jd in joins]
        self.descs = (SdbDimDesc * max(self.n, 1))()
        for i, args in enumerate(inputs):
            self.descs[i] = dim_desc(*args)
        if workspaces is None:
            workspaces = [torch.empty(dim_required_bytes(self.descs[i]), dtype=torch.uint8,
                                      device=inputs[i][0].device) for i in range(self.n)]
        if len(workspaces) != self.n:
            raise ValueError(f"{len(workspaces)} workspaces for {self.n} joins")
        for i, w in enumerate(workspaces):
            check_column(w, f"workspace of join {i}", device=inputs[i][0].device, dtype="uint8")
        self.ws_ptrs = (C.c_void_p * max(self.n, 1))(*[_ptr(w) for w in workspaces])
        self.ws_bytes = (C.c_int64 * max(self.n, 1))(*[w.numel() for w in workspaces])
        self.outs = (SdbDim * max(self.n, 1))()
        # each table's handle is a view of self.outs, which every build refills
        self.tables = [DimTable(self.outs[i], self.descs[i], workspaces[i],
                                [inputs[i][0]] + list(inputs[i][1].values())) for i in range(self.n)]

    def build(self, stream=None) -> list:
        if self.n:
            _check(lib().sdb_build_dims(self.n, self.descs, self.ws_ptrs, self.ws_bytes, _stream_handle(stream),
                                        self.outs))
        return self.tables


def build_dims(dims: dict, dim_keys: dict, query: dict, stream=None, workspaces=None) -> list:
    """One DimTable per join of ``query`` (dims: name -> {column: int32 device
    tensor}), built by one batched call (two stream synchronizations in all).
    ``workspaces`` (one uint8 device tensor per join, large enough) are reused
    when given."""
    return PreparedDims(dims, dim_keys, query, workspaces).build(stream)


# ---------------------------------------------------------------------------
# queries
# ---------------------------------------------------------------------------

@dataclass
class QueryResult:
    keys: np.ndarray      # int64 [n_groups, n_keys]
    sums: np.ndarray      # int64 [n_groups]
    counts: np.ndarray    # int64 [n_groups]

    def as_rows(self):
        return [(tuple(int(x) for x in k), int(s), int(c))
                for k, s, c in zip(self.keys, self.sums, self.counts)]


class StarQuery:
    """The C query descriptor for one star query over device columns.

    ``fact`` maps column name to an int32 device tensor; ``tables`` is the
    list of DimTable per join (``build_dims``); ``query`` the plain-data
    description. ``force`` may hold terminal ('scalar'|'lds'|'global'|'part'),
    ipt, vector (1 / -1), order (True = keep query order), grid, lds, xcd,
    eager, block, range (-1: no key-range probes), coarse, slice (-1: no
    sliced hash probe, 1: wherever allowed), unroll and window (-1: no LDS
    window, 1: the largest that fits, k >= 2: at most 128 k slots), the
    sdb_query force_* fields of the same names, and segments (-1: one stage
    order for the whole table, 1: an order per row range wherever the
    sampled rows favour one).
    """

    def __init__(self, fact: dict, tables: list, query: dict, force: dict | None = None):
        import torch
        force = dict(force or {})
        needed = []
        for p in query.get("fact_preds", []):
            needed.append(p["col"])
        for jd in query.get("joins", []):
            needed.append(jd["fact_key"])
        agg = query["agg"]
        needed.append(agg["a"])
        if agg["kind"] != "col":
            needed.append(agg["b"])
        names = list(dict.fromkeys(needed))
        if len(names) > MAX_FACT_COLS:
            raise ValueError("too many fact columns")
        idx = {n: i for i, n in enumerate(names)}
        q = SdbQuery()
        n = None
        dev = None
        for i, name in enumerate(names):
            t = fact[name]
            check_column(t, f"fact column {name!r}", n, dev)
            n, dev = t.numel(), t.device
            q.cols[i] = _ptr(t)
        for j, tab in enumerate(tables):
            if dev is not None and tab.workspace.device != dev:
                raise ValueError(f"the table of join {j} is on {tab.workspace.device}, the fact columns on {dev}")
        q.n_fact = int(n or 0)
        q.n_cols = len(names)
        preds = query.get("fact_preds", [])
        if len(preds) > MAX_FACT_PREDS or len(tables) > MAX_JOINS:
            raise ValueError("too many predicates or joins")
        q.n_preds = len(preds)
        for i, p in enumerate(preds):
            q.preds[i] = _pred(p, idx)
        joins = query.get("joins", [])
        assert len(joins) == len(tables)
        q.n_joins = len(joins)
        for j, (jd, tab) in enumerate(zip(joins, tables)):
            q.joins[j] = SdbJoin(idx[jd["fact_key"]], C.pointer(tab.handle))
        gb = query.get("group_by", [])
        if len(gb) > MAX_GROUP_KEYS:
            raise ValueError("too many group keys")
        q.n_group_keys = len(gb)
        for k, (ref, payload) in enumerate(gb):
            j = ref if isinstance(ref, int) else next(i for i, jd in enumerate(joins) if jd["dim"] == ref)
            q.group_keys[k] = SdbGroupKey(j, list(joins[j]["payloads"]).index(payload))
        q.agg = SdbAgg(AGGS[agg["kind"]], idx[agg["a"]], idx[agg["b"]] if agg["kind"] != "col" else 0)
        q.force_terminal = TERMINALS[force.get("terminal", "auto")]
        q.force_ipt = int(force.get("ipt", 0))
        q.force_vector = int(force.get("vector", 0))
        q.force_order = 1 if force.get("order") else 0
        q.grid_blocks = int(force.get("grid", 0))
        q.force_lds = int(force.get("lds", 0))
        q.force_xcd = int(force.get("xcd", 0))
        q.force_eager = int(force.get("eager", 0))
        q.force_block = int(force.get("block", 0))
        q.force_range = int(force.get("range", 0))
        q.force_coarse = int(force.get("coarse", 0))
        q.force_slice = int(force.get("slice", 0))
        q.force_unroll = int(force.get("unroll", 0))
        q.force_window = int(force.get("window", 0))
        q.force_segments = int(force.get("segments", 0))
        q.force_prefilter = int(force.get("prefilter", 0))
        self.q = q
        self.query = query
        self.tables = tables
        self.fact = fact
        self.n_keys = len(gb)
        self.plan_obj = None
        self._plan_scratch = None
        self._run_scratch = None

    # -- steps ------------------------------------------------------------
    def plan(self, stream=None) -> SdbPlan:
        import torch
        if self._plan_scratch is None:
            dev = next(iter(self.fact.values())).device
            self._plan_scratch = torch.empty(PLAN_SCRATCH_BYTES, dtype=torch.uint8, device=dev)
        p = SdbPlan()
        _check(lib().sdb_plan_star_query(C.byref(self.q), _ptr(self._plan_scratch),
                                         self._plan_scratch.numel(), _stream_handle(stream),
                                         C.byref(p)))
        self.plan_obj = p
        return p

    def alloc_outputs(self, plan: SdbPlan | None = None):
        import torch
        plan = plan or self.plan_obj
        dev = next(iter(self.fact.values())).device
        g = int(plan.n_groups)
        return (torch.empty(g, dtype=torch.int64, device=dev), torch.empty(g, dtype=torch.int64, device=dev))

    def run_scratch(self, plan: SdbPlan | None = None):
        """Device scratch for sdb_run_star_query (None when the plan needs none)."""
        import torch
        plan = plan or self.plan_obj
        need = int(plan.run_scratch_bytes)
        if need == 0:
            return None
        if self._run_scratch is None or self._run_scratch.numel() < need:
            dev = next(iter(self.fact.values())).device
            self._run_scratch = torch.empty(need, dtype=torch.uint8, device=dev)
        return self._run_scratch

    def baseline_scratch(self, device):
        """Per-row flags and group ids for :meth:`run_baseline`."""
        import torch
        need = i64(0)
        _check(lib().sdb_baseline_scratch_bytes(int(self.q.n_fact), C.byref(need)))
        return torch.empty(max(int(need.value), 256), dtype=torch.uint8, device=device)

    def run_baseline(self, mode: str, sums, counts, plan: SdbPlan | None = None, stream=None,
                     scratch=None) -> None:
        """The same query as a slow baseline of the fusion ablation: ``mode``
        'per_operator' (one kernel per operator) or 'global_handoff' (one
        kernel whose operators pass flags and group ids through global memory)."""
        plan = plan or self.plan_obj
        if scratch is None:
            scratch = self.baseline_scratch(sums.device)
        self._check_outputs(sums, counts, scratch)
        _check(lib().sdb_run_star_query_baseline(C.byref(self.q), C.byref(plan), BASELINES[mode], _ptr(sums),
                                                 _ptr(counts), sums.numel(), _ptr(scratch), scratch.numel(),
                                                 _stream_handle(stream)))

    def _check_outputs(self, sums, counts, scratch) -> None:
        dev = next(iter(self.fact.values())).device if self.fact else None
        check_column(sums, "sums", device=dev, dtype="int64")
        if counts is not None:
            check_column(counts, "counts", sums.numel(), dev, dtype="int64")
        if scratch is not None:
            check_column(scratch, "run scratch", device=dev, dtype="uint8")

    def run(self, sums, counts, plan: SdbPlan | None = None, stream=None, scratch=None) -> None:
        plan = plan or self.plan_obj
        if scratch is None:
            scratch = self.run_scratch(plan)
        self._check_outputs(sums, counts, scratch)
        nbytes = 0 if scratch is None else scratch.numel()
        _check(lib().sdb_run_star_query(C.byref(self.q), C.byref(plan), _ptr(sums), _ptr(counts),
                                        sums.numel(), _ptr(scratch), nbytes, _stream_handle(stream)))

    def run_noalloc(self, sums, counts, plan: SdbPlan | None = None, stream=None) -> None:
        """sdb_run_star_query_noalloc: the run with the library's fixed device
        scratch (NOALLOC_SCRATCH_BYTES per device) instead of a caller buffer."""
        plan = plan or self.plan_obj
        self._check_outputs(sums, counts, None)
        _check(lib().sdb_run_star_query_noalloc(C.byref(self.q), C.byref(plan), _ptr(sums), _ptr(counts),
                                                sums.numel(), _stream_handle(stream)))

    def finalize(self, sums, counts, plan: SdbPlan | None = None, stream=None, outputs=None):
        """Device compaction; returns (keys, sums, counts, n) device tensors (n: int64[1])."""
        import torch
        plan = plan or self.plan_obj
        dev = sums.device
        g = int(plan.n_groups)
        if outputs is None:
            nb = i64(0)
            _check(lib().sdb_finalize_scratch_bytes(C.byref(plan), C.byref(nb)))
            outputs = (torch.empty((g, max(self.n_keys, 1)), dtype=torch.int32, device=dev),
                       torch.empty(g, dtype=torch.int64, device=dev),
                       torch.empty(g, dtype=torch.int64, device=dev),
                       torch.empty(1, dtype=torch.int64, device=dev),
                       torch.empty(nb.value, dtype=torch.uint8, device=dev))
        k, s, c, n, scratch = outputs
        _check(lib().sdb_finalize_groups(C.byref(plan), _ptr(sums), _ptr(counts), _ptr(k), _ptr(s),
                                         _ptr(c), g, _ptr(n), _ptr(scratch), scratch.numel(),
                                         _stream_handle(stream)))
        return outputs

    def execute(self, stream=None, replan: bool = True, baseline: str | None = None) -> QueryResult:
        """plan -> fused pass (or a ``baseline`` execution, see
        :meth:`run_baseline`) -> compaction, then copy the groups to the host."""
        import torch
        if replan or self.plan_obj is None:
            self.plan(stream)
        sums, counts = self.alloc_outputs()
        if baseline is None:
            self.run(sums, counts, stream=stream)
        else:
            self.run_baseline(baseline, sums, counts, stream=stream)
        k, s, c, n, _ = self.finalize(sums, counts, stream=stream)
        (stream or torch.cuda.current_stream()).synchronize()
        m = int(n.item())
        keys = k[:m, :self.n_keys].to(torch.int64).cpu().numpy()
        return QueryResult(keys.reshape(m, self.n_keys), s[:m].cpu().numpy(), c[:m].cpu().numpy())


def plan_summary(plan: SdbPlan, query: dict | None = None) -> dict:
    stages = []
    for s in range(plan.n_stages):
        kind, i = plan.stage_kind[s], plan.stage_index[s]
        name = None
        if query is not None:
            name = (query["fact_preds"][i]["col"] if kind == 0 else query["joins"][i]["dim"])
        st = {"kind": "pred" if kind == 0 else "probe", "index": i, "name": name,
              "pass": round(plan.stage_pass[s], 6), "pass_alone": round(plan.stage_pass_alone[s], 6)}
        if kind == 1 and plan.stage_range[s]:
            st["table"] = "key_range"
        elif kind == 1:
            st["table"] = LDS_NAMES.get(plan.stage_lds[s], plan.stage_lds[s])
            if plan.stage_coarse[s]:
                st["coarse_slots_per_bit"] = 1 << plan.stage_coarse[s]
            if plan.stage_lds[s] == 5:
                st["window"] = [int(plan.stage_window_lo[s]), int(plan.stage_window_slots[s])]
                st["window_cover"] = round(plan.stage_window_cover[s], 6)
            if plan.stage_defer[s] >= 0:
                st["deferred_gather"] = True
            if plan.slice_bits and s == plan.slice_stage:
                st["table_slices"] = 1 << plan.slice_bits
                if plan.slice_prefilter:
                    st["prefilter"] = True
        stages.append(st)
    return {"stages": stages, "terminal": TERMINAL_NAMES.get(plan.terminal, plan.terminal),
            "ipt": plan.ipt, "vector": plan.vector, "eager": plan.eager, "block": plan.block, "grid": plan.grid,
            "xcd_copies": plan.xcd_copies, "lds_bytes": plan.lds_bytes,
            "n_parts": plan.n_parts, "part_subs": plan.part_subs, "part_cap": int(plan.part_cap),
            "slice_bits": plan.slice_bits, "slice_grid": plan.slice_grid, "unroll": plan.unroll,
            "segments": [{"rows": [int(plan.segment_start[g]), int(plan.segment_start[g + 1])],
                          "order": [int(plan.segment_order[g][i]) for i in range(plan.n_stages)]}
                         for g in range(plan.n_segments)] if plan.n_segments > 1 else None,
            "est_cost": round(plan.est_cost, 4),
            "n_groups": int(plan.n_groups), "sampled_rows": int(plan.sampled_rows),
            "radix": [int(plan.radix[k]) for k in range(plan.n_group_keys)]}


def read_columns(cols: list, out, stream=None, blocks_per_cu: int = 0) -> None:
    """Streaming read of int32 device columns (equal length, 16-byte aligned):
    adds all their values into ``out`` (int64 device tensor of one element),
    asynchronously; the bandwidth reference for the fused pass."""
    n = int(cols[0].numel()) if cols else 0
    ptrs = (vp * max(len(cols), 1))(*[_ptr(c) for c in cols])
    _check(lib().sdb_read_columns(ptrs, len(cols), n, int(blocks_per_cu), _ptr(out), _stream_handle(stream)))


def set_fused_events(start=None, stop=None) -> None:
    """Times the fused kernel of later runs on this thread between two
    torch.cuda.Event objects (recorded on the run's stream), or stops doing so
    when called without events."""
    if start is None or stop is None:
        _check(lib().sdb_set_fused_events(None, None))
        return
    for e in (start, stop):
        if not e.cuda_event:                       # torch creates the HIP event on first record
            e.record()
    _check(lib().sdb_set_fused_events(C.c_void_p(start.cuda_event), C.c_void_p(stop.cuda_event)))
