"""Helpers for the GPU tests: upload a workload, run it through the C ABI, compare."""

import numpy as np

import oracle


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm GPU")
    from paper_2607_07632_amd import sdb
    sdb.lib()        # raises when libsdb.so is missing: no fallback


def upload(w, device="cuda", offset: int = 0):
    """Device copies of a workload's columns. ``offset`` > 0 places every fact
    column ``offset`` int32 elements into a larger buffer (misaligned views)."""
    import torch
    fact = {}
    for k, v in w.fact.items():
        t = torch.from_numpy(np.ascontiguousarray(v))
        if offset:
            buf = torch.zeros(v.size + offset + 8, dtype=torch.int32, device=device)
            buf[offset:offset + v.size] = t.to(device)
            fact[k] = buf[offset:offset + v.size]
        else:
            fact[k] = t.to(device)
    dims = {d: {c: torch.from_numpy(np.ascontiguousarray(a)).to(device) for c, a in t.items()}
            for d, t in w.dims.items()}
    return fact, dims


def run_gpu(w, force=None, dev=None, tables=None):
    from paper_2607_07632_amd import sdb
    fact, dims = dev if dev is not None else upload(w)
    if tables is None:
        tables = sdb.build_dims(dims, w.dim_keys, w.query)
    q = sdb.StarQuery(fact, tables, w.query, force)
    res = q.execute()
    return res, q


def oracle_rows(w):
    r = oracle.star_query(w.fact, w.dims, w.dim_keys, w.query)
    return r.as_rows()


def assert_same(got_rows, want_rows, label=""):
    if got_rows != want_rows:
        g, o = dict((k, (s, c)) for k, s, c in got_rows), dict((k, (s, c)) for k, s, c in want_rows)
        missing = [k for k in o if k not in g][:5]
        extra = [k for k in g if k not in o][:5]
        diff = [(k, g[k], o[k]) for k in o if k in g and g[k] != o[k]][:5]
        raise AssertionError(f"{label}: {len(got_rows)} GPU groups vs {len(want_rows)} oracle groups; "
                             f"missing {missing} extra {extra} differing {diff}")
