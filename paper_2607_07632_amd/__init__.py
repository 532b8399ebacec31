"""A fused star-schema query engine for one AMD Instinct MI355X (gfx950).

The GPU work lives in libsdb.so (HIP kernels behind the C ABI of
include/sdb.h); ``paper_2607_07632_amd.sdb`` is its ctypes binding.
"""

from . import sdb  # noqa: F401
from .sdb import (  # noqa: F401
    DimTable,
    QueryResult,
    SdbError,
    StarQuery,
    build_dim,
    build_dims,
    lib,
    plan_summary,
)
