"""Seeded synthetic star schemas (inputs only).

This package produces the fact columns, dimension tables and query descriptions
that both the CPU oracle and the GPU library consume. It holds none of the
query's arithmetic: no predicate is evaluated, no key is joined and nothing is
summed here. Every array is generated from a counter-addressed seed, so any row
range of any column can be regenerated on its own.
"""

from .star import (  # noqa: F401
    CONFIGS,
    FULL_ROWS,
    Workload,
    make_workload,
    fact_column,
    fact_rows,
    zipf_cdf,
)
