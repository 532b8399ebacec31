"""CPU oracle for the fused star-schema query (test infrastructure only).

This package is the reference the GPU library is checked against. It is plain,
slow and written to be read against the paper: an inner join of the fact table
with each filtered dimension table, the fact-side predicates, and a scalar or
grouped 64-bit integer SUM (the query shape of the paper's Sections 3.3 and
4.2). It shares no code with the GPU library and never calls it.

Only the test suite, the smoke entry point and the benchmark's CPU-baseline leg
may import this package; the product path never does.
"""

from .star import (  # noqa: F401
    DuplicateKeyError,
    OracleResult,
    star_query,
    eval_pred,
)
