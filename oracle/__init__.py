"""CPU oracle for sorted segment reduction (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the bench's ``cpu_baseline``
leg may import this package. The GPU library never uses it.
"""
from .oracle import (  # noqa: F401
    OPS,
    SOURCE,
    OracleError,
    OracleLib,
    OracleMT,
    MT_SOURCE,
    build,
    build_mt,
    build_all,
    default,
    mt,
    host_threads,
    lib_path,
    check_index,
    segment_reduce,
    gather_scatter,
    abs_term_sum,
    index_stats,
    segment_reduce_backward,
    gather_scatter_backward,
)
