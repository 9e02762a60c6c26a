"""The multi-threaded oracle equals the serial oracle bit for bit (CPU only).

It computes every output element with the serial oracle's operations in the
same order, only on a thread of its own, so sum, mean, max and the sums of
|terms| must all be identical, for any thread count (1, 3, 8 and more
threads than segments) and for the segment and fused forms, weighted or not,
with empty segments, NaN and signed zeros.
"""
import numpy as np
import pytest

import oracle
from workloads import random_gather_problem, random_problem

OPS = ("sum", "mean", "max")


def same_bits(a, b):
    return a.dtype == b.dtype and a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("threads", [1, 3, 8, 5000])
def test_segment_form_bit_identical(threads):
    m = oracle.OracleMT(oracle.mt().path, threads)
    for seed, nnz, S, F, dist, ef in ((1, 20000, 900, 3, "zipf", 0.1), (2, 5000, 3000, 16, "lognormal", 0.5),
                                      (3, 30000, 1, 2, "fixed", 0.0), (4, 1, 40, 5, "uniform", 0.0)):
        p = random_problem(seed, nnz, S, F, dist, "normal", ef)
        src, idx = p["src"], p["index"]
        if seed == 2:   # NaN and zeros of both signs in some rows
            src[::97, 0] = np.nan
            src[1::5, 1] = -0.0
            src[2::5, 1] = 0.0
        for op in OPS:
            assert same_bits(m.segment_reduce(src, idx, S, op), oracle.segment_reduce(src, idx, S, op)), (seed, op)
            assert same_bits(m.abs_term_sum(src, idx, S, op), oracle.abs_term_sum(src, idx, S, op)), (seed, op)


@pytest.mark.parametrize("weighted", [True, False])
def test_fused_form_bit_identical(weighted):
    q = random_gather_problem(7, 20000, 1500, 900, 6, "zipf", "normal", weighted, 0.1)
    X, col, w, row = q["X"], q["col"], q["weight"], q["index"]
    for threads in (1, 4, 16):
        m = oracle.OracleMT(oracle.mt().path, threads)
        for op in OPS:
            assert same_bits(m.gather_scatter(X, col, w, row, 1500, op),
                             oracle.gather_scatter(X, col, w, row, 1500, op)), (threads, op)
            assert same_bits(m.abs_term_sum(X, row, 1500, op, col, w),
                             oracle.abs_term_sum(X, row, 1500, op, col=col, weight=w)), (threads, op)


def test_errors_match_the_serial_oracle():
    m = oracle.mt()
    src = np.zeros((3, 2), dtype=np.float32)
    with pytest.raises(oracle.OracleError) as e:
        m.segment_reduce(src, np.array([1, 0, 2]), 3, "sum")
    assert e.value.code == 2
    with pytest.raises(oracle.OracleError) as e:
        m.segment_reduce(src, np.array([0, 1, 3]), 3, "sum")
    assert e.value.code == 3
    with pytest.raises(oracle.OracleError) as e:
        m.gather_scatter(src, np.array([0, 9]), None, np.array([0, 1]), 2, "sum")
    assert e.value.code == 3
