"""Helpers for the GPU parity tests: upload, run through the C-ABI binding, compare with the oracle.

Comparison bar:
* max: equal element by element (``==``, so +0 and -0 agree), i.e. exact;
* sum / mean: |gpu - oracle| <= 1e-5 * sum|terms| + 1e-6 per element, where
  sum|terms| comes from the oracle (terms divided by the count for mean).
"""
from __future__ import annotations

import sys

import numpy as np

import oracle

REL, ABS = 1e-5, 1e-6


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare(got, ref, op, abs_terms=None, what=""):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    if op == "max":
        bad = ~(got == ref)
        if bad.any():
            i = np.argwhere(bad)[0]
            raise AssertionError(f"{what}: max differs at {tuple(i)}: gpu {got[tuple(i)]!r} "
                                 f"oracle {ref[tuple(i)]!r} ({int(bad.sum())} elements)")
        return
    assert abs_terms is not None
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    lim = REL * abs_terms + ABS
    bad = ~(err <= lim)
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {op} differs at {i}: gpu {got[i]!r} oracle {ref[i]!r} "
                             f"err {err[i]:.3e} > {lim[i]:.3e} ({int(bad.sum())} elements)")


def oracle_segment(src, index, S, op):
    ref = oracle.segment_reduce(src, index, S, op)
    terms = None if op == "max" else oracle.abs_term_sum(src, index, S, op)
    return ref, terms


def oracle_gather(X, col, w, row, R, op):
    ref = oracle.gather_scatter(X, col, w, row, R, op)
    terms = None if op == "max" else oracle.abs_term_sum(X, row, R, op, col=col, weight=w)
    return ref, terms
