"""Helpers for the GPU parity tests: upload, run through the C-ABI binding, compare with the oracle.

Comparison bar:
* max: the same fp32 bit pattern element by element (so the sign of a zero counts),
  or NaN on both sides; i.e. exact;
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
        g32 = np.ascontiguousarray(got, dtype=np.float32)
        r32 = np.ascontiguousarray(ref, dtype=np.float32)
        bad = ~((g32.view(np.uint32) == r32.view(np.uint32)) | (np.isnan(g32) & np.isnan(r32)))
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


def bits_equal(a, b) -> bool:
    """Same shape and the same fp32 bit patterns (so +0 and -0 differ, and NaN equals itself)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    return a.shape == b.shape and np.array_equal(a.view(np.uint32), b.view(np.uint32))


def forward_for_gradient(ref_out, gpu_out, what=""):
    """The forward result a max gradient is taken at: the oracle's `ref_out`.

    Both the library's gradient and the oracle's gradient are given this same array, so
    no expected value derives from a GPU output. The GPU forward `gpu_out` (a tensor or
    an array) must equal it bit for bit, which is checked here first."""
    got = gpu_out.cpu().numpy() if hasattr(gpu_out, "cpu") else np.asarray(gpu_out)
    assert bits_equal(got, ref_out), f"{what}: GPU forward max differs from the oracle's"
    return np.ascontiguousarray(ref_out, dtype=np.float32)
