"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each ``pin_*`` function takes an oracle implementation (``oracle.OracleLib``)
and raises ``AssertionError`` when the implementation disagrees with:

* hand-worked examples (``tests/golden/hand_examples.json``);
* brute force over every non-decreasing index of tiny problems, written as the
  literal per-segment filter of the definition (Section II-B) with exact
  integer / rational arithmetic;
* invariants of the definition (conservation of totals, mean times count equals
  sum, empty segments, max is a member and dominates, length-1 segments, S = 1);
* library routines: numpy's unbuffered ``add.at`` / ``maximum.at``, torch's
  ``scatter_reduce`` and a dense fp64 matrix product for the fused form;
* the fusion identity of Listing "GeoT solution for fusion" with the messages
  formed by numpy's own fp32 multiply.

The pins are shared by ``test_oracle_pins.py`` (real oracle must pass every
pin) and ``test_oracle_mutants.py`` (planted mistakes must each fail one).
"""
from __future__ import annotations

import itertools
import json
import os
from fractions import Fraction

import numpy as np

from workloads import random_gather_problem, random_problem

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_examples.json")
OPS = ("sum", "mean", "max")


def within_tol(got, ref, abs_terms, rel=1e-5, absol=1e-6):
    """The fp32 sum/mean bound: |got - ref| <= rel * sum|terms| + absol, per element."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return np.all(np.abs(got - ref) <= rel * np.asarray(abs_terms) + absol)


def _f32(x):
    return np.float32(x)


def _golden_value(entry, op):
    if op == "mean":
        return np.array([[np.float32(n / d) for (n, d) in row] for row in entry], dtype=np.float32)
    return np.array(entry, dtype=np.float32)


# ----------------------------------------------------------------------------
def pin_golden(impl):
    g = json.load(open(GOLDEN))
    sr = g["segment_reduce"]
    src = np.array(sr["src"], dtype=np.float32)
    idx = np.array(sr["index"], dtype=np.int64)
    for op in OPS:
        got = impl.segment_reduce(src, idx, sr["num_segments"], op)
        assert np.array_equal(got, _golden_value(sr[op], op)), f"golden segment_reduce {op}"
    gs = g["gather_scatter"]
    X = np.array(gs["X"], dtype=np.float32)
    col = np.array(gs["col"], dtype=np.int64)
    row = np.array(gs["row"], dtype=np.int64)
    w = np.array(gs["weight"], dtype=np.float32)
    for key, weight in (("weighted", w), ("unweighted", None)):
        for op in OPS:
            got = impl.gather_scatter(X, col, weight, row, gs["num_rows"], op)
            assert np.array_equal(got, _golden_value(gs[key][op], op)), f"golden gather {key} {op}"


# ----------------------------------------------------------------------------
def _brute_segment(values_int, idx, S, F, op):
    """Literal definition: for each segment, filter the rows whose index equals it."""
    out = np.zeros((S, F), dtype=np.float32)
    for s in range(S):
        members = [i for i in range(len(idx)) if idx[i] == s]
        for f in range(F):
            terms = [values_int[i][f] for i in members]
            if not terms:
                out[s, f] = 0.0
            elif op == "sum":
                out[s, f] = _f32(sum(terms))
            elif op == "mean":
                out[s, f] = _f32(float(Fraction(sum(terms), len(terms))))
            else:
                out[s, f] = _f32(max(terms))
    return out


def pin_bruteforce_segment(impl, max_nnz=5, max_S=4, Fs=(1, 3)):
    rng = np.random.default_rng(11)
    for S in range(1, max_S + 1):
        for nnz in range(0, max_nnz + 1):
            for idx_t in itertools.combinations_with_replacement(range(S), nnz):
                idx = np.array(idx_t, dtype=np.int64)
                for F in Fs:
                    vals = rng.integers(-8, 9, size=(nnz, F))
                    src = vals.astype(np.float32).reshape(nnz, F)
                    for op in OPS:
                        want = _brute_segment(vals.tolist(), idx_t, S, F, op)
                        got = impl.segment_reduce(src, idx, S, op)
                        assert np.array_equal(got, want), f"brute segment {op} idx={idx_t} F={F}"


def pin_bruteforce_gather(impl, max_nnz=4, max_R=3, n_x=3, F=2):
    rng = np.random.default_rng(12)
    for R in range(1, max_R + 1):
        for nnz in range(0, max_nnz + 1):
            for row_t in itertools.combinations_with_replacement(range(R), nnz):
                row = np.array(row_t, dtype=np.int64)
                col = rng.integers(0, n_x, nnz).astype(np.int64)
                Xi = rng.integers(-8, 9, size=(n_x, F))
                X = Xi.astype(np.float32)
                wq = rng.integers(-4, 5, nnz)  # weights in quarter steps: products exact
                w = (wq / 4.0).astype(np.float32)
                for weighted in (True, False):
                    msgs = []
                    for e in range(nnz):
                        scale = Fraction(int(wq[e]), 4) if weighted else Fraction(1)
                        msgs.append([scale * int(Xi[col[e], f]) for f in range(F)])
                    for op in OPS:
                        want = np.zeros((R, F), dtype=np.float32)
                        for r in range(R):
                            members = [e for e in range(nnz) if row_t[e] == r]
                            for f in range(F):
                                terms = [msgs[e][f] for e in members]
                                if not terms:
                                    continue
                                if op == "sum":
                                    want[r, f] = _f32(float(sum(terms)))
                                elif op == "mean":
                                    want[r, f] = _f32(float(sum(terms) / len(terms)))
                                else:
                                    want[r, f] = _f32(float(max(terms)))
                        got = impl.gather_scatter(X, col, w if weighted else None, row, R, op)
                        assert np.array_equal(got, want), \
                            f"brute gather {op} weighted={weighted} row={row_t} col={col.tolist()}"


# ----------------------------------------------------------------------------
_INV_CASES = (
    # seed, nnz, S, F, dist, values, empty_frac
    (21, 3000, 200, 3, "uniform", "uniform", 0.1),
    (22, 5000, 300, 1, "zipf", "normal", 0.05),
    (23, 4000, 150, 8, "lognormal", "uniform", 0.0),
    (24, 2000, 50, 5, "one_heavy", "normal", 0.2),
    (25, 1000, 100, 4, "uniform", "negative", 0.1),
)


def pin_invariants(impl):
    for seed, nnz, S, F, dist, values, ef in _INV_CASES:
        p = random_problem(seed, nnz, S, F, dist, values, ef)
        src, idx, L = p["src"], p["index"], p["lengths"]
        out = {op: impl.segment_reduce(src, idx, S, op) for op in OPS}
        abs_sum = np.zeros((S, F))
        np.add.at(abs_sum, idx, np.abs(src.astype(np.float64)))
        # conservation of per-feature totals (sum)
        tot = src.astype(np.float64).sum(axis=0)
        got_tot = out["sum"].astype(np.float64).sum(axis=0)
        assert np.all(np.abs(got_tot - tot) <= 1e-5 * abs_sum.sum(axis=0) + 1e-6 * S), \
            f"conservation case {seed}"
        # empty segments hold 0 for every op
        empty = L == 0
        for op in OPS:
            assert np.all(out[op][empty] == 0.0), f"empty fill {op} case {seed}"
        # mean * count == sum within the bound
        ne = ~empty
        assert within_tol(out["mean"][ne] * L[ne, None], out["sum"][ne], abs_sum[ne]), \
            f"mean*count case {seed}"
        # max: a member of its segment and >= every member
        starts = np.concatenate([[0], np.cumsum(L)])
        for s in np.flatnonzero(ne):
            seg = src[starts[s]:starts[s + 1]]
            assert np.all(out["max"][s] >= seg), f"max dominance seg {s} case {seed}"
            assert np.all((seg == out["max"][s]).any(axis=0)), f"max membership seg {s} case {seed}"
        # length-1 segments return their row unchanged for every op
        for s in np.flatnonzero(L == 1):
            for op in OPS:
                assert np.array_equal(out[op][s], src[starts[s]]), f"length-1 {op} case {seed}"


def pin_single_segment(impl):
    """S = 1 is a column reduction: numpy's fp64 sum / max / mean over axis 0."""
    p = random_problem(31, 4000, 1, 6, "uniform", "normal")
    src, idx = p["src"], p["index"]
    s64 = src.astype(np.float64)
    absum = np.abs(s64).sum(axis=0)
    for op, ref in (("sum", s64.sum(axis=0)), ("mean", s64.mean(axis=0))):
        got = impl.segment_reduce(src, idx, 1, op)[0].astype(np.float64)
        scale = absum if op == "sum" else absum / len(src)
        # one fp32 rounding of the result plus fp64 reordering noise
        assert np.all(np.abs(got - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-12 * scale), f"S=1 {op}"
    assert np.array_equal(impl.segment_reduce(src, idx, 1, "max")[0], src.max(axis=0)), "S=1 max"


def pin_column_independence(impl):
    p = random_problem(32, 3000, 120, 3, "zipf", "normal", 0.1)
    src, idx, S = p["src"], p["index"], p["num_segments"]
    for op in OPS:
        whole = impl.segment_reduce(src, idx, S, op)
        for f in range(3):
            part = impl.segment_reduce(np.ascontiguousarray(src[:, f:f + 1]), idx, S, op)
            assert np.array_equal(whole[:, f:f + 1], part), f"column independence {op} f={f}"


def pin_library_scatter(impl):
    import torch

    for seed, dist, F in ((41, "lognormal", 4), (42, "zipf", 7), (43, "uniform", 1)):
        p = random_problem(seed, 6000, 400, F, dist, "normal", 0.05)
        src, idx, S, L = p["src"], p["index"], p["num_segments"], p["lengths"]
        s64 = src.astype(np.float64)
        acc = np.zeros((S, F))
        np.add.at(acc, idx, s64)  # unbuffered, in row order, fp64
        assert np.array_equal(impl.segment_reduce(src, idx, S, "sum"), acc.astype(np.float32)), \
            f"add.at sum {seed}"
        cnt = np.maximum(L, 1)[:, None]
        assert np.array_equal(impl.segment_reduce(src, idx, S, "mean"),
                              (acc / cnt).astype(np.float32)), f"add.at mean {seed}"
        mx = np.full((S, F), -np.inf, dtype=np.float32)
        np.maximum.at(mx, idx, src)
        mx[L == 0] = 0.0
        assert np.array_equal(impl.segment_reduce(src, idx, S, "max"), mx), f"maximum.at {seed}"
        # torch scatter_reduce on the CPU as a third opinion
        ts = torch.from_numpy(src)
        ti = torch.from_numpy(idx)[:, None].expand(-1, F)
        abs_sum = np.zeros((S, F))
        np.add.at(abs_sum, idx, np.abs(s64))
        for op, tname in (("sum", "sum"), ("mean", "mean"), ("max", "amax")):
            t = torch.zeros(S, F, dtype=torch.float32).scatter_reduce(0, ti, ts, tname,
                                                                     include_self=False).numpy()
            got = impl.segment_reduce(src, idx, S, op)
            if op == "max":
                assert np.array_equal(got, t), f"torch amax {seed}"
            else:
                tol = abs_sum / cnt if op == "mean" else abs_sum
                assert within_tol(got, t, tol), f"torch {op} {seed}"


def pin_dense_matmul(impl):
    for seed, weighted in ((51, True), (52, False)):
        p = random_gather_problem(seed, 3000, 150, 90, 5, "zipf", "normal", weighted, 0.1)
        X, col, w, row, R = p["X"], p["col"], p["weight"], p["index"], p["num_segments"]
        A = np.zeros((R, X.shape[0]))
        np.add.at(A, (row, col), 1.0 if w is None else w.astype(np.float64))
        dense = A @ X.astype(np.float64)
        absA = np.zeros_like(A)
        np.add.at(absA, (row, col), 1.0 if w is None else np.abs(w.astype(np.float64)))
        bound = absA @ np.abs(X.astype(np.float64))
        got = impl.gather_scatter(X, col, w, row, R, "sum")
        assert within_tol(got, dense, bound), f"dense A@X weighted={weighted}"


def pin_fusion_equivalence(impl):
    p = random_gather_problem(61, 4000, 300, 200, 6, "lognormal", "normal", True, 0.05)
    X, col, w, row, R = p["X"], p["col"], p["weight"], p["index"], p["num_segments"]
    msgs = (w[:, None] * X[col]).astype(np.float32)  # numpy fp32 multiply, one rounding
    for op in OPS:
        assert np.array_equal(impl.gather_scatter(X, col, w, row, R, op),
                              impl.segment_reduce(msgs, row, R, op)), f"fusion identity {op}"
        assert np.array_equal(impl.gather_scatter(X, col, None, row, R, op),
                              impl.segment_reduce(np.ascontiguousarray(X[col]), row, R, op)), \
            f"fusion identity unweighted {op}"


def pin_errors(impl):
    from oracle import OracleError

    src = np.ones((4, 2), dtype=np.float32)
    for idx, code in (([0, 2, 1, 3], 2), ([0, 1, 1, 5], 3), ([-1, 0, 0, 1], 3)):
        try:
            impl.segment_reduce(src, np.array(idx, dtype=np.int64), 4, "sum")
        except OracleError as e:
            assert e.code == code, f"error code for {idx}"
        else:
            raise AssertionError(f"no error for {idx}")
    try:
        impl.gather_scatter(src, np.array([0, 9]), None, np.array([0, 1]), 2, "sum")
    except OracleError as e:
        assert e.code == 3
    else:
        raise AssertionError("no error for column out of range")


def pin_max_nan_and_signed_zeros(impl):
    """Max is the IEEE 754-2019 maximum folded over a segment (the paper is silent on NaN and
    on the sign of zero): a NaN member gives NaN wherever it sits, +0 ranks above -0 in either
    order, a segment of only -0 gives -0, and infinities order as numbers. Hand-listed cases,
    compared as fp32 bit patterns; the fused form forms its terms first (w = -1 turns +0
    into -0)."""
    nan, inf = np.float32(np.nan), np.float32(np.inf)
    cases = [
        ([1.0, nan, 5.0], "nan"), ([nan, 1.0], "nan"), ([2.0, 3.0, nan], "nan"),
        ([-0.0, 0.0], 0.0), ([0.0, -0.0], 0.0), ([-0.0, -0.0], -0.0), ([-0.0], -0.0),
        ([-1.0, -0.0, -2.0], -0.0), ([-inf, -3.0], -3.0), ([inf, nan], "nan"), ([-5.0, inf, 2.0], inf),
    ]
    vals = np.array([v for c, _ in cases for v in c], dtype=np.float32).reshape(-1, 1)
    idx = np.repeat(np.arange(len(cases)), [len(c) for c, _ in cases]).astype(np.int64)
    got = impl.segment_reduce(vals, idx, len(cases), "max")[:, 0]
    for k, (c, want) in enumerate(cases):
        if want == "nan":
            assert np.isnan(got[k]), f"max of {c} must be NaN"
        else:
            assert got[k].view(np.uint32) == np.float32(want).view(np.uint32), f"max of {c}: {got[k]!r}"
    X = np.array([[0.0], [3.0], [-0.0]], dtype=np.float32)
    col = np.array([0, 2, 0, 0], dtype=np.int64)
    w = np.array([-1.0, 1.0, 2.0, -1.0], dtype=np.float32)
    row = np.array([0, 0, 1, 1], dtype=np.int64)
    got = impl.gather_scatter(X, col, w, row, 2, "max")[:, 0]
    # row 0: terms -0 and -0 -> -0; row 1: terms +0 and -0 -> +0
    assert got.view(np.uint32).tolist() == [0x80000000, 0x00000000], f"fused max of zeros: {got!r}"


def pin_abs_term_sum(impl):
    p = random_gather_problem(71, 2000, 100, 50, 3, "zipf", "normal", True, 0.1)
    X, col, w, row, R, L = p["X"], p["col"], p["weight"], p["index"], p["num_segments"], p["lengths"]
    msgs = np.abs((w[:, None] * X[col]).astype(np.float32).astype(np.float64))
    want = np.zeros((R, 3))
    np.add.at(want, row, msgs)
    got = impl.abs_term_sum(X, row, R, "sum", col, w)
    assert np.allclose(got, want, rtol=1e-12, atol=0), "abs term sum"
    got_mean = impl.abs_term_sum(X, row, R, "mean", col, w)
    assert np.allclose(got_mean, want / np.maximum(L, 1)[:, None], rtol=1e-12, atol=0), "abs mean"
    # the segment form: the terms are the rows themselves
    q = random_problem(72, 3000, 120, 4, "lognormal", "normal", 0.1)
    src, idx, S, Lq = q["src"], q["index"], q["num_segments"], q["lengths"]
    want = np.zeros((S, 4))
    np.add.at(want, idx, np.abs(src.astype(np.float64)))
    assert np.allclose(impl.abs_term_sum(src, idx, S, "sum"), want, rtol=1e-12, atol=0), "abs segment sum"
    assert np.allclose(impl.abs_term_sum(src, idx, S, "mean"), want / np.maximum(Lq, 1)[:, None],
                       rtol=1e-12, atol=0), "abs segment mean"


def pin_index_stats(impl):
    for seed, dist, ef in ((81, "zipf", 0.1), (82, "fixed", 0.0), (83, "lognormal", 0.3)):
        p = random_problem(seed, 5000, 700, 1, dist, "uniform", ef)
        L = np.bincount(p["index"], minlength=700)
        st = impl.index_stats(p["index"], 700)
        assert st["max_len"] == L.max() and st["num_empty"] == int((L == 0).sum())
        assert st["sum_len_sq"] == int((L.astype(np.int64) ** 2).sum())
        assert abs(st["mean_len"] - L.mean()) <= 1e-12 * L.mean()
        assert abs(st["var_len"] - L.var()) <= 1e-9 * max(L.var(), 1.0)


# ----------------------------------------------------------------------------
# gradients
# ----------------------------------------------------------------------------
def _fd_loss(impl, g, fwd):
    return float((g.astype(np.float64) * fwd().astype(np.float64)).sum())


def pin_backward_finite_differences(impl):
    """grad = d/d input of sum(grad_out * forward(input)), by central differences of the
    (independently pinned) forward oracle. Integer data and half steps keep sum exact;
    mean adds one fp32 rounding; max uses well-separated values so the step never
    changes which member is largest."""
    rng = np.random.default_rng(91)
    for S, F in ((5, 2), (7, 3)):
        L = rng.integers(0, 5, size=S)
        idx = np.repeat(np.arange(S), L).astype(np.int64)
        n = idx.size
        g = rng.integers(-3, 4, size=(S, F)).astype(np.float32)
        for op in ("sum", "mean", "max"):
            if op == "max":
                src = (rng.permutation(n * F).reshape(n, F) * 4.0).astype(np.float32)
            else:
                src = rng.integers(-8, 9, size=(n, F)).astype(np.float32)
            out = impl.segment_reduce(src, idx, S, op)
            got = impl.segment_reduce_backward(g, idx, op, src, out)
            h = 0.5
            for i in range(n):
                for f in range(F):
                    sp, sm = src.copy(), src.copy()
                    sp[i, f] += h
                    sm[i, f] -= h
                    fd = (_fd_loss(impl, g, lambda: impl.segment_reduce(sp, idx, S, op)) -
                          _fd_loss(impl, g, lambda: impl.segment_reduce(sm, idx, S, op))) / (2 * h)
                    tol = 1e-6 * (1 + abs(fd)) if op == "mean" else 0.0
                    assert abs(fd - float(got[i, f])) <= tol, f"segment backward {op} ({i},{f})"
    # fused form: w.r.t. X and weights (quarter-step weights, integer X: exact products)
    for weighted in (True, False):
        R, nx, F = 4, 3, 2
        L = rng.integers(0, 4, size=R)
        row = np.repeat(np.arange(R), L).astype(np.int64)
        n = row.size
        col = rng.integers(0, nx, n).astype(np.int64)
        g = rng.integers(-3, 4, size=(R, F)).astype(np.float32)
        for op in ("sum", "mean", "max"):
            if op == "max":
                X = (rng.permutation(nx * F).reshape(nx, F) * 8.0 + 1.0).astype(np.float32)
                w = (rng.permutation(n) + 1.0).astype(np.float32) if weighted else None
            else:
                X = rng.integers(-8, 9, size=(nx, F)).astype(np.float32)
                w = (rng.integers(-4, 5, n) / 4.0).astype(np.float32) if weighted else None
            out = impl.gather_scatter(X, col, w, row, R, op)
            gX, gw = impl.gather_scatter_backward(X, col, w, row, g, op, out)
            fwd = lambda Xv, wv: impl.gather_scatter(Xv, col, wv, row, R, op)
            h = 0.125 if op == "max" else 0.5
            for c in range(nx):
                for f in range(F):
                    Xp, Xm = X.copy(), X.copy()
                    Xp[c, f] += h
                    Xm[c, f] -= h
                    fd = (_fd_loss(impl, g, lambda: fwd(Xp, w)) - _fd_loss(impl, g, lambda: fwd(Xm, w))) / (2 * h)
                    assert abs(fd - gX[c, f]) <= 1e-6 * (1 + abs(fd)), f"gather grad_X {op} ({c},{f})"
            if weighted:
                hw = 1.0 / 64 if op == "max" else 0.25
                for e in range(n):
                    wp, wm = w.copy(), w.copy()
                    wp[e] += hw
                    wm[e] -= hw
                    fd = (_fd_loss(impl, g, lambda: fwd(X, wp)) - _fd_loss(impl, g, lambda: fwd(X, wm))) / (2 * hw)
                    assert abs(fd - gw[e]) <= 1e-6 * (1 + abs(fd)), f"gather grad_w {op} e={e}"


def pin_backward_max_ties(impl):
    """With ties, the max gradient is a subgradient: per (segment, feature) it sums to
    grad_out, goes to one member that attains the max, and (the tie reading) to the
    lowest-indexed such member. The same for the fused form's X gradient."""
    rng = np.random.default_rng(95)
    p = random_problem(96, 4000, 300, 3, "zipf", "int", 0.1)  # values in [-8, 8]: many ties
    src, idx, S, L = p["src"], p["index"], p["num_segments"], p["lengths"]
    g = rng.integers(1, 5, size=(S, 3)).astype(np.float32)
    out = impl.segment_reduce(src, idx, S, "max")
    got = impl.segment_reduce_backward(g, idx, "max", src, out)
    starts = np.concatenate([[0], np.cumsum(L)])
    for s_ in np.flatnonzero(L > 0):
        seg = src[starts[s_]:starts[s_ + 1]]
        gs = got[starts[s_]:starts[s_ + 1]]
        for f in range(3):
            nz = np.flatnonzero(gs[:, f])
            assert nz.size == 1 and gs[nz[0], f] == g[s_, f], f"one recipient seg {s_} f {f}"
            assert seg[nz[0], f] == out[s_, f], f"recipient attains the max seg {s_}"
            assert nz[0] == np.flatnonzero(seg[:, f] == out[s_, f])[0], f"lowest index seg {s_}"
    q = random_gather_problem(97, 3000, 200, 40, 2, "zipf", "int", True, 0.1)
    X, col, w, row, R = q["X"], q["col"], q["weight"], q["index"], q["num_segments"]
    g = rng.integers(1, 5, size=(R, 2)).astype(np.float32)
    out = impl.gather_scatter(X, col, w, row, R, "max")
    gX, gw = impl.gather_scatter_backward(X, col, w, row, g, "max", out)
    # every (row, feature) routes exactly one term: total |dX| mass = sum_r,f |w_e*| g
    nonempty = np.bincount(row, minlength=R) > 0
    msgs = (w[:, None] * X[col]).astype(np.float32)
    want_total = 0.0
    starts = np.concatenate([[0], np.cumsum(q["lengths"])])
    for r in np.flatnonzero(nonempty):
        for f in range(2):
            e = starts[r] + np.flatnonzero(msgs[starts[r]:starts[r + 1], f] == out[r, f])[0]
            want_total += float(w[e]) * float(g[r, f])
    assert abs(gX.sum() - want_total) <= 1e-9 * max(1.0, abs(want_total)), "fused max recipients"


def pin_backward_absolute_terms(impl):
    """The fused gradients' sums of |terms| (what the gradient tolerance is made of), against
    numpy's unbuffered add.at of the absolute per-edge terms: |coef(e) * grad_out[row[e], f]|
    into grad_X[col[e], f] and |grad_out[row[e], f] * X[col[e], f]| into grad_w[e], divided by
    the row's edge count for mean; for max only the lowest edge of each (row, feature) whose
    rounded product equals the maximum (found here with numpy's maximum.at) contributes."""
    rng = np.random.default_rng(98)
    for weighted in (True, False):
        q = random_gather_problem(99, 2500, 160, 70, 3, "zipf", "int", weighted, 0.1)
        X, col, w, row, R, L = q["X"], q["col"], q["weight"], q["index"], q["num_segments"], q["lengths"]
        n, F = row.size, 3
        g = rng.standard_normal((R, F)).astype(np.float32)
        coef = (w if weighted else np.ones(n, dtype=np.float32)).astype(np.float64)
        msgs = (w[:, None] * X[col]).astype(np.float32) if weighted else X[col]
        mx = np.full((R, F), -np.inf, dtype=np.float32)
        np.maximum.at(mx, row, msgs)
        mx[L == 0] = 0.0
        starts = np.concatenate([[0], np.cumsum(L)])
        for op in OPS:
            use = np.ones((n, F), dtype=bool)
            if op == "max":
                use[:] = False
                for r in np.flatnonzero(L > 0):
                    for f in range(F):
                        e = starts[r] + np.flatnonzero(msgs[starts[r]:starts[r + 1], f] == mx[r, f])[0]
                        use[e, f] = True
            div = np.maximum(L, 1)[row].astype(np.float64)[:, None] if op == "mean" else 1.0
            gr = g[row].astype(np.float64)
            tx = np.where(use, np.abs(coef[:, None] * gr) / div, 0.0)
            tw = np.where(use, np.abs(gr * X[col].astype(np.float64)) / div, 0.0)
            want_x = np.zeros((X.shape[0], F))
            np.add.at(want_x, col, tx)
            want_w = tw.sum(axis=1)
            out = impl.gather_scatter(X, col, w, row, R, op) if op == "max" else None
            ax, aw = impl.gather_scatter_backward(X, col, w, row, g, op, out, absolute=True)
            assert np.allclose(ax, want_x, rtol=1e-12, atol=0), f"|terms| of grad_X {op} weighted={weighted}"
            if weighted:
                assert np.allclose(aw, want_w, rtol=1e-12, atol=0), f"|terms| of grad_w {op}"
            # and they bound the signed gradients
            sx, sw = impl.gather_scatter_backward(X, col, w, row, g, op, out)
            assert np.all(np.abs(sx) <= ax * (1 + 1e-12)), f"|grad_X| <= sum |terms| {op}"
            if weighted:
                assert np.all(np.abs(sw) <= aw * (1 + 1e-12)), f"|grad_w| <= sum |terms| {op}"


def pin_backward_torch_autograd(impl):
    """torch's autograd of scatter_reduce / index_select on the CPU (tie-free data)."""
    import torch

    rng = np.random.default_rng(92)
    p = random_problem(93, 3000, 200, 5, "zipf", "normal", 0.1)
    src, idx, S = p["src"], p["index"], p["num_segments"]
    g = rng.standard_normal((S, 5)).astype(np.float32)
    for op, tname in (("sum", "sum"), ("mean", "mean"), ("max", "amax")):
        ts = torch.from_numpy(src.astype(np.float64)).requires_grad_(True)
        ti = torch.from_numpy(idx)[:, None].expand(-1, 5)
        o = torch.zeros(S, 5, dtype=torch.float64).scatter_reduce(0, ti, ts, tname, include_self=False)
        (o * torch.from_numpy(g.astype(np.float64))).sum().backward()
        out = impl.segment_reduce(src, idx, S, op)
        got = impl.segment_reduce_backward(g, idx, op, src, out)
        assert np.allclose(got, ts.grad.numpy(), rtol=1e-6, atol=1e-7), f"torch autograd {op}"
    q = random_gather_problem(94, 2000, 150, 120, 4, "lognormal", "normal", True, 0.1)
    X, col, w, row, R = q["X"], q["col"], q["weight"], q["index"], q["num_segments"]
    g = rng.standard_normal((R, 4)).astype(np.float32)
    for op, tname in (("sum", "sum"), ("mean", "mean")):
        tX = torch.from_numpy(X.astype(np.float64)).requires_grad_(True)
        tw = torch.from_numpy(w.astype(np.float64)).requires_grad_(True)
        msg = tX[torch.from_numpy(col)] * tw[:, None]
        ti = torch.from_numpy(row)[:, None].expand(-1, 4)
        o = torch.zeros(R, 4, dtype=torch.float64).scatter_reduce(0, ti, msg, tname, include_self=False)
        (o * torch.from_numpy(g.astype(np.float64))).sum().backward()
        gX, gw = impl.gather_scatter_backward(X, col, w, row, g, op)
        assert np.allclose(gX, tX.grad.numpy(), rtol=1e-9, atol=1e-9), f"torch grad_X {op}"
        assert np.allclose(gw, tw.grad.numpy(), rtol=1e-9, atol=1e-9), f"torch grad_w {op}"


ALL_PINS = (
    pin_golden,
    pin_bruteforce_segment,
    pin_bruteforce_gather,
    pin_invariants,
    pin_single_segment,
    pin_column_independence,
    pin_library_scatter,
    pin_dense_matmul,
    pin_fusion_equivalence,
    pin_errors,
    pin_max_nan_and_signed_zeros,
    pin_abs_term_sum,
    pin_index_stats,
    pin_backward_finite_differences,
    pin_backward_max_ties,
    pin_backward_absolute_terms,
    pin_backward_torch_autograd,
)
