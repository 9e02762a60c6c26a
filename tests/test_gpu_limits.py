"""GPU parity at the size limits: more than 2^31 rows (64-bit row and chunk
arithmetic, 64-bit counts in the partial levels), one segment of more than
2^31 rows, and a fused call over more than 2^31 edges (forward and gradients).

Inputs are built on the GPU with torch's seeded generator (ternary values, so
every partial sum below 2^24 is exact in fp32); the oracle runs on the rows of
sampled segments copied back to the host.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import compare, forward_for_gradient, say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
BIG = (1 << 31) + 999_999


def lengths(seed, S, total):
    rng = np.random.default_rng(seed)
    w = rng.lognormal(0.0, 0.6, S)
    L = np.floor(w / w.sum() * total).astype(np.int64)
    L[: total - int(L.sum())] += 1
    assert int(L.sum()) == total
    return L


def ternary(n, F, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return torch.randint(-1, 2, (n, F), dtype=torch.int8, device=DEV, generator=g).float()


def sample(L, k, seed):
    rng = np.random.default_rng(seed)
    picks = {0, L.size - 1, int(np.argmax(L)), int(np.argmin(L))}
    picks.update(int(x) for x in rng.choice(L.size, size=k, replace=False))
    return sorted(picks)


def test_more_than_2_31_rows():
    S, F = 3000, 1
    L = lengths(7, S, BIG)
    starts = np.concatenate([[0], np.cumsum(L)])
    idx = torch.repeat_interleave(torch.arange(S, device=DEV), torch.from_numpy(L).to(DEV))
    src = ternary(BIG, F, 7)
    say("limits: 2^31+ rows uploaded")
    for itype in (torch.int64, torch.int32):
        ix = idx if itype == torch.int64 else idx.to(torch.int32)
        outs = {op: geot.segment_reduce(src, ix, S, op).cpu().numpy() for op in ("sum", "mean", "max")}
        say(f"limits: 2^31+ rows reduced ({itype})")
        # the max recording its recipients: row numbers above 2^31 in 32 bits, ternary values so
        # every maximum ties and the lowest attaining row must win
        out_r, arg_r = geot.segment_reduce_max_arg(src, ix, S)
        assert np.array_equal(out_r.cpu().numpy().view(np.uint32), outs["max"].view(np.uint32))
        argh = arg_r.cpu().numpy().view(np.uint32)
        for s in sample(L, 12, 9):
            a, b = int(starts[s]), int(starts[s + 1])
            rows = src[a:b].cpu().numpy()
            m = oracle.segment_reduce(rows, np.zeros(b - a, dtype=np.int64), 1, "max")
            assert argh[s, 0] == a + int(np.flatnonzero(rows[:, 0] == m[0, 0])[0]), (itype, s)
        for s in sample(L, 12, 8):
            a, b = int(starts[s]), int(starts[s + 1])
            rows = src[a:b].cpu().numpy()
            z = np.zeros(b - a, dtype=np.int64)
            for op in ("sum", "max"):   # partial sums are integers below 2^24: exact
                ref = oracle.segment_reduce(rows, z, 1, op)
                assert np.array_equal(outs[op][s:s + 1], ref), (itype, op, s)
            ref = oracle.segment_reduce(rows, z, 1, "mean")
            compare(outs["mean"][s:s + 1], ref, "mean", oracle.abs_term_sum(rows, z, 1, "mean"),
                    f"limits mean segment {s}")
        # the gradients over the same rows: segments from the offsets pass, 64-bit block and row
        # arithmetic, and (max) a 32-bit recipient table holding row numbers above 2^31
        g = torch.from_numpy(np.random.default_rng(12).standard_normal((S, F)).astype(np.float32)).to(DEV)
        gh = g.cpu().numpy()
        # max: the gradient is taken at a forward result whose sampled rows are the oracle's (each
        # equal bit for bit to the GPU forward's), so the compared gradients depend on no GPU output
        gsamp = sample(L, 12, 13)
        out_max = outs["max"].copy()
        for s in gsamp:
            a, b = int(starts[s]), int(starts[s + 1])
            rows = src[a:b].cpu().numpy()
            out_max[s:s + 1] = forward_for_gradient(
                oracle.segment_reduce(rows, np.zeros(b - a, dtype=np.int64), 1, "max"), outs["max"][s:s + 1],
                f"limits max segment {s}")
        for op in ("sum", "mean", "max"):
            out = torch.from_numpy(out_max).to(DEV) if op == "max" else None
            gs = geot.segment_reduce_backward(g, ix, op, src if op == "max" else None, out)
            say(f"limits: 2^31+ rows, gradient {op} ({itype})")
            if op == "max":   # from the recorded recipients: the same gradient
                assert torch.equal(geot.segment_reduce_backward_max_arg(g, ix, arg_r).view(torch.int32),
                                   gs.view(torch.int32)), itype
            for s in gsamp:
                a, b = int(starts[s]), int(starts[s + 1])
                rows = src[a:b].cpu().numpy()
                z = np.zeros(b - a, dtype=np.int64)
                got = gs[a:b].cpu().numpy()
                ref = oracle.segment_reduce_backward(gh[s:s + 1], z, op, rows, out_max[s:s + 1])
                if op == "mean":
                    compare(got, ref, "mean", np.abs(ref.astype(np.float64)), f"limits gradient mean {s}")
                else:
                    assert np.array_equal(got, ref), (itype, op, s)
            del gs
        del ix
    # per-feature conservation over every row (fp64 totals of exact integers)
    tot = torch.sum(src, dim=0, dtype=torch.float64).cpu().numpy()
    assert np.array_equal(np.sum(outs["sum"].astype(np.float64), axis=0), tot)


def test_one_segment_of_more_than_2_31_rows():
    """The count of the only segment exceeds 32 bits; sums pass 2^24, so they are
    compared within the bound (terms = the row count)."""
    F = 2
    src = torch.ones((BIG, F), device=DEV)
    idx = torch.zeros(BIG, dtype=torch.int64, device=DEV)
    say("limits: one 2^31+ segment uploaded")
    got = {op: geot.segment_reduce(src, idx, 1, op).cpu().numpy() for op in ("sum", "mean", "max")}
    terms = np.full((1, F), float(BIG))
    compare(got["sum"], np.full((1, F), float(BIG), dtype=np.float32), "sum", terms, "one segment sum")
    compare(got["mean"], np.ones((1, F), dtype=np.float32), "mean", np.ones((1, F)), "one segment mean")
    assert np.array_equal(got["max"], np.ones((1, F), dtype=np.float32))


def test_fused_more_than_2_31_edges():
    R, nx, F = 1500, 4000, 2
    L = lengths(9, R, BIG)
    starts = np.concatenate([[0], np.cumsum(L)])
    row = torch.repeat_interleave(torch.arange(R, device=DEV), torch.from_numpy(L).to(DEV))
    g = torch.Generator(device=DEV)
    g.manual_seed(9)
    col = torch.randint(0, nx, (BIG,), device=DEV, generator=g)
    X = ternary(nx, F, 10)
    say("limits: 2^31+ edges uploaded")
    got = {op: geot.gather_scatter(X, col, None, row, R, op).cpu().numpy() for op in ("sum", "max")}
    Xh = X.cpu().numpy()
    for r in sample(L, 8, 11):
        a, b = int(starts[r]), int(starts[r + 1])
        c = col[a:b].cpu().numpy()
        z = np.zeros(b - a, dtype=np.int64)
        for op in ("sum", "max"):
            ref = oracle.gather_scatter(Xh, c, None, z, 1, op)
            assert np.array_equal(got[op][r:r + 1], ref), (op, r)
    # The gradients of the sum over the same edges (unit weights): grad_X through the radix
    # transposition (bins of one column) of more than 2^31 records, grad_w over more than 2^31 edges. grad_out is
    # ternary, so every partial sum is an integer below 2^24 and exact in any order.
    g = ternary(R, F, 14)
    w = torch.ones(BIG, device=DEV)
    gx, gw = geot.gather_scatter_backward(X, col, w, row, g, "sum")
    say("limits: 2^31+ edges, gradients")
    gh = g.cpu().numpy()
    # grad_X depends on the edges only through the multiplicity of each (row, column) pair: the
    # oracle takes the distinct pairs as edges weighted by their multiplicity
    mult = torch.zeros(R * nx, dtype=torch.int64, device=DEV)
    step = 1 << 28
    for a in range(0, BIG, step):
        mult += torch.bincount(row[a:a + step] * nx + col[a:a + step], minlength=R * nx)
    mult = mult.cpu().numpy()
    pairs = np.nonzero(mult)[0]                       # row-major: sorted by row
    assert int(mult.sum()) == BIG and int(mult.max()) < (1 << 24)
    rx, _ = oracle.gather_scatter_backward(Xh, pairs % nx, mult[pairs].astype(np.float32), pairs // nx, gh, "sum")
    assert np.array_equal(gx.cpu().numpy(), rx.astype(np.float32)), "grad_X over 2^31+ edges"
    # grad_w on sampled edges (the first, the last, and random ones; sorted, so rows stay sorted)
    rng = np.random.default_rng(15)
    es = np.unique(np.concatenate([[0, BIG - 1], rng.integers(0, BIG, 20000)]))
    et = torch.from_numpy(es).to(DEV)
    _, rw = oracle.gather_scatter_backward(Xh, col[et].cpu().numpy(), np.ones(es.size, dtype=np.float32),
                                           row[et].cpu().numpy(), gh, "sum")
    assert np.array_equal(gw[et].cpu().numpy(), rw.astype(np.float32)), "grad_w over 2^31+ edges"


def test_most_segments():
    """num_segments = 2^31 - 1 (the largest accepted) with 1,000 rows: runs of empty
    segments of about 2.1 M each and one of about 10^9 after the last row, more records
    than the gap list holds (the rest are written by their row groups)."""
    S, F, n = (1 << 31) - 1, 1, 1000
    rng = np.random.default_rng(12)
    idx = np.unique(rng.integers(0, S // 2, size=n)).astype(np.int64)   # sorted, distinct
    idx[-1] = S // 2 + 12345
    n = idx.size
    src = rng.integers(-8, 9, size=(n, F)).astype(np.float32)
    out = torch.full((S, F), 7.0, device=DEV)
    say("limits: 2^31-1 segments")
    geot.segment_reduce(torch.from_numpy(src).to(DEV), torch.from_numpy(idx).to(DEV), S, "sum", out=out)
    torch.cuda.synchronize()
    seg, first = np.unique(idx, return_index=True)
    want = np.add.reduceat(src[:, 0].astype(np.float64), first).astype(np.float32)
    got = out[torch.from_numpy(seg).to(DEV), 0].cpu().numpy()
    assert np.array_equal(got, want)
    assert int(torch.count_nonzero(out).item()) == int(np.count_nonzero(want))
