"""The max with recorded recipients (geot_segment_reduce_max_arg, geot_gather_scatter_max_arg)
and the max gradients that take them (geot_*_backward_max_arg), on the GPU.

Bar:
* out bit-identical to the plain max call's and to the oracle's;
* arg equal, element by element, to the recipients the definition gives on the oracle's
  forward: the lowest row (edge) of the segment whose term equals the maximum (== test, so
  either zero attains a zero maximum), 0xFFFFFFFF where there is none (empty segment, NaN
  maximum). The terms are the rows, or the fp32 products w * x of the fused form;
* the gradients from arg equal to the oracle's max gradients, which find the recipients
  themselves by a forward scan (segment form and grad_w bit for bit, grad_X of the fused
  form within the sum bound, its terms being added in the transposed list's order), and to
  the library's own max gradients, which find them again on the GPU.
Every forced element-parallel shape: many partial levels (one row per group), several
lanes and vector widths, column tiles, tile-major order; long runs of empty segments (the
gap list); bf16 / int32.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import compare, say
from workloads import make_config, random_gather_problem, random_problem

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
NONE = 0xFFFFFFFF


def up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def expected_recipients(terms, index, S, out):
    """The definition on the oracle's forward: per (segment, feature), the lowest row whose
    term equals the maximum (numpy, unbuffered minimum over the rows)."""
    n = terms.shape[0]
    with np.errstate(invalid="ignore"):
        eq = terms == out[index]
    rows = np.where(eq, np.arange(n, dtype=np.uint64)[:, None], np.uint64(NONE))
    arg = np.full(out.shape, NONE, dtype=np.uint64)
    np.minimum.at(arg, index, rows)
    return arg.astype(np.uint32)


def check_arg(got, want, what):
    got = got.cpu().numpy().view(np.uint32)
    bad = got != want
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: recipient differs at {i}: gpu {got[i]} definition {want[i]} "
                             f"({int(bad.sum())} elements)")


CHOICES = [
    None,
    dict(family="ep", rows=1),                      # one row per group: several partial levels
    dict(family="ep", lanes=64, rows=1),            # 4 rows per block
    dict(family="ep", lanes=1, rows=5),
    dict(family="ep", vec=1, rows=3),
    dict(family="ep", lanes=2, rows=7),             # several column tiles
    dict(family="ep", lanes=2, rows=3, flags=4),    # the same tiles one after another
]

SEG_CASES = [
    # seed, nnz, S, F, dist, values, empty_frac
    (11, 20000, 900, 1, "zipf", "int", 0.1),        # integer values: ties everywhere
    (12, 30000, 1500, 3, "lognormal", "normal", 0.05),
    (13, 25000, 700, 32, "uniform", "int", 0.2),
    (14, 8000, 400, 33, "one_heavy", "normal", 0.1),
    (15, 6000, 300, 256, "zipf", "int", 0.0),
    (16, 7000, 6000, 6, "uniform", "normal", 0.6),   # many empty segments
    (17, 4000, 200, 300, "zipf", "normal", 0.1),     # more columns than one tile
]


@pytest.mark.parametrize("case", SEG_CASES, ids=lambda c: f"seed{c[0]}-F{c[3]}-{c[5]}")
def test_segment_max_with_recipients(case):
    seed, nnz, S, F, dist, values, ef = case
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    src, idx = p["src"], p["index"]
    ref = oracle.segment_reduce(src, idx, S, "max")
    want = expected_recipients(src, idx, S, ref)
    g = np.random.default_rng(seed).standard_normal((S, F)).astype(np.float32)
    ref_grad = oracle.segment_reduce_backward(g, idx, "max", src, ref)
    s, i = up(src), up(idx)
    plain = geot.segment_reduce(s, i, S, "max").cpu().numpy()
    for ch in CHOICES:
        say(f"segment max with recipients seed={seed} F={F} choice={ch}")
        out, arg = geot.segment_reduce_max_arg(s, i, S, choice=ch)
        compare(out.cpu().numpy(), ref, "max", None, f"out seed={seed} {ch}")
        assert np.array_equal(out.cpu().numpy().view(np.uint32), plain.view(np.uint32)), f"out vs plain {ch}"
        check_arg(arg, want, f"segment seed={seed} F={F} {ch}")
        gs = geot.segment_reduce_backward_max_arg(up(g), i, arg).cpu().numpy()
        assert np.array_equal(gs.view(np.uint32), ref_grad.astype(np.float32).view(np.uint32)), \
            f"gradient from recipients seed={seed} {ch}"
    # and the library's own max gradient (recipients found again) agrees bit for bit
    mine = geot.segment_reduce_backward(up(g), i, "max", s, up(ref)).cpu().numpy()
    assert np.array_equal(mine.view(np.uint32), gs.view(np.uint32))


GATHER_CASES = [
    # seed, nnz, R, n_x, F, dist, values, weighted
    (21, 30000, 2000, 500, 4, "zipf", "int", True),
    (22, 30000, 2000, 3000, 16, "lognormal", "normal", True),
    (23, 20000, 1000, 200, 3, "uniform", "int", False),
    (24, 12000, 600, 800, 64, "one_heavy", "normal", True),
    (25, 9000, 500, 300, 128, "zipf", "int", True),
    (26, 5000, 300, 400, 300, "zipf", "normal", False),
]


@pytest.mark.parametrize("case", GATHER_CASES, ids=lambda c: f"seed{c[0]}-F{c[4]}-w{int(c[7])}")
def test_gather_max_with_recipients(case):
    seed, nnz, R, nx, F, dist, values, weighted = case
    q = random_gather_problem(seed, nnz, R, nx, F, dist, values, weighted, 0.05)
    X, col, w, row = q["X"], q["col"], q["weight"], q["index"]
    ref = oracle.gather_scatter(X, col, w, row, R, "max")
    terms = (w[:, None] * X[col]).astype(np.float32) if weighted else X[col]
    want = expected_recipients(terms, row, R, ref)
    g = np.random.default_rng(seed).standard_normal((R, F)).astype(np.float32)
    rx, rw = oracle.gather_scatter_backward(X, col, w, row, g, "max", ref)
    ax, aw = oracle.gather_scatter_backward(X, col, w, row, g, "max", ref, absolute=True)
    x, c, wt, r = up(X), up(col), up(w), up(row)
    plain = geot.gather_scatter(x, c, wt, r, R, "max").cpu().numpy()
    for ch in CHOICES:
        say(f"gather max with recipients seed={seed} F={F} choice={ch}")
        out, arg = geot.gather_scatter_max_arg(x, c, wt, r, R, choice=ch)
        compare(out.cpu().numpy(), ref, "max", None, f"out seed={seed} {ch}")
        assert np.array_equal(out.cpu().numpy().view(np.uint32), plain.view(np.uint32)), f"out vs plain {ch}"
        check_arg(arg, want, f"gather seed={seed} F={F} {ch}")
    gx, gw = geot.gather_scatter_backward_max_arg(x, c, wt, r, up(g), arg)
    compare(gx.cpu().numpy(), rx, "sum", ax, f"grad_X from recipients seed={seed}")
    mx, mw = geot.gather_scatter_backward(x, c, wt, r, up(g), "max", up(ref))
    compare(mx.cpu().numpy(), rx, "sum", ax, f"grad_X of the library's own max gradient seed={seed}")
    if weighted:
        compare(gw.cpu().numpy(), rw, "sum", aw, f"grad_w from recipients seed={seed}")
        assert np.array_equal(gw.cpu().numpy().view(np.uint32), mw.cpu().numpy().view(np.uint32))
    else:
        assert gw is None


def test_recipients_of_nan_zeros_and_empty_segments():
    """NaN maxima have no recipient; -0 and +0 both attain a zero maximum, the lower row
    receives; empty segments (long runs of them through the gap list too) have none."""
    nan = np.float32(np.nan)
    rows = [[1.0, nan], [nan, -0.0], [3.0, 0.0], [3.0, -0.0], [-0.0, 2.0], [0.0, 2.0]]
    idx = [0, 0, 2, 2, 50_000, 50_000]
    src = np.array(rows, dtype=np.float32)
    index = np.array(idx, dtype=np.int64)
    S = 60_000
    ref = oracle.segment_reduce(src, index, S, "max")
    want = expected_recipients(src, index, S, ref)
    assert want[0, 0] == NONE and want[0, 1] == NONE   # NaN in both columns
    assert want[2, 0] == 2 and want[2, 1] == 2 and want[50_000, 0] == 4
    for ch in (None, dict(family="ep", rows=1)):
        out, arg = geot.segment_reduce_max_arg(up(src), up(index), S, choice=ch)
        compare(out.cpu().numpy(), ref, "max", None, f"nan/zeros out {ch}")
        check_arg(arg, want, f"nan/zeros {ch}")
    out, arg = geot.segment_reduce_max_arg(up(src[:0]), up(index[:0]), 7)
    assert torch.all(out == 0) and torch.all(arg == -1)


@pytest.mark.parametrize("gather", [False, True])
def test_recipients_with_16bit_storage_and_int32_ids(gather):
    """bf16 storage, int32 ids: the terms are the widened values (and their fp32 products)."""
    if gather:
        q = random_gather_problem(31, 40000, 3000, 900, 32, "zipf", "int", True, 0.05)
        Xb = torch.from_numpy(q["X"]).to(torch.bfloat16)
        Xw = Xb.float().numpy()
        ref = oracle.gather_scatter(Xw, q["col"], q["weight"], q["index"], 3000, "max")
        terms = (q["weight"][:, None] * Xw[q["col"]]).astype(np.float32)
        want = expected_recipients(terms, q["index"], 3000, ref)
        out, arg = geot.gather_scatter_max_arg(Xb.to(DEV), up(q["col"].astype(np.int32)), up(q["weight"]),
                                               up(q["index"].astype(np.int32)), 3000)
    else:
        p = random_problem(32, 50000, 2500, 64, "lognormal", "int", 0.05)
        sb = torch.from_numpy(p["src"]).to(torch.bfloat16)
        sw = sb.float().numpy()
        ref = oracle.segment_reduce(sw, p["index"], 2500, "max")
        want = expected_recipients(sw, p["index"], 2500, ref)
        out, arg = geot.segment_reduce_max_arg(sb.to(DEV), up(p["index"].astype(np.int32)), 2500)
    compare(out.cpu().numpy(), ref, "max", None, "bf16 out")
    check_arg(arg, want, "bf16 / int32")
    # the gradients from these recipients, in the same storage and id types, equal the
    # library's own typed max gradients (which find the recipients again)
    R = out.shape[0]
    g = torch.from_numpy(np.random.default_rng(33).standard_normal((R, out.shape[1])).astype(np.float32)).to(DEV)
    if gather:
        x, c, r, wt = Xb.to(DEV), up(q["col"].astype(np.int32)), up(q["index"].astype(np.int32)), up(q["weight"])
        gx, gw = geot.gather_scatter_backward_max_arg(x, c, wt, r, g, arg)
        mx, mw = geot.gather_scatter_backward(x, c, wt, r, g, "max", out)
        assert torch.equal(gw.view(torch.int32), mw.view(torch.int32)), "bf16 grad_w from recipients"
        assert torch.allclose(gx, mx, rtol=1e-5, atol=1e-5), "bf16 grad_X from recipients"
    else:
        i32 = up(p["index"].astype(np.int32))
        gs = geot.segment_reduce_backward_max_arg(g, i32, arg, torch.bfloat16)
        mine = geot.segment_reduce_backward(g, i32, "max", sb.to(DEV), out)
        assert gs.dtype == torch.bfloat16
        assert torch.equal(gs.view(torch.int16), mine.view(torch.int16)), "bf16 grad_src from recipients"
        # and the oracle's gradient on the widened rows, rounded once to bf16
        ref_g = oracle.segment_reduce_backward(g.cpu().numpy(), p["index"], "max", sw, ref)
        want_g = torch.from_numpy(ref_g.astype(np.float32)).to(torch.bfloat16)
        assert torch.equal(gs.cpu().view(torch.int16), want_g.view(torch.int16)), "bf16 grad_src vs oracle"


def test_spmm_max_with_recipients_sampled():
    """The SpMM workload (61,859,140 edges, 128 columns): out bit-identical to the plain max
    call, recipients equal to the definition on 200 sampled rows (the longest included),
    and the gradients from them bit-identical to the library's own max gradients."""
    c = make_config("c4_spmm")
    X, col, w, row, R, L = c["X"], c["col"], c["weight"], c["index"], c["num_segments"], c["lengths"]
    x, cc, wt, r = up(X), up(col), up(w), up(row)
    say("c4 max with recipients")
    out, arg = geot.gather_scatter_max_arg(x, cc, wt, r, R)
    plain = geot.gather_scatter(x, cc, wt, r, R, "max")
    assert torch.equal(out.view(torch.int32), plain.view(torch.int32))
    starts = np.concatenate([[0], np.cumsum(L)])
    rng = np.random.default_rng(5)
    sample = np.unique(np.concatenate([np.argsort(L)[-8:], rng.integers(0, R, 192)]))
    got = arg[torch.from_numpy(sample).to(DEV)].cpu().numpy().view(np.uint32)
    for k, s in enumerate(sample):   # the oracle's forward on each sampled row's own edges
        a, b = int(starts[s]), int(starts[s + 1])
        z = np.zeros(b - a, dtype=np.int64)
        o = oracle.gather_scatter(X, col[a:b], w[a:b], z, 1, "max")
        terms = (w[a:b, None] * X[col[a:b]]).astype(np.float32)
        want = expected_recipients(terms, z, 1, o)[0]
        want = np.where(want == NONE, NONE, want.astype(np.uint64) + a).astype(np.uint32)
        assert np.array_equal(got[k], want), f"c4 row {s}"
    say("c4 gradients from recipients")
    g = torch.randn(R, 128, device=DEV)
    gx, gw = geot.gather_scatter_backward_max_arg(x, cc, wt, r, g, arg)
    mx, mw = geot.gather_scatter_backward(x, cc, wt, r, g, "max", out)
    assert torch.equal(gw.view(torch.int32), mw.view(torch.int32))
    # grad_X sums each column's recipients' terms in the transposed list's order, which
    # depends on timing: equal up to the rounding of a few terms
    assert torch.allclose(gx, mx, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("ch", [None, dict(family="ep", rows=1), dict(family="ep", lanes=1, rows=3),
                                dict(family="ep", vec=1, rows=2)], ids=["default", "rows1", "lanes1", "vec1"])
def test_recipients_of_minus_infinity(ch):
    """Terms equal to the neutral value of max (-inf), alone in a segment or first in a row
    group's run (one-row runs put every row first): the recipient is the lowest such row
    (edge), not none. Segment and fused forms, against the definition on the oracle's out."""
    rng = np.random.default_rng(95)
    S, F, n = 3000, 4, 9000
    idx = np.sort(rng.integers(0, S, n)).astype(np.int64)
    src = rng.integers(-3, 4, (n, F)).astype(np.float32)
    src[rng.random((n, F)) < 0.5] = -np.inf
    ref = oracle.segment_reduce(src, idx, S, "max")
    want = expected_recipients(src, idx, S, ref)
    say(f"recipients of -inf, segment form, choice={ch}")
    out, arg = geot.segment_reduce_max_arg(up(src), up(idx), S, choice=ch)
    compare(out.cpu().numpy(), ref, "max", None, f"segment -inf {ch}")
    check_arg(arg, want, f"segment -inf {ch}")
    nx = 500
    col = rng.integers(0, nx, n).astype(np.int64)
    X = rng.integers(-3, 4, (nx, F)).astype(np.float32)
    X[rng.random((nx, F)) < 0.5] = -np.inf
    w = np.ones(n, dtype=np.float32)
    refg = oracle.gather_scatter(X, col, w, idx, S, "max")
    terms = X[col] * w[:, None]
    wantg = expected_recipients(terms, idx, S, refg)
    say(f"recipients of -inf, fused form, choice={ch}")
    out, arg = geot.gather_scatter_max_arg(up(X), up(col), up(w), up(idx), S, choice=ch)
    compare(out.cpu().numpy(), refg, "max", None, f"gather -inf {ch}")
    check_arg(arg, wantg, f"gather -inf {ch}")
