"""GPU parity of the gradients (geot_segment_reduce_backward, geot_gather_scatter_backward)
against the CPU oracle.

Bar: segment sum and max gradients copy values, so they are bit-exact; mean is one
division (within the fp32 bound); the fused gradients are sums within
1e-5 * sum|terms| + 1e-6 per element, with sum|terms| from the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import forward_for_gradient, say
from workloads import make_config, random_gather_problem, random_problem

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def within(got, ref, terms, what):
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    lim = 1e-5 * terms + 1e-6
    bad = ~(err <= lim)
    assert not bad.any(), f"{what}: {int(bad.sum())} elements, first at {np.argwhere(bad)[0]}"


SEG_CASES = [
    (1, 20000, 900, 1, "zipf", "normal", 0.1),
    (2, 30000, 1500, 3, "lognormal", "normal", 0.05),
    (3, 25000, 700, 32, "uniform", "int", 0.2),
    (4, 8000, 400, 33, "one_heavy", "normal", 0.1),
    (5, 6000, 300, 256, "zipf", "normal", 0.0),
    (6, 7000, 400, 6, "zipf", "int", 0.1),          # 2-wide vectors; integer values tie often
    (7, 4000, 200, 300, "zipf", "normal", 0.1),     # more vectors than a row's 64 threads
]


@pytest.mark.parametrize("case", SEG_CASES, ids=lambda c: f"seed{c[0]}-F{c[3]}")
def test_segment_backward_parity(case):
    seed, nnz, S, F, dist, values, ef = case
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    src, idx = p["src"], p["index"]
    g = np.random.default_rng(seed).standard_normal((S, F)).astype(np.float32)
    for op in ("sum", "mean", "max"):
        say(f"segment backward seed={seed} F={F} {op}")
        out_np = None
        if op == "max":
            out_np = forward_for_gradient(oracle.segment_reduce(src, idx, S, op),
                                          geot.segment_reduce(up(src), up(idx), S, op), f"seed={seed}")
        got = geot.segment_reduce_backward(up(g), up(idx), op, up(src), up(out_np)).cpu().numpy()
        ref = oracle.segment_reduce_backward(g, idx, op, src, out_np)
        if op == "mean":
            terms = np.abs(ref.astype(np.float64))
            within(got, ref, terms, f"segment backward mean seed={seed}")
        else:
            assert np.array_equal(got, ref), f"segment backward {op} seed={seed} F={F}"


def _offsets_case(case):
    """(src, index, S, F) of a gradient case that takes its segments from the offsets: at least
    64 MB of grad_src and segments averaging at least a block's rows (128 at F = 32, fp32)."""
    seed, kind, F = case
    if kind == "tiny_then_long":
        # 2,000 segments of 0 or 1 rows first (a block spans several hundred segment ends: its
        # rows read their ids), then 1,000 segments of about 3,000 rows
        rng = np.random.default_rng(seed)
        L = np.concatenate([(rng.random(2000) < 0.2).astype(np.int64), rng.integers(2500, 3500, 1000)])
        idx = np.repeat(np.arange(L.size), L)
        src = rng.integers(-3, 4, (idx.size, F)).astype(np.float32)
        return src, idx, L.size, F
    nnz, S, dist, ef = {"one_heavy": (6_000_000, 40_000, "one_heavy", 0.3),
                        "zipf": (4_000_000, 20_000, "zipf", 0.2),
                        "one_segment": (700_001, 1, "uniform", 0.0),
                        "wide": (300_000, 1000, "zipf", 0.1)}[kind]
    p = random_problem(seed, nnz, S, F, dist, "int", ef)   # integer values: max ties
    return p["src"], p["index"], S, F


@pytest.mark.parametrize("case", [
    (8, "one_heavy", 32),        # one segment of most rows, many short and empty ones
    (9, "tiny_then_long", 32),   # blocks spanning > 255 segment ends
    (10, "zipf", 64),
    (11, "one_segment", 32),     # every block lies in it; ragged last block
    (12, "wide", 300),           # 75 vectors a row: more than a row's 64 threads, 16 rows a block
], ids=lambda c: f"seed{c[0]}-{c[1]}")
def test_segment_backward_from_offsets(case):
    """Large gradients: each row's segment comes from the offsets (staged per block) rather than
    the ids; sum and max bit-exact, mean within the bound, against the oracle."""
    src, idx, S, F = _offsets_case(case)
    seed = case[0]
    assert src.nbytes >= (64 << 20) and idx.size >> {32: 7, 64: 6, 300: 4}[F] >= S
    g = np.random.default_rng(seed).standard_normal((S, F)).astype(np.float32)
    for op in ("sum", "mean", "max"):
        say(f"segment backward from offsets seed={seed} {case[1]} {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.segment_reduce(src, idx, S, op),
                                       geot.segment_reduce(up(src), up(idx), S, op), f"seed={seed}")
        got = geot.segment_reduce_backward(up(g), up(idx), op, up(src) if out is not None else None,
                                           up(out)).cpu().numpy()
        ref = oracle.segment_reduce_backward(g, idx, op, src, out)
        if op == "mean":
            within(got, ref, np.abs(ref.astype(np.float64)), f"mean seed={seed}")
        else:
            assert np.array_equal(got, ref), f"{op} seed={seed}"


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float16], ids=["bf16", "f16"])
@pytest.mark.parametrize("case", [(9, "tiny_then_long", 32), (12, "wide", 300)],
                         ids=lambda c: f"seed{c[0]}-{c[1]}")
def test_segment_backward_from_offsets_16bit(case, dt):
    """The same from 16-bit storage with int32 ids (8-element vectors and 256 rows a block at
    F = 32; 4-element vectors and 16 rows at F = 300; the gradient stored non-temporally in
    src's type): sum and max are the oracle's gradient
    rounded once to the type (torch rounds to nearest even, as the library does), mean is
    within half a unit in the last place (plus the fp32 bound) of the exact quotient. The
    integer source values are exact in both types."""
    src, idx, S, F = _offsets_case(case)
    seed = case[0]
    assert src.size * 2 >= (64 << 20) and idx.size >> {32: 8, 300: 4}[F] >= S
    s16 = up(src).to(dt)
    i32 = up(idx).to(torch.int32)
    g = np.random.default_rng(seed).standard_normal((S, F)).astype(np.float32)
    half_ulp = 2.0 ** -8 if dt == torch.bfloat16 else 2.0 ** -11
    for op in ("sum", "mean", "max"):
        say(f"16-bit segment backward from offsets seed={seed} {case[1]} {dt} {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.segment_reduce(src, idx, S, op),
                                       geot.segment_reduce(s16, i32, S, op), f"seed={seed} {dt}")
        got = geot.segment_reduce_backward(up(g), i32, op, s16 if out is not None else None, up(out),
                                           dtype=dt).cpu()
        assert got.dtype == dt
        ref = oracle.segment_reduce_backward(g, idx, op, src, out)
        if op == "mean":
            r = np.abs(ref.astype(np.float64))
            err = np.abs(got.float().numpy().astype(np.float64) - ref.astype(np.float64))
            assert np.all(err <= (half_ulp + 1e-6) * r + 2.0 ** -25), f"mean seed={seed} {dt}"
        else:
            assert torch.equal(got, torch.from_numpy(np.ascontiguousarray(ref)).to(dt)), f"{op} seed={seed} {dt}"


GS_CASES = [
    (11, 20000, 1200, 900, 32, "zipf", "normal", True),
    (12, 15000, 800, 2000, 3, "lognormal", "normal", True),
    (13, 10000, 500, 700, 64, "uniform", "normal", False),
    (14, 8000, 300, 3000, 128, "one_heavy", "normal", True),
    (15, 5000, 400, 400, 17, "poisson", "int", True),
    (16, 6000, 500, 600, 6, "zipf", "int", True),        # 2-wide vectors, ties
    (17, 3000, 200, 400, 300, "zipf", "int", True),      # 75 vectors a row: more than a row's 64 threads
    (18, 5000, 300, 500, 256, "zipf", "int", True),      # 64 threads a row: whole-wave groups, ties
    (19, 7000, 400, 600, 100, "one_heavy", "normal", False),   # 25 vectors on 32 threads (7 idle)
    (20, 8000, 500, 900, 16, "poisson", "normal", True),    # 4 threads a row: every lane stores an edge
]


@pytest.mark.parametrize("case", GS_CASES, ids=lambda c: f"seed{c[0]}-F{c[4]}-w{int(c[7])}")
def test_gather_backward_parity(case):
    seed, nnz, R, nx, F, dist, values, weighted = case
    q = random_gather_problem(seed, nnz, R, nx, F, dist, values, weighted, 0.05)
    X, col, w, row = q["X"], q["col"], q["weight"], q["index"]
    g = np.random.default_rng(seed).standard_normal((R, F)).astype(np.float32)
    for op in ("sum", "mean", "max"):
        say(f"gather backward seed={seed} F={F} {op}")
        out_np = None
        if op == "max":
            out_np = forward_for_gradient(oracle.gather_scatter(X, col, w, row, R, op),
                                          geot.gather_scatter(up(X), up(col), up(w), up(row), R, op),
                                          f"seed={seed}")
        gx, gw = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(g), op, up(out_np))
        rx, rw = oracle.gather_scatter_backward(X, col, w, row, g, op, out_np)
        ax, aw = oracle.gather_scatter_backward(X, col, w, row, g, op, out_np, absolute=True)
        within(gx.cpu().numpy(), rx, ax, f"grad_X {op} seed={seed}")
        if weighted:
            within(gw.cpu().numpy(), rw, aw, f"grad_w {op} seed={seed}")
        else:
            assert gw is None


@pytest.mark.parametrize("F", [3, 8, 64, 300])
def test_gather_backward_max_nonfinite_values(F):
    """Max gradients where X holds infinities and NaNs: an edge takes part in a feature's
    weight-gradient product only where it is that feature's recipient, so an infinity or NaN in
    another feature of its X row cannot turn its gradient into NaN (0 * inf). Columns repeat
    inside rows, so +inf maxima tie and the first edge receives. Against the oracle, which
    sums over the recipient features only: the same non-finite entries, the rest within the
    bound. Widths with one vector per thread and with more vectors than a row's threads."""
    rng = np.random.default_rng(90 + F)
    nx, R = 40, 30
    X = rng.standard_normal((nx, F)).astype(np.float32)
    u = rng.random((nx, F))
    X[u < 0.15] = np.inf
    X[(u >= 0.15) & (u < 0.2)] = np.nan
    lengths = rng.integers(0, 9, R)
    row = np.repeat(np.arange(R), lengths).astype(np.int64)
    col = rng.integers(0, nx, row.size).astype(np.int64)
    col[1::3] = col[0::3][:col[1::3].size]   # repeated columns next to each other
    w = rng.uniform(0.5, 1.5, row.size).astype(np.float32)
    g = rng.standard_normal((R, F)).astype(np.float32)
    out_np = forward_for_gradient(oracle.gather_scatter(X, col, w, row, R, "max"),
                                  geot.gather_scatter(up(X), up(col), up(w), up(row), R, "max"), f"F={F}")
    gx, gw = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(g), "max", up(out_np))
    rx, rw = oracle.gather_scatter_backward(X, col, w, row, g, "max", out_np)
    ax, aw = oracle.gather_scatter_backward(X, col, w, row, g, "max", out_np, absolute=True)
    within(gx.cpu().numpy(), rx, ax, f"grad_X max, non-finite X, F={F}")
    got = gw.cpu().numpy().astype(np.float64)
    fin = np.isfinite(rw)
    assert np.array_equal(np.isnan(got), np.isnan(rw)), f"grad_w NaN pattern F={F}"
    assert np.array_equal(got[np.isinf(rw)], rw[np.isinf(rw)]), f"grad_w infinities F={F}"
    assert (~fin).any() and fin.any()
    within(got[fin], rw[fin], aw[fin], f"grad_w max, non-finite X, F={F}")


def test_backward_edge_cases():
    # no rows: grad_src is empty; fused form with no edges: grad_X is all zeros
    g = up(np.ones((4, 3), dtype=np.float32))
    e = geot.segment_reduce_backward(g, up(np.zeros(0, dtype=np.int64)), "sum")
    assert e.shape == (0, 3)
    X = up(np.ones((5, 3), dtype=np.float32))
    gx, _ = geot.gather_scatter_backward(X, up(np.zeros(0, dtype=np.int64)), None,
                                         up(np.zeros(0, dtype=np.int64)), g, "sum", need_weight=False)
    assert torch.all(gx == 0)
    with pytest.raises(ValueError):
        geot.segment_reduce_backward(g, up(np.zeros(2, dtype=np.int64)), "max")


def test_gradients_match_a_torch_training_step():
    """A GNN-style step: loss = sum(out * t) with out = gather_scatter(X, w); the library's
    gradients equal torch autograd of the same expression in fp64 on the GPU."""
    q = random_gather_problem(16, 40000, 2000, 2000, 16, "zipf", "normal", True, 0.0)
    X, col, w, row, R = q["X"], q["col"], q["weight"], q["index"], q["num_segments"]
    t = np.random.default_rng(17).standard_normal((R, 16)).astype(np.float32)
    tX = torch.from_numpy(X).to(DEV).double().requires_grad_(True)
    tw = torch.from_numpy(w).to(DEV).double().requires_grad_(True)
    msg = tX[up(col)] * tw[:, None]
    o = torch.zeros(R, 16, dtype=torch.float64, device=DEV).index_add(0, up(row), msg)
    (o * up(t).double()).sum().backward()
    gx, gw = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(t), "sum")
    ax, aw = oracle.gather_scatter_backward(X, col, w, row, t, "sum", absolute=True)
    within(gx.cpu().numpy(), tX.grad.cpu().numpy(), ax, "grad_X vs torch")
    within(gw.cpu().numpy(), tw.grad.cpu().numpy(), aw, "grad_w vs torch")


@pytest.mark.parametrize("weighted", [True, False])
@pytest.mark.parametrize("op", ["sum", "mean"])
def test_transpose_edges(weighted, op):
    """geot_transpose_edges: the same (column, row, coefficient) triples, sorted by column
    (the order inside a column is free, so both sides are compared in a canonical order),
    and the forward gather over them equals the oracle's gradient w.r.t. X."""
    p = random_gather_problem(41, 30000, 1200, 1700, 24, "zipf", "normal", weighted, 0.1)
    X, col, w, row = p["X"], p["col"], p["weight"], p["index"]
    n = row.size
    sc, rt, cf = geot.transpose_edges(up(col), up(w), up(row), 1700, 1200, op)
    sc, rt, cf = sc.cpu().numpy(), rt.cpu().numpy(), cf.cpu().numpy()
    assert np.all(np.diff(sc) >= 0)
    coef = w.copy() if w is not None else np.ones(n, dtype=np.float32)
    if op == "mean":
        deg = np.bincount(row, minlength=1200).astype(np.float32)
        coef = (coef / deg[row]).astype(np.float32)   # one fp32 division, as the library
    want = np.lexsort((coef.view(np.uint32), row, col))
    got = np.lexsort((cf.view(np.uint32), rt, sc))
    assert np.array_equal(sc[got], col[want]) and np.array_equal(rt[got], row[want])
    assert np.array_equal(cf[got].view(np.uint32), coef[want].view(np.uint32))
    g = np.random.default_rng(42).standard_normal((1200, 24)).astype(np.float32)
    gx = geot.gather_scatter(up(g), up(rt), up(cf), up(sc), 1700, "sum").cpu().numpy()
    rx, _ = oracle.gather_scatter_backward(X, col, w, row, g, op)
    tx, _ = oracle.gather_scatter_backward(X, col, w, row, g, op, absolute=True)
    within(gx, rx, tx, f"transposed gather grad_X {op} weighted={weighted}")


def same_triples(sc, rt, cf, col, row, coef):
    """The transposed list holds exactly the (column, row, coefficient) triples of the edges,
    sorted by column (the order inside a column is free: both sides in a canonical order)."""
    assert np.all(np.diff(sc) >= 0)
    want = np.lexsort((coef.view(np.uint32), row, col))
    got = np.lexsort((cf.view(np.uint32), rt, sc))
    assert np.array_equal(sc[got], col[want]) and np.array_equal(rt[got], row[want])
    assert np.array_equal(cf[got].view(np.uint32), coef[want].view(np.uint32))


def mean_coef(w, row, R):
    deg = np.bincount(row, minlength=R).astype(np.float32)
    return (w / deg[row]).astype(np.float32)   # one fp32 division, as the library


@pytest.mark.parametrize("nx,hub", [(300_000, False), (5_000_000, False), (300_000, True), (200, False),
                                    (1 << 23, False), (100, False), (1, False)])
def test_transpose_edges_radix(nx, hub):
    """Inputs of over 2^20 edges take the radix partition: bins of columns (586 bins of 512
    columns for 300,000 columns; 2,442 of 2,048 for 5,000,000; 4,096 of 2,048 for 2^23, the
    most columns it takes), grouped by coarse buckets and split into bins in LDS-staged runs,
    then each bin sorted by column in LDS. `hub` sends 40 % of the edges to one column, so its
    bin exceeds what the final pass holds in registers and is walked twice; 200, 100 and 1
    columns give bins of one column, which are copied (with at most 256 bins the grouping
    pass places them directly). Same canonical comparison as above, sum and mean,
    and the gradient w.r.t. X through the library's own transposition against the oracle."""
    n, R, F = 1_300_000, 200_000, 4
    rng = np.random.default_rng(43)
    row = np.sort(rng.integers(0, R, n)).astype(np.int64)
    col = rng.integers(0, nx, n).astype(np.int64)
    if hub:
        col[rng.random(n) < 0.4] = 12345
    w = rng.random(n, dtype=np.float32)
    for op in ("sum", "mean"):
        say(f"radix transpose nx={nx} hub={hub} {op}")
        sc, rt, cf = (t.cpu().numpy() for t in geot.transpose_edges(up(col), up(w), up(row), nx, R, op))
        same_triples(sc, rt, cf, col, row, w if op == "sum" else mean_coef(w, row, R))
    X = rng.standard_normal((nx, F)).astype(np.float32)
    g = rng.standard_normal((R, F)).astype(np.float32)
    for op in ("sum", "mean"):
        gx, _ = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(g), op, need_weight=False)
        rx, _ = oracle.gather_scatter_backward(X, col, w, row, g, op)
        tx, _ = oracle.gather_scatter_backward(X, col, w, row, g, op, absolute=True)
        within(gx.cpu().numpy(), rx, tx, f"radix grad_X nx={nx} hub={hub} {op}")


@pytest.mark.parametrize("it", ["i64", "i32"])
@pytest.mark.parametrize("aligned", [True, False], ids=["aligned", "offset"])
def test_radix_id_loads(it, aligned):
    """The radix passes load 4 int32 or 2 int64 ids (and weights) per lane where col, row and
    the weights are 16-byte aligned, else one at a time: a ragged edge count (1,300,003: the
    last tile and the last counting block end inside a vector), int32 and int64 ids, arrays
    that start at element 0 of their buffers or one element in. The gradients w.r.t. X of sum
    and mean, and of max with w.r.t. the weights (the max pull reads the edge numbers the
    grouping pass records), against the oracle; with int64 ids also geot_transpose_edges."""
    n, R, nx, F = 1_300_003, 150_000, 400_000, 4
    rng = np.random.default_rng(53)
    row = np.sort(rng.integers(0, R, n)).astype(np.int64)
    col = rng.integers(0, nx, n).astype(np.int64)
    col[rng.random(n) < 0.05] = 777    # a column of about 65,000 edges
    w = rng.random(n, dtype=np.float32)
    dt = {"i64": torch.int64, "i32": torch.int32}[it]

    def dev(a, t):
        k = 0 if aligned else 1
        buf = torch.empty(a.size + 1, dtype=t, device=DEV)
        v = buf[k:k + a.size]
        v.copy_(torch.from_numpy(a).to(t))
        assert (v.data_ptr() % 16 == 0) == aligned
        return v

    cd, rd, wd = dev(col, dt), dev(row, dt), dev(w, torch.float32)
    X = rng.standard_normal((nx, F)).astype(np.float32)
    g = rng.standard_normal((R, F)).astype(np.float32)
    for op in ("sum", "mean", "max"):
        say(f"radix id loads {it} aligned={aligned} {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.gather_scatter(X, col, w, row, R, op),
                                       geot.gather_scatter(up(X), cd, wd, rd, R, op), f"{it} aligned={aligned}")
        gx, gw = geot.gather_scatter_backward(up(X), cd, wd, rd, up(g), op, up(out), need_weight=op == "max")
        rx, rw = oracle.gather_scatter_backward(X, col, w, row, g, op, out)
        tx, tw = oracle.gather_scatter_backward(X, col, w, row, g, op, out, absolute=True)
        within(gx.cpu().numpy(), rx, tx, f"radix id loads grad_X {it} aligned={aligned} {op}")
        if op == "max":
            within(gw.cpu().numpy(), rw, tw, f"radix id loads grad_w {it} aligned={aligned}")
        if it == "i64" and op != "max":
            sc, rt, cf = (t.cpu().numpy() for t in geot.transpose_edges(cd, wd, rd, nx, R, op))
            same_triples(sc, rt, cf, col, row, w if op == "sum" else mean_coef(w, row, R))


def test_transpose_edges_sparse_tail():
    """3,000,000 edges over 2^23 columns, 99.9 % of them in the first 2^20 columns: the tail's
    coarse buckets hold a few records each, so a splitting tile there spans more bins than its
    LDS counts take and places each record with an atomic, and most of the tail's bins are
    empty (their column starts still written). Canonical comparison, sum and mean, and the
    gradient w.r.t. X of both (max pulled over the column starts) against the oracle."""
    n, R, nx, F = 3_000_000, 100_000, 1 << 23, 2
    rng = np.random.default_rng(47)
    row = np.sort(rng.integers(0, R, n)).astype(np.int64)
    col = rng.integers(0, 1 << 20, n).astype(np.int64)
    tail = rng.random(n) < 0.001
    col[tail] = rng.integers(1 << 20, nx, int(tail.sum()))
    w = rng.random(n, dtype=np.float32)
    for op in ("sum", "mean"):
        say(f"transpose sparse tail {op}")
        sc, rt, cf = (t.cpu().numpy() for t in geot.transpose_edges(up(col), up(w), up(row), nx, R, op))
        same_triples(sc, rt, cf, col, row, w if op == "sum" else mean_coef(w, row, R))
    X = rng.integers(-3, 4, (nx, F)).astype(np.float32)
    g = rng.standard_normal((R, F)).astype(np.float32)
    for op in ("sum", "mean", "max"):
        say(f"sparse tail grad_X {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.gather_scatter(X, col, w, row, R, "max"),
                                       geot.gather_scatter(up(X), up(col), up(w), up(row), R, "max"), "sparse tail")
        gx, _ = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(g), op,
                                             None if out is None else up(out), need_weight=False)
        rx, _ = oracle.gather_scatter_backward(X, col, w, row, g, op, out)
        tx, _ = oracle.gather_scatter_backward(X, col, w, row, g, op, out, absolute=True)
        within(gx.cpu().numpy(), rx, tx, f"sparse tail grad_X {op}")


def _mix64(x):
    """splitmix64's finaliser on uint64 (wrapping)."""
    x = (x ^ (x >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    x = (x ^ (x >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return x ^ (x >> np.uint64(31))


def test_transpose_edges_spmm_graph_full():
    """The SpMM graph's 61,859,140 edges over 2,449,029 columns (19,134 bins of 128 columns,
    128 per coarse bucket): the sorted columns equal the sorted input columns, and per column
    the wrapping sum of a 64-bit mix of (row, coefficient bits) equals the input's, so every
    column holds exactly its edges' (row, coefficient) pairs."""
    c = make_config("c4_spmm")
    col, w, row, nx, R = c["col"], c["weight"], c["index"], c["X"].shape[0], c["num_segments"]
    del c
    say("transpose spmm graph")
    sc, rt, cf = (t.cpu().numpy() for t in geot.transpose_edges(up(col), up(w), up(row), nx, R, "sum"))
    torch.cuda.empty_cache()
    assert np.array_equal(sc, np.sort(col))
    with np.errstate(over="ignore"):
        def h(r, cbits):
            return _mix64((r.astype(np.uint64) << np.uint64(32)) | cbits.astype(np.uint64))
        starts = np.searchsorted(sc, np.arange(nx))
        nonempty = np.diff(np.append(starts, sc.size)) > 0
        got = np.add.reduceat(h(rt, cf.view(np.uint32)), starts[nonempty])
        order = np.argsort(col, kind="stable")
        want = np.add.reduceat(h(row[order], w[order].view(np.uint32)), starts[nonempty])
    assert np.array_equal(got, want)


def test_gather_backward_max_hub_column_keeps_the_fp32_bound():
    """Max gradient w.r.t. X when one column receives the maximum of most rows: its row of
    grad_X sums about 600,000 positive terms over the transposed list. The pull adds them in
    runs of 256 records, so the fp32 error stays within the bound (one serial chain of that
    many same-signed terms would not)."""
    rng = np.random.default_rng(93)
    R, nx, F, per = 600_000, 5000, 4, 3
    row = np.repeat(np.arange(R), per).astype(np.int64)
    n = row.size
    col = rng.integers(1, nx, n).astype(np.int64)
    col[::per] = 0                                      # every row has one edge to column 0
    X = (rng.random((nx, F), dtype=np.float32) + 0.5).astype(np.float32)
    X[0] = 100.0                                        # ... which attains its maximum
    w = (rng.random(n, dtype=np.float32) + 0.5).astype(np.float32)
    w[::per] = 1.0
    g = (rng.random((R, F), dtype=np.float32) + 0.5).astype(np.float32)
    say("max gradient, hub column")
    out = forward_for_gradient(oracle.gather_scatter(X, col, w, row, R, "max"),
                               geot.gather_scatter(up(X), up(col), up(w), up(row), R, "max"), "hub column")
    gx, _ = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(g), "max", up(out), need_weight=False)
    rx, _ = oracle.gather_scatter_backward(X, col, w, row, g, "max", out)
    ax, _ = oracle.gather_scatter_backward(X, col, w, row, g, "max", out, absolute=True)
    within(gx.cpu().numpy(), rx, ax, "hub column max grad_X")


@pytest.mark.parametrize("n", [30_000, 1_300_000])
def test_transpose_mean_with_rows_out_of_range(n):
    """Row ids outside [0, num_rows) break the precondition: their values are unspecified,
    but the mean coefficient must not read row starts out of bounds (the edges' rows are
    checked before the division). The edges with rows in range still carry weight / the
    in-range edge count of their row. Direct placement (30,000 edges) and buckets (1.3 M)."""
    R, nx = 5000, 40_000
    rng = np.random.default_rng(44)
    row = np.sort(rng.integers(-50, R + 50, n)).astype(np.int64)
    col = rng.integers(0, nx, n).astype(np.int64)
    w = rng.random(n, dtype=np.float32)
    say(f"transpose mean, rows out of range, n={n}")
    sc, rt, cf = (t.cpu().numpy() for t in geot.transpose_edges(up(col), up(w), up(row), nx, R, "mean"))
    assert np.array_equal(sc, np.sort(col))
    ok = (row >= 0) & (row < R)
    deg = np.bincount(row[ok], minlength=R).astype(np.float32)
    coef = (w[ok] / deg[row[ok]]).astype(np.float32)
    keep = (rt >= 0) & (rt < R)
    want = np.lexsort((coef.view(np.uint32), row[ok], col[ok]))
    got = np.lexsort((cf[keep].view(np.uint32), rt[keep], sc[keep]))
    assert np.array_equal(rt[keep][got], row[ok][want]) and np.array_equal(sc[keep][got], col[ok][want])
    assert np.array_equal(cf[keep][got].view(np.uint32), coef[want].view(np.uint32))


@pytest.mark.parametrize("itype", [torch.int64, torch.int32])
def test_offsets_pass_unaligned_index(itype):
    """An index view one element into its buffer (not 16-byte aligned) takes the per-row offsets
    pass: mean gradients and the index statistics equal the aligned call's and the oracle's."""
    p = random_problem(21, 300_000, 9000, 8, "zipf", "normal", 0.2)
    idx = p["index"]
    buf = torch.empty(idx.size + 1, dtype=itype, device=DEV)
    view = buf[1:]
    view.copy_(torch.from_numpy(idx).to(itype))
    assert view.data_ptr() % 16 != 0
    g = np.random.default_rng(22).standard_normal((9000, 8)).astype(np.float32)
    got = geot.segment_reduce_backward(up(g), view, "mean").cpu().numpy()
    aligned = geot.segment_reduce_backward(up(g), torch.from_numpy(idx).to(itype).to(DEV), "mean").cpu().numpy()
    assert np.array_equal(got, aligned)
    ref = oracle.segment_reduce_backward(g, idx, "mean")
    within(got, ref, np.abs(ref.astype(np.float64)), "unaligned index mean")
    if itype == torch.int64:
        st, ref_st = geot.index_stats(view, 9000), oracle.index_stats(idx, 9000)
        assert st["max_len"] == ref_st["max_len"] and st["num_empty"] == ref_st["num_empty"]


@pytest.mark.parametrize("weighted", [True, False])
def test_gather_backward_max_radix(weighted):
    """Max gradient w.r.t. X pulled over a transposed list from the radix partition with edge
    numbers (16-byte records; 2,000,000 edges): each X row sums its column's records whose
    edge is the recipient; integer values, so ties are frequent and the lowest-edge rule
    decides. Both gradients against the oracle's."""
    q = random_gather_problem(23, 2_000_000, 50_000, 60_000, 8, "zipf", "int", weighted, 0.05)
    X, col, w, row = q["X"], q["col"], q["weight"], q["index"]
    g = np.random.default_rng(24).standard_normal((50_000, 8)).astype(np.float32)
    out = forward_for_gradient(oracle.gather_scatter(X, col, w, row, 50_000, "max"),
                               geot.gather_scatter(up(X), up(col), up(w), up(row), 50_000, "max"), "radix")
    gx, gw = geot.gather_scatter_backward(up(X), up(col), up(w), up(row), up(g), "max", up(out))
    rx, rw = oracle.gather_scatter_backward(X, col, w, row, g, "max", out)
    ax, aw = oracle.gather_scatter_backward(X, col, w, row, g, "max", out, absolute=True)
    within(gx.cpu().numpy(), rx, ax, f"radix max grad_X weighted={weighted}")
    if weighted:
        within(gw.cpu().numpy(), rw, aw, "radix max grad_w")
