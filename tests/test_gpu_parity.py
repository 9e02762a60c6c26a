"""GPU parity: libgeot_hip (through its C-ABI) against the CPU oracle, element by element.

Covers every kernel family and tiling choice on exhaustive tiny inputs, random
inputs with several length distributions and feature widths (odd F, F that is
not a multiple of the vector width, F above one column tile), multi-level
partial combining (forced small row runs), the fused gather form, exact
arithmetic (bit-exact sums), determinism, edge cases, index statistics and the
precondition check.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import compare, oracle_gather, oracle_segment, say
from workloads import random_gather_problem, random_problem

pytestmark = pytest.mark.gpu
OPS = ("sum", "mean", "max")
DEV = "cuda:0"


def up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_sr(src, idx, S, op, choice=None):
    out = geot.segment_reduce(up(src), up(idx), S, op, choice=choice)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def run_gs(X, col, w, row, R, op, choice=None):
    out = geot.gather_scatter(up(X), up(col), up(w), up(row), R, op, choice=choice)
    torch.cuda.synchronize()
    return out.cpu().numpy()


TINY_CHOICES = [
    None,
    dict(family="ep", rows=1),
    dict(family="ep", lanes=64, rows=1),           # 4 rows per block: partials cross blocks
    dict(family="ep", lanes=64, vec=1, rows=2),
    dict(family="ep", lanes=1, rows=3),
    dict(family="sp", groups=1),
    dict(family="sp", lanes=4, groups=16),
]


@pytest.mark.parametrize("F", [1, 3, 4, 5, 7, 8])
def test_tiny_exhaustive_bit_exact(F):
    """Every non-decreasing index with nnz <= 5 over S <= 4 segments, integer values:
    every partial sum is exact, so sum and max must be bit-exact for every kernel choice."""
    rng = np.random.default_rng(100 + F)
    for S in range(1, 5):
        for nnz in range(1, 6):
            for idx_t in itertools.combinations_with_replacement(range(S), nnz):
                idx = np.array(idx_t, dtype=np.int64)
                src = rng.integers(-8, 9, size=(nnz, F)).astype(np.float32)
                refs = {op: oracle_segment(src, idx, S, op) for op in OPS}
                for ci, ch in enumerate(TINY_CHOICES):
                    for op in OPS:
                        got = run_sr(src, idx, S, op, ch)
                        ref, terms = refs[op]
                        if op == "mean":
                            compare(got, ref, op, terms, f"tiny F={F} idx={idx_t} choice={ch}")
                        else:
                            assert np.array_equal(got, ref), \
                                f"tiny {op} F={F} idx={idx_t} choice={ch}: {got} vs {ref}"


RANDOM_CASES = [
    # seed, nnz, S, F, dist, values, empty_frac
    (1, 30000, 2000, 32, "zipf", "uniform", 0.05),
    (2, 25000, 400, 1, "lognormal", "normal", 0.1),
    (3, 20000, 3000, 3, "uniform", "normal", 0.2),
    (4, 40000, 50, 64, "one_heavy", "normal", 0.3),
    (5, 15000, 1500, 15, "poisson", "uniform", 0.0),
    (6, 12000, 700, 17, "zipf", "normal", 0.1),
    (7, 10000, 600, 128, "lognormal", "uniform", 0.05),
    (8, 6000, 300, 255, "uniform", "normal", 0.1),
    (9, 5000, 200, 256, "zipf", "normal", 0.0),
    (10, 4000, 300, 300, "uniform", "normal", 0.1),
    (11, 20000, 20000, 8, "uniform", "normal", 0.6),
    (12, 30000, 1, 16, "fixed", "normal", 0.0),
    (13, 9000, 9000, 2, "fixed", "negative", 0.0),
]

RANDOM_CHOICES = [
    None,
    dict(family="ep", rows=1),
    dict(family="ep", lanes=64, rows=1),
    dict(family="ep", lanes=2, vec=1, rows=7),
    dict(family="ep", rows=33),
    dict(family="ep", lanes=4, rows=9, flags=4),   # 16-column tiles, one tile after another
    dict(family="sp"),
    dict(family="sp", lanes=16, groups=2),
]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=lambda c: f"seed{c[0]}-F{c[3]}-{c[4]}")
def test_random_parity_all_choices(case):
    seed, nnz, S, F, dist, values, ef = case
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    src, idx = p["src"], p["index"]
    for op in OPS:
        ref, terms = oracle_segment(src, idx, S, op)
        for ch in RANDOM_CHOICES:
            say(f"segment_reduce seed={seed} F={F} op={op} choice={ch}")
            got = run_sr(src, idx, S, op, ch)
            compare(got, ref, op, terms, f"seed={seed} F={F} op={op} choice={ch}")


GATHER_CASES = [
    # seed, nnz, R, n_x, F, dist, values, weighted, empty_frac
    (21, 30000, 2000, 1500, 32, "zipf", "normal", True, 0.05),
    (22, 20000, 500, 3000, 1, "lognormal", "normal", True, 0.1),
    (23, 15000, 1000, 800, 3, "uniform", "uniform", False, 0.1),
    (24, 10000, 300, 5000, 128, "one_heavy", "normal", True, 0.2),
    (25, 8000, 900, 900, 17, "poisson", "normal", False, 0.0),
    (26, 6000, 400, 700, 256, "zipf", "normal", True, 0.0),
]


@pytest.mark.parametrize("case", GATHER_CASES, ids=lambda c: f"seed{c[0]}-F{c[4]}-w{int(c[7])}")
def test_gather_parity_all_choices(case):
    seed, nnz, R, nx, F, dist, values, weighted, ef = case
    p = random_gather_problem(seed, nnz, R, nx, F, dist, values, weighted, ef)
    X, col, w, row = p["X"], p["col"], p["weight"], p["index"]
    for op in OPS:
        ref, terms = oracle_gather(X, col, w, row, R, op)
        for ch in RANDOM_CHOICES:
            say(f"gather_scatter seed={seed} F={F} op={op} choice={ch}")
            got = run_gs(X, col, w, row, R, op, ch)
            compare(got, ref, op, terms, f"gather seed={seed} F={F} op={op} choice={ch}")


def _special_values(rng, shape, nan_frac):
    """Values from {+0, -0, +-1, +-2, +-inf} with a fraction of NaNs: ties, zeros of both
    signs and infinities are frequent, so the max's NaN and signed-zero rules decide."""
    pool = np.array([0.0, -0.0, 1.0, -1.0, 2.0, -2.0, np.inf, -np.inf, -0.0, 0.0], dtype=np.float32)
    v = pool[rng.integers(0, pool.size, shape)]
    v[rng.random(shape) < nan_frac] = np.nan
    return v


@pytest.mark.parametrize("F", [1, 3, 16, 33])
def test_max_nan_and_signed_zeros_bitwise(F):
    """Max is IEEE 754-2019 maximum on both sides (NaN propagates, +0 above -0): the GPU
    result has the oracle's bit pattern (or NaN where the oracle's is NaN) for every kernel
    choice, in the segment and the fused form, with fp32 and bf16 storage; the max gradient
    (recipient: the first member == the maximum) matches the oracle exactly."""
    rng = np.random.default_rng(500 + F)
    p = random_problem(501 + F, 6000, 700, F, "zipf", "normal", 0.1)
    idx, S = p["index"], 700
    for nan_frac in (0.0, 0.002):
        src = _special_values(rng, (idx.size, F), nan_frac)
        ref = oracle.segment_reduce(src, idx, S, "max")
        for ch in RANDOM_CHOICES:
            say(f"max specials F={F} nan={nan_frac} choice={ch}")
            compare(run_sr(src, idx, S, "max", ch), ref, "max", None, f"specials F={F} choice={ch}")
        t16 = torch.from_numpy(src).to(torch.bfloat16)   # +-0, +-inf, NaN and small integers are exact
        got = geot.segment_reduce(t16.to(DEV), up(idx).to(torch.int32), S, "max").cpu().numpy()
        compare(got, ref, "max", None, f"specials bf16 F={F}")
        q = random_gather_problem(502 + F, 5000, 400, 300, F, "lognormal", "normal", True, 0.1)
        X = _special_values(rng, (300, F), nan_frac)
        w = np.where(rng.random(q["col"].size) < 0.5, -1.0, 2.0).astype(np.float32)
        gref = oracle.gather_scatter(X, q["col"], w, q["index"], 400, "max")
        for ch in RANDOM_CHOICES:
            compare(run_gs(X, q["col"], w, q["index"], 400, "max", ch), gref, "max", None,
                    f"fused specials F={F} choice={ch}")
    src = _special_values(rng, (idx.size, F), 0.0)
    out = oracle.segment_reduce(src, idx, S, "max")
    g = rng.standard_normal((S, F)).astype(np.float32)
    got = geot.segment_reduce_backward(up(g), up(idx), "max", up(src), up(out)).cpu().numpy()
    assert np.array_equal(got, oracle.segment_reduce_backward(g, idx, "max", src, out)), f"max gradient F={F}"


RAGGED_F = [3, 5, 6, 7, 13, 15, 17, 31, 33, 63, 65, 127, 129, 255, 257, 301, 513]
RAGGED_CHOICES = [
    None,                                               # 4-float vectors (3 for F = 3) by default
    dict(family="ep", vec=4, rows=1),                   # many blocks: partial levels
    dict(family="ep", vec=4, lanes=2, rows=5),          # several column tiles, the last one ragged
    dict(family="ep", vec=4, lanes=2, rows=3, flags=4),  # the same tiles one after another
    dict(family="ep", vec=1, rows=7),                   # exact 1-float vectors, for comparison
]


@pytest.mark.parametrize("F", RAGGED_F)
def test_ragged_rows_all_choices(F):
    """Widths that are no multiple of 4: fp32 rows move in 4-float vectors at 4-byte aligned
    addresses, the vector that would cross a row's end overlapping its neighbour (3-float
    vectors for F = 3). Segment and fused forms, every op, every choice, against the oracle;
    and the default choice bit-identical to exact 1-float vectors for max and to the oracle
    for sum and mean."""
    p = random_problem(600 + F, 9000, 700, F, "zipf", "normal", 0.1)
    src, idx = p["src"], p["index"]
    q = random_gather_problem(601 + F, 7000, 500, 400, F, "lognormal", "normal", True, 0.1)
    for op in OPS:
        ref, terms = oracle_segment(src, idx, 700, op)
        gref, gterms = oracle_gather(q["X"], q["col"], q["weight"], q["index"], 500, op)
        for ch in RAGGED_CHOICES:
            say(f"ragged F={F} {op} choice={ch}")
            compare(run_sr(src, idx, 700, op, ch), ref, op, terms, f"ragged F={F} {op} {ch}")
            compare(run_gs(q["X"], q["col"], q["weight"], q["index"], 500, op, ch), gref, op, gterms,
                    f"ragged gather F={F} {op} {ch}")
    c = geot.select(9000, 700, F, "sum")
    assert c["vec"] == (3 if F == 3 else 4), c
    # a view that starts 4 bytes into its buffer: rows stay 4-byte aligned only
    buf = torch.empty(src.size + 1, dtype=torch.float32, device=DEV)
    view = buf[1:].view(src.shape)
    view.copy_(up(src))
    got = geot.segment_reduce(view, up(idx), 700, "max").cpu().numpy()
    compare(got, oracle.segment_reduce(src, idx, 700, "max"), "max", None, f"ragged F={F} offset view")


SMALL_CALL_CASES = [
    # seed, nnz, S, F, dist, values, empty_frac: small inputs (one or two partial levels)
    (41, 65536, 4096, 32, "zipf", "normal", 0.05),
    (42, 20000, 19000, 4, "uniform", "normal", 0.6),    # long runs of empty segments, few rows
    (43, 50000, 1500, 300, "zipf", "normal", 0.5),      # two column tiles
    (44, 3000, 3000, 3, "one_heavy", "normal", 0.3),
    (45, 200000, 100, 1, "lognormal", "normal", 0.2),
    (46, 7, 5, 6, "uniform", "normal", 0.0),            # one block
]


def _runs_problem(seed, nnz, S, F, nseg):
    """nnz rows in `nseg` segments spread over S: runs of about S / nseg empty segments
    between them (the empty-run list gets records), and leading and trailing runs."""
    rng = np.random.default_rng(seed)
    ids = np.sort(rng.choice(np.arange(40, S - 40), size=nseg, replace=False))
    cuts = np.sort(rng.choice(np.arange(1, nnz), size=nseg - 1, replace=False))
    lengths = np.diff(np.concatenate([[0], cuts, [nnz]]))
    index = np.repeat(ids, lengths).astype(np.int64)
    return dict(src=rng.standard_normal((nnz, F)).astype(np.float32), index=index)


@pytest.mark.parametrize("case", SMALL_CALL_CASES + [(47, 20000, 16000, 4, "runs", None, 10),
                                                     (48, 9000, 1700, 300, "runs", None, 7)],
                         ids=lambda c: f"seed{c[0]}-F{c[3]}-{c[4]}")
def test_small_calls_repeat_and_replay(case):
    """Small inputs: calls repeated on one stream (five times), through a caller workspace
    and captured in a HIP graph (replayed with new inputs) all match the oracle; the list
    of empty-segment runs empties itself after every call. The "runs" cases have long runs
    of empty segments, which go through that list."""
    seed, nnz, S, F, dist, values, ef = case
    if dist == "runs":
        p = _runs_problem(seed, nnz, S, F, ef)
    else:
        p = random_problem(seed, nnz, S, F, dist, values, ef)
    src, idx = up(p["src"]), up(p["index"])
    for op in OPS:
        ref, terms = oracle_segment(p["src"], p["index"], S, op)
        for k in range(5):
            compare(geot.segment_reduce(src, idx, S, op).cpu().numpy(), ref, op, terms, f"small {op} call {k}")
        ws = torch.empty(geot.workspace_size(nnz, S, F, op), dtype=torch.uint8, device=DEV)
        compare(geot.segment_reduce_ws(src, idx, S, op, ws).cpu().numpy(), ref, op, terms, f"small {op} ws")
    st = torch.cuda.Stream()
    out = torch.empty((S, F), device=DEV)
    with torch.cuda.stream(st):
        geot.segment_reduce(src, idx, S, "sum", out=out)
    st.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=st):
        geot.segment_reduce(src, idx, S, "sum", out=out)
    rng = np.random.default_rng(seed)
    for k in range(3):
        v = rng.standard_normal(p["src"].shape).astype(np.float32)
        src.copy_(torch.from_numpy(v))
        out.fill_(9.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        ref, terms = oracle_segment(v, p["index"], S, "sum")
        compare(out.cpu().numpy(), ref, "sum", terms, f"small replay {k}")


def test_fusion_identity_on_gpu():
    """gather_scatter(X, col, w, row) equals segment_reduce(w * X[col], row) (Section IV):
    bit-exact for max, within the bound for sum and mean."""
    p = random_gather_problem(31, 50000, 3000, 4000, 24, "lognormal", "normal", True, 0.05)
    X, col, w, row, R = p["X"], p["col"], p["weight"], p["index"], p["num_segments"]
    msgs = (w[:, None] * X[col]).astype(np.float32)
    for op in OPS:
        a = run_gs(X, col, w, row, R, op)
        b = run_sr(msgs, row, R, op)
        _, terms = oracle_segment(msgs, row, R, op)
        compare(a, b, op, None if op == "max" else 2 * terms, f"fusion identity {op}")


def test_exact_arithmetic_at_scale_is_bit_exact():
    """Values in {-1, 0, 1}: every partial sum is an integer below 2^24, so sums are
    exact in any order and the GPU must match the oracle bit for bit, long segments included."""
    p = random_problem(41, 3_000_000, 5000, 16, "one_heavy", "ternary", 0.1)
    src, idx, S = p["src"], p["index"], p["num_segments"]
    ref = oracle.segment_reduce(src, idx, S, "sum")
    for ch in (None, dict(family="ep", rows=1), dict(family="ep", lanes=64, rows=4), dict(family="sp")):
        say(f"exact arithmetic choice={ch}")
        got = run_sr(src, idx, S, "sum", ch)
        assert np.array_equal(got, ref), f"exact sum choice={ch}"


def test_results_are_deterministic():
    """No atomics on the reduction path: repeated calls give identical bits for every op."""
    p = random_problem(42, 400000, 3000, 32, "lognormal", "normal", 0.05)
    s, i = up(p["src"]), up(p["index"])
    for op in OPS:
        outs = [geot.segment_reduce(s, i, 3000, op).cpu().numpy() for _ in range(3)]
        assert all(np.array_equal(outs[0], o) for o in outs[1:]), op


def test_empty_and_degenerate_inputs():
    F = 5
    # nnz == 0: every segment is empty
    out = geot.segment_reduce(torch.empty((0, F), device=DEV), torch.empty(0, dtype=torch.int64, device=DEV),
                              7, "max")
    assert torch.all(out == 0)
    # S == 0: no-op returning an empty tensor
    out = geot.segment_reduce(torch.ones((3, F), device=DEV), torch.zeros(3, dtype=torch.int64, device=DEV),
                              0, "sum")
    assert out.shape == (0, F)
    # nnz == 1 with leading and trailing empties; a non-empty all-negative max is not clipped at 0
    src = np.full((1, F), -3.5, dtype=np.float32)
    for op in OPS:
        got = run_sr(src, np.array([2], dtype=np.int64), 5, op)
        want = np.zeros((5, F), dtype=np.float32)
        want[2] = -3.5
        assert np.array_equal(got, want), op
    # every row in the last segment of many
    src = np.arange(4000 * 3, dtype=np.float32).reshape(4000, 3) / 7
    idx = np.full(4000, 999, dtype=np.int64)
    for op in OPS:
        ref, terms = oracle_segment(src, idx, 1000, op)
        compare(run_sr(src, idx, 1000, op), ref, op, terms, f"all-in-last {op}")


def test_misaligned_views_use_narrower_vectors():
    """Views with a storage offset break 16-byte alignment; results must not change."""
    p = random_problem(43, 20000, 500, 8, "zipf", "normal", 0.1)
    big = torch.zeros(20000 * 8 + 1, device=DEV)
    big[1:] = up(p["src"]).reshape(-1)
    view = big[1:].view(20000, 8)
    idx = up(p["index"])
    for op in OPS:
        got = geot.segment_reduce(view, idx, 500, op).cpu().numpy()
        assert geot.last_choice()["vec"] == 1
        ref, terms = oracle_segment(p["src"], p["index"], 500, op)
        compare(got, ref, op, terms, f"misaligned {op}")


def test_out_is_overwritten_not_accumulated():
    p = random_problem(44, 5000, 300, 4, "uniform", "normal", 0.2)
    out = torch.full((300, 4), 123.0, device=DEV)
    geot.segment_reduce(up(p["src"]), up(p["index"]), 300, "sum", out=out)
    ref, terms = oracle_segment(p["src"], p["index"], 300, "sum")
    compare(out.cpu().numpy(), ref, "sum", terms, "overwrite")


def test_index_stats_match_oracle():
    for seed, dist, ef in ((51, "zipf", 0.1), (52, "fixed", 0.0), (53, "one_heavy", 0.5)):
        p = random_problem(seed, 200000, 7000, 1, dist, "uniform", ef)
        got = geot.index_stats(up(p["index"]), 7000)
        want = oracle.index_stats(p["index"], 7000)
        for k in ("max_len", "num_empty", "sum_len_sq"):
            assert got[k] == want[k], k
        assert got["nnz"] == 200000 and got["num_segments"] == 7000
        assert abs(got["mean_len"] - want["mean_len"]) <= 1e-12 * want["mean_len"]
        assert abs(got["var_len"] - want["var_len"]) <= 1e-9 * max(1.0, want["var_len"])


def test_check_index_reports_violations():
    idx = up(np.array([0, 0, 1, 3, 3], dtype=np.int64))
    assert geot.check_index(idx, 4) == 0
    assert geot.check_index(idx, 3) == 3
    assert geot.check_index(up(np.array([0, 2, 1, 3], dtype=np.int64)), 4) == 2
    assert geot.check_index(idx, 4, col=up(np.array([0, 1, 2, 3, 9], dtype=np.int64)), num_x_rows=5) == 3
    assert geot.check_index(idx, 4, col=up(np.array([0, 1, 2, 3, 4], dtype=np.int64)), num_x_rows=5) == 0


def test_profile_hooks_record_main_kernel_time():
    p = random_problem(54, 200000, 5000, 32, "lognormal", "normal", 0.0)
    s, i = up(p["src"]), up(p["index"])
    geot.profile_begin(8)
    for _ in range(3):
        geot.segment_reduce(s, i, 5000, "sum")
    ms = geot.profile_end()
    assert len(ms) == 3 and all(0.0 < t < 1000.0 for t in ms)


def test_two_streams_and_scratch_release():
    """Calls on two streams in flight use separate cached buffers; releasing them and
    calling again gives the same results."""
    p = random_problem(55, 300000, 2000, 32, "lognormal", "normal", 0.05)
    q = random_problem(56, 200000, 1500, 32, "zipf", "normal", 0.05)
    sp, ip = up(p["src"]), up(p["index"])
    sq, iq = up(q["src"]), up(q["index"])
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    outs = []
    for _ in range(3):
        with torch.cuda.stream(s1):
            a = geot.segment_reduce(sp, ip, 2000, "sum")
        with torch.cuda.stream(s2):
            b = geot.segment_reduce(sq, iq, 1500, "max")
        outs.append((a, b))
    torch.cuda.synchronize()
    ref_a, terms_a = oracle_segment(p["src"], p["index"], 2000, "sum")
    ref_b, _ = oracle_segment(q["src"], q["index"], 1500, "max")
    for a, b in outs:
        compare(a.cpu().numpy(), ref_a, "sum", terms_a, "stream 1")
        compare(b.cpu().numpy(), ref_b, "max", None, "stream 2")
    geot.release_scratch()
    a = geot.segment_reduce(sp, ip, 2000, "sum").cpu().numpy()
    assert np.array_equal(a, outs[0][0].cpu().numpy())


@pytest.mark.parametrize("lanes", [1, 2, 4, 8, 16, 32, 64])
def test_scan_every_lane_width_exact(lanes):
    """One row per row group and very short segments: every lane of every wave sits next to
    a segment boundary, so the segmented scan (DPP row shifts and broadcasts for narrow
    groups, lane shuffles for wide ones), the cross-wave LDS step and the partial levels
    are all exercised. Integer values make sums exact: results must be bit-identical."""
    rng = np.random.default_rng(200 + lanes)
    for trial in range(3):
        L = rng.integers(0, 4, size=6000)            # lengths 0..3: empties everywhere
        idx = np.repeat(np.arange(L.size, dtype=np.int64), L)
        F = 4 * lanes if trial == 0 else lanes      # vec 4, then vec 1 (F = lanes)
        src = rng.integers(-8, 9, size=(idx.size, F)).astype(np.float32)
        for op in ("sum", "max"):
            ref = oracle.segment_reduce(src, idx, L.size, op)
            for rows in (1, 2, 5):
                ch = dict(family="ep", lanes=lanes, rows=rows)
                got = run_sr(src, idx, L.size, op, ch)
                assert np.array_equal(got, ref), f"lanes={lanes} F={F} rows={rows} {op}"


def test_long_runs_of_empty_segments():
    """Outputs that are mostly empty: long leading, interior and trailing runs of empty
    segments (filled by whole blocks), and blocks with more long runs than their queue
    holds (the rest filled by the row group)."""
    rng = np.random.default_rng(57)
    cases = []
    # few rows over many segments, one huge trailing run
    cases.append((np.sort(rng.integers(1000, 5000, 3000)).astype(np.int64), 400000, 8))
    # rows spaced ~40 segments apart: every boundary is a long run
    cases.append((np.cumsum(rng.integers(33, 48, 20000)).astype(np.int64), 1000000, 4))
    # one row in the middle of a million segments
    cases.append((np.array([500000], dtype=np.int64), 1000000, 32))
    for idx, S, F in cases:
        src = rng.standard_normal((idx.size, F)).astype(np.float32)
        for op in ("sum", "max"):
            ref, terms = oracle_segment(src, idx, S, op)
            for ch in (None, dict(family="ep", lanes=1, rows=1), dict(family="ep", rows=1),
                       dict(family="ep", rows=64), dict(family="sp")):
                say(f"gaps S={S} nnz={idx.size} F={F} op={op} choice={ch}")
                got = run_sr(src, idx, S, op, ch)
                compare(got, ref, op, terms, f"gaps S={S} F={F} {op} {ch}")


@pytest.mark.parametrize("F", [32, 33, 64, 100, 128, 256, 300])
def test_non_temporal_row_loads_match_ordinary_loads(F):
    """The two load policies read the same values and reduce them in the same order:
    outputs are bitwise identical, and both match the oracle."""
    p = random_problem(900 + F, 40000, 700, F, "lognormal", "normal", 0.1)
    s, i = up(p["src"]), up(p["index"])
    for op in OPS:
        ref, terms = oracle_segment(p["src"], p["index"], 700, op)
        for base in (dict(family="ep"), dict(family="ep", rows=3), dict(family="ep", lanes=64, vec=1, rows=2)):
            say(f"load policies F={F} {op} {base}")
            cached = geot.segment_reduce(s, i, 700, op, choice=dict(base, flags=2))
            assert geot.last_choice()["flags"] == 0
            try:
                nt = geot.segment_reduce(s, i, 700, op, choice=dict(base, flags=1))
            except geot.GeotError as e:   # the tile of this shape is narrower than 128 bytes
                assert e.status == 5, e
                continue
            assert geot.last_choice()["flags"] == 1
            assert torch.equal(nt, cached), f"F={F} {op} {base}"
            compare(nt.cpu().numpy(), ref, op, terms, f"non-temporal F={F} {op} {base}")
    # 16-bit storage: 64 bf16 columns are 128 bytes
    t = torch.from_numpy(p["src"][:, :64].copy()).to(torch.bfloat16)
    s16 = t.to(DEV)
    a = geot.segment_reduce(s16, i, 700, "sum", choice=dict(family="ep", flags=1)) if F >= 64 else None
    if a is not None:
        b = geot.segment_reduce(s16, i, 700, "sum", choice=dict(family="ep", flags=2))
        assert torch.equal(a, b)


@pytest.mark.parametrize("F", [33, 64, 128, 256, 300])
def test_tile_major_order_matches_adjacent_tiles(F):
    """Tile-major block order changes which blocks run together, not what a block reduces:
    outputs are bitwise identical to the adjacent order, for the gather and rows modes, with
    several partial levels (small row runs) and long runs of empty segments."""
    R, nx = 3000, 2500
    p = random_gather_problem(950 + F, 30000, R, nx, F, "zipf", "normal", True, 0.3)
    X, col, w, row = up(p["X"]), up(p["col"]), up(p["weight"]), up(p["index"])
    q = random_problem(960 + F, 30000, 5000, F, "lognormal", "normal", 0.4)
    s, i = up(q["src"]), up(q["index"])
    for op in OPS:
        gref, gterms = oracle_gather(p["X"], p["col"], p["weight"], p["index"], R, op)
        sref, sterms = oracle_segment(q["src"], q["index"], 5000, op)
        for base in (dict(family="ep", lanes=16, rows=64), dict(family="ep", lanes=8, rows=3),
                     dict(family="ep", lanes=2, vec=2, rows=17)):
            say(f"tile-major F={F} {op} {base}")
            a = geot.gather_scatter(X, col, w, row, R, op, choice=base)
            b = geot.gather_scatter(X, col, w, row, R, op, choice=dict(base, flags=4))
            tiled = geot.last_choice()["flags"] & 4
            # fp32 rows of 4 floats or more take 4-float vectors whatever F (the last one
            # overlapping); an explicit vec 2 needs an even F
            V = 4 if base.get("vec", 4) == 4 and F >= 4 else (2 if F % 2 == 0 else 1)
            assert bool(tiled) == (F > base["lanes"] * V), geot.last_choice()   # reported when tiles > 1
            assert torch.equal(a, b), f"gather F={F} {op} {base}"
            compare(b.cpu().numpy(), gref, op, gterms, f"tile-major gather F={F} {op} {base}")
            a = geot.segment_reduce(s, i, 5000, op, choice=base)
            b = geot.segment_reduce(s, i, 5000, op, choice=dict(base, flags=4))
            assert torch.equal(a, b), f"rows F={F} {op} {base}"
            compare(b.cpu().numpy(), sref, op, sterms, f"tile-major rows F={F} {op} {base}")
    # 16-bit X with int32 ids: 8-wide loads, tiles of 8 * lanes columns
    Xb = up(p["X"]).to(torch.bfloat16)
    c32, r32 = col.to(torch.int32), row.to(torch.int32)
    base = dict(family="ep", lanes=4, vec=8, rows=32)
    if F % 8 == 0:
        a = geot.gather_scatter(Xb, c32, w, r32, R, "sum", choice=base)
        b = geot.gather_scatter(Xb, c32, w, r32, R, "sum", choice=dict(base, flags=4))
        assert geot.last_choice()["flags"] & 4
        assert torch.equal(a, b), f"bf16 gather F={F}"


def test_selection_with_index_statistics():
    """With the index's length statistics the selector also sees the spread of the lengths:
    short, even segments take the segment-parallel family, a heavy tail keeps the element-
    parallel one; either way every op matches the oracle. A Graph keeps its ids' statistics
    for its gathers."""
    even = random_problem(700, 400_000, 20_000, 15, "poisson", "normal", 0.0)
    heavy = random_problem(701, 400_000, 20_000, 15, "one_heavy", "normal", 0.1)
    for name, p, fam in (("even", even, 2), ("heavy", heavy, 1)):
        s, i = up(p["src"]), up(p["index"])
        st = geot.index_stats(i, 20_000)
        for op in OPS:
            say(f"statistics {name} {op}")
            got = geot.segment_reduce(s, i, 20_000, op, stats=st)
            assert geot.last_choice()["family"] == fam, (name, geot.last_choice())
            ref, terms = oracle_segment(p["src"], p["index"], 20_000, op)
            compare(got.cpu().numpy(), ref, op, terms, f"statistics {name} {op}")
    from paper_2404_03019_amd.autograd import Graph, gather_scatter
    q = random_gather_problem(702, 300_000, 15_000, 9_000, 15, "poisson", "normal", True, 0.0)
    graph = Graph(up(q["col"]), up(q["index"]), 15_000, up(q["weight"]), num_src=9_000)
    got = gather_scatter(up(q["X"]), graph.col, graph.weight, graph.row, 15_000, "sum", graph)
    assert graph.stats()["max_len"] == int(q["lengths"].max())
    ref, terms = oracle_gather(q["X"], q["col"], q["weight"], q["index"], 15_000, "sum")
    compare(got.detach().cpu().numpy(), ref, "sum", terms, "graph gather with statistics")


@pytest.mark.parametrize("choice", [dict(family="sp", groups=1), dict(family="sp", groups=4),
                                    dict(family="ep", rows=4096)],
                         ids=["sp-groups1", "sp-groups4", "ep-rows4096"])
def test_long_segments_of_one_sign_keep_the_fp32_bound(choice):
    """Segments of 700,000 positive terms: one group's serial fp32 chain over such a segment
    would be off by about 3e-5 of the absolute sum; the segment-parallel kernel adds its rows
    in runs of 256 (and the element-parallel one in row runs of at most 4,096 rows), so sum
    and mean stay within 1e-5 * sum|terms| + 1e-6, rows mode and gather mode."""
    rng = np.random.default_rng(91)
    S, F, n = 3, 4, 2_100_000
    idx = np.repeat(np.arange(S), n // S).astype(np.int64)
    src = rng.random((n, F), dtype=np.float32) + 0.5
    s, i = torch.from_numpy(src).to("cuda"), torch.from_numpy(idx).to("cuda")
    for op in ("sum", "mean"):
        say(f"long one-signed segments {op} {choice}")
        ref, terms = oracle_segment(src, idx, S, op)
        compare(geot.segment_reduce(s, i, S, op, choice=choice).cpu().numpy(), ref, op, terms,
                f"rows {op} {choice}")
    nx = 1000
    col = rng.integers(0, nx, n).astype(np.int64)
    w = rng.random(n, dtype=np.float32) + 0.5
    X = rng.random((nx, F), dtype=np.float32) + 0.5
    c, wt, xg = torch.from_numpy(col).to("cuda"), torch.from_numpy(w).to("cuda"), torch.from_numpy(X).to("cuda")
    for op in ("sum", "mean"):
        ref, terms = oracle_gather(X, col, w, idx, S, op)
        compare(geot.gather_scatter(xg, c, wt, i, S, op, choice=choice).cpu().numpy(), ref, op, terms,
                f"gather {op} {choice}")
