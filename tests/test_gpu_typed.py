"""GPU parity of the typed entry points: bf16 / fp16 storage and int32 ids.

A bf16 or fp16 value widens to fp32 exactly, so the oracle runs on the widened
fp32 copy of the very data the GPU reads (rounded to the storage type on the
host by torch, then widened on the host): the typed call meets the fp32 bar on
it, max exact and sum / mean within 1e-5 * sum|terms| + 1e-6. int32 ids are the
int64 ids narrowed, which changes nothing the oracle sees.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import compare, forward_for_gradient, oracle_gather, oracle_segment, say
from workloads import make_config, random_gather_problem, random_problem

pytestmark = pytest.mark.gpu
OPS = ("sum", "mean", "max")
DEV = "cuda:0"
DT = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}
IT = {"i64": torch.int64, "i32": torch.int32}


def stored(a, dt):
    """(host tensor in the storage type, its exact fp32 widening as numpy)."""
    t = torch.from_numpy(np.ascontiguousarray(a)).to(DT[dt])
    return t, t.float().numpy()


def ids(a, it):
    return torch.from_numpy(np.ascontiguousarray(a)).to(IT[it]).to(DEV)


def up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


CHOICES = [
    None,
    dict(family="ep", lanes=64, vec=1, rows=2),   # many blocks: several partial levels
    dict(family="ep", lanes=1, rows=3),
    dict(family="ep", lanes=4, vec=2, rows=7),
    dict(family="ep", lanes=2, vec=8, rows=5),    # 16-byte loads of 16-bit storage
    dict(family="ep", lanes=64, vec=8, rows=1),   # lanes capped at 32; partial levels run 4-wide on 64 lanes
]


def choices(dt):
    """vec 8 is for 16-bit storage only (fp32 data with vec 8 is refused)."""
    return [c for c in CHOICES if dt != "f32" or c is None or c.get("vec") != 8]

CASES = [
    # seed, nnz, S, F, dist, values, empty_frac
    (11, 30000, 2000, 32, "zipf", "uniform", 0.05),
    (12, 25000, 400, 1, "lognormal", "normal", 0.1),
    (13, 20000, 3000, 3, "uniform", "normal", 0.2),
    (14, 40000, 50, 64, "one_heavy", "normal", 0.3),
    (15, 9000, 700, 130, "poisson", "uniform", 0.0),
    (16, 5000, 6000, 8, "uniform", "negative", 0.5),   # more segments than rows, all-negative max
    (17, 6000, 300, 512, "zipf", "normal", 0.1),       # two column tiles of 256 at vec 8
]


ROW64_CASES = [
    # seed, nnz, S, dist, values, empty_frac
    (21, 50000, 3000, "zipf", "normal", 0.1),
    (22, 70001, 7, "one_heavy", "uniform", 0.0),     # odd row count
    (23, 12345, 20000, "uniform", "negative", 0.6),  # more segments than rows, long empty runs
]
ROW64_CHOICES = [
    None,
    dict(family="ep", lanes=4, vec=8, rows=1),    # many blocks, several partial levels
    dict(family="ep", lanes=4, vec=8, rows=3),
    dict(family="ep", lanes=4, vec=8, rows=33),
    dict(family="ep", lanes=4, vec=8, rows=8, flags=2),   # cached loads asked for explicitly
]


@pytest.mark.parametrize("dt,it", [("bf16", "i64"), ("bf16", "i32"), ("f16", "i64"), ("f16", "i32")])
@pytest.mark.parametrize("case", ROW64_CASES, ids=lambda c: f"seed{c[0]}")
def test_segment_reduce_64_byte_rows(dt, it, case):
    """16-bit rows of 64 bytes (F = 32: 8-element vectors, 4 lanes a row, half a cache line
    a row): odd row counts per group, an odd total, several partial levels and long empty
    runs, with src at the start of its allocation and 64 bytes into it. Every op and the
    recording max against the oracle: max and the recipients exact, sum / mean within the
    bound."""
    seed, nnz, S, dist, values, ef = case
    F = 32
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    t, wide = stored(p["src"], dt)
    i = ids(p["index"], it)
    padded = torch.zeros((nnz + 1, F), dtype=DT[dt])
    padded[1:] = t
    for name, s in (("aligned", t.to(DEV)), ("offset", padded.to(DEV)[1:])):
        assert (s.data_ptr() % 128 == 0) == (name == "aligned")
        for op in OPS:
            ref, terms = oracle_segment(wide, p["index"], S, op)
            for ch in ROW64_CHOICES:
                say(f"64-byte rows {dt}/{it} seed={seed} {name} {op} choice={ch}")
                got = geot.segment_reduce(s, i, S, op, choice=ch).cpu().numpy()
                compare(got, ref, op, terms, f"64-byte rows {dt}/{it} seed={seed} {name} {op} {ch}")
        ref = oracle.segment_reduce(wide, p["index"], S, "max")
        for ch in ROW64_CHOICES:
            out, arg = geot.segment_reduce_max_arg(s, i, S, choice=ch)
            compare(out.cpu().numpy(), ref, "max", None, f"64-byte rows recording {dt}/{it} {name} {ch}")
            a = arg.cpu().numpy().view(np.uint32).astype(np.int64)
            idx = p["index"]
            # the lowest row of each segment whose value equals the maximum (none: 2^32 - 1)
            want = np.full((S, F), (1 << 32) - 1, dtype=np.int64)
            hit = wide == ref[idx]
            rows = np.broadcast_to(np.arange(nnz)[:, None], (nnz, F))
            seg_f = idx[:, None] * F + np.arange(F)[None, :]
            flat = want.reshape(-1)
            np.minimum.at(flat, seg_f[hit], rows[hit])
            assert np.array_equal(a, want), f"64-byte rows recipients {dt}/{it} seed={seed} {name} {ch}"


@pytest.mark.parametrize("dt,it", [("bf16", "i64"), ("bf16", "i32"), ("f16", "i64"), ("f16", "i32"),
                                   ("f32", "i32")])
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c[0]}_F{c[3]}")
def test_segment_reduce_typed(dt, it, case):
    seed, nnz, S, F, dist, values, ef = case
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    t, wide = stored(p["src"], dt)
    s, i = t.to(DEV), ids(p["index"], it)
    for op in OPS:
        ref, terms = oracle_segment(wide, p["index"], S, op)
        for ch in choices(dt):
            say(f"typed segment {dt}/{it} seed={seed} F={F} {op} choice={ch}")
            got = geot.segment_reduce(s, i, S, op, choice=ch).cpu().numpy()
            compare(got, ref, op, terms, f"{dt}/{it} seed={seed} {op} choice={ch}")


GATHER_CASES = [
    # seed, nnz, R, n_x, F, dist, weighted, empty_frac
    (21, 30000, 1500, 900, 32, "zipf", True, 0.05),
    (22, 20000, 800, 5000, 5, "lognormal", False, 0.1),
    (23, 15000, 3000, 64, 128, "uniform", True, 0.0),
    (24, 8000, 9000, 300, 2, "one_heavy", True, 0.4),
]


@pytest.mark.parametrize("dt,it", [("bf16", "i32"), ("f16", "i64"), ("f32", "i32"), ("bf16", "i64")])
@pytest.mark.parametrize("case", GATHER_CASES, ids=lambda c: f"seed{c[0]}_F{c[4]}")
def test_gather_scatter_typed(dt, it, case):
    seed, nnz, R, nx, F, dist, weighted, ef = case
    p = random_gather_problem(seed, nnz, R, nx, F, dist, "normal", weighted, ef)
    t, wide = stored(p["X"], dt)
    X = t.to(DEV)
    col, row = ids(p["col"], it), ids(p["index"], it)
    w = torch.from_numpy(p["weight"]).to(DEV) if p["weight"] is not None else None
    for op in OPS:
        ref, terms = oracle_gather(wide, p["col"], p["weight"], p["index"], R, op)
        for ch in choices(dt):
            say(f"typed gather {dt}/{it} seed={seed} F={F} {op} choice={ch}")
            got = geot.gather_scatter(X, col, w, row, R, op, choice=ch).cpu().numpy()
            compare(got, ref, op, terms, f"gather {dt}/{it} seed={seed} {op} choice={ch}")


def test_typed_exact_arithmetic():
    """Values in {-1, 0, 1} are exact in every storage type and every partial sum
    is an integer below 2^24: sums are bit-exact at any kernel choice."""
    p = random_problem(31, 200000, 300, 16, "lognormal", "ternary", 0.1)
    ref = oracle.segment_reduce(p["src"], p["index"], 300, "sum")
    for dt in ("bf16", "f16"):
        t, wide = stored(p["src"], dt)
        assert np.array_equal(wide, p["src"])
        for it in ("i64", "i32"):
            for ch in CHOICES:
                got = geot.segment_reduce(t.to(DEV), ids(p["index"], it), 300, "sum", choice=ch)
                assert np.array_equal(got.cpu().numpy(), ref), f"{dt}/{it} choice={ch}"


def test_typed_misaligned_storage_and_empty_input():
    """A bf16 view that starts 2 bytes into its buffer only allows 2-byte loads;
    nnz == 0 fills zeros as the fp32 call does."""
    p = random_problem(32, 7000, 500, 4, "zipf", "normal", 0.1)
    t, wide = stored(p["src"], "bf16")
    buf = torch.empty(t.numel() + 1, dtype=torch.bfloat16, device=DEV)
    view = buf[1:].view(t.shape)
    view.copy_(t.to(DEV))
    assert view.data_ptr() % 4 == 2
    for op in OPS:
        ref, terms = oracle_segment(wide, p["index"], 500, op)
        got = geot.segment_reduce(view, ids(p["index"], "i32"), 500, op)
        assert geot.last_choice()["vec"] == 1
        compare(got.cpu().numpy(), ref, op, terms, f"misaligned bf16 {op}")
    empty = torch.empty((0, 4), dtype=torch.float16, device=DEV)
    out = torch.full((9, 4), 7.0, device=DEV)
    geot.segment_reduce(empty, torch.empty(0, dtype=torch.int32, device=DEV), 9, "max", out=out)
    assert torch.count_nonzero(out).item() == 0


def test_typed_selector_never_runs_segment_parallel():
    """Where the tree picks the segment-parallel family (fp32, int64), a typed call
    of the same shape runs the element-parallel family and still matches."""
    p = random_problem(33, 2_000_000, 100_000, 8, "poisson", "normal", 0.0)
    geot.segment_reduce(torch.from_numpy(p["src"]).to(DEV), torch.from_numpy(p["index"]).to(DEV),
                        100_000, "mean")
    say("fp32 choice", geot.last_choice())
    t, wide = stored(p["src"], "bf16")
    got = geot.segment_reduce(t.to(DEV), ids(p["index"], "i32"), 100_000, "mean").cpu().numpy()
    assert geot.last_choice()["family"] == 1
    ref, terms = oracle_segment(wide, p["index"], 100_000, "mean")
    compare(got, ref, "mean", terms, "typed mean, fp32 shape")


def test_c3_powerlaw_graph_bf16_i32_full():
    """The power-law workload (114,615,892 x 32) stored as bf16 with int32 ids: every output
    element against the (multi-threaded) oracle run on the stored rows widened to fp32."""
    c = make_config("c3_powerlaw_graph")
    src, idx, S = c["src"], c["index"], c["num_segments"]
    s = torch.from_numpy(src).to(DEV).to(torch.bfloat16)
    say("c3 bf16 uploaded")
    got = geot.segment_reduce(s, ids(idx, "i32"), S, "sum").cpu().numpy()
    # the fp32 leaf for this shape, loaded 8 wide: half the lanes, twice the rows
    fp, lc = geot.select(idx.size, S, 32, "sum"), geot.last_choice()
    assert (lc["vec"], lc["lanes"], lc["rows"]) == (8, fp["lanes"] // 2, 2 * fp["rows"]), (lc, fp)
    wide = s.float().cpu().numpy()   # the stored rows, widened exactly
    del s
    torch.cuda.empty_cache()
    m = oracle.mt()
    compare(got, m.segment_reduce(wide, idx, S, "sum"), "sum", m.abs_term_sum(wide, idx, S, "sum"),
            "c3 bf16 (every element)")


def test_c4_spmm_bf16_i32_full():
    """The SpMM workload with X stored as bf16 and int32 col / row: every output element."""
    c = make_config("c4_spmm")
    X, col, w, row, R = c["X"], c["col"], c["weight"], c["index"], c["num_segments"]
    t, wide = stored(X, "bf16")
    say("c4 bf16 uploaded")
    got = geot.gather_scatter(t.to(DEV), ids(col, "i32"), torch.from_numpy(w).to(DEV), ids(row, "i32"),
                              R, "sum").cpu().numpy()
    m = oracle.mt()
    compare(got, m.gather_scatter(wide, col, w, row, R, "sum"), "sum", m.abs_term_sum(wide, row, R, "sum", col, w),
            "c4 bf16 (every element)")


BWD_CASES = [
    # seed, nnz, S, F, dist, values, empty_frac
    (41, 20000, 900, 32, "zipf", "normal", 0.1),      # 8-wide 16-bit vectors
    (42, 15000, 700, 3, "lognormal", "normal", 0.05),  # 1-wide
    (43, 12000, 500, 12, "uniform", "int", 0.2),       # 4-wide; integer values tie under max
    (44, 8000, 300, 6, "one_heavy", "int", 0.1),       # 2-wide
    (45, 4_000_000, 10_000, 32, "zipf", "normal", 0.3),  # >= 64 MB, segments of >= a block's rows: offsets
]
HALF_ULP = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11, "f32": 2.0 ** -23}
# one rounding in the subnormal range is absolute: half the spacing 2^-24 of binary16's
# subnormals (bf16 shares fp32's exponent range, so its subnormals are far below these values)
HALF_SUBNORMAL = {"bf16": 0.0, "f16": 2.0 ** -25, "f32": 0.0}


@pytest.mark.parametrize("dt,it", [("bf16", "i64"), ("bf16", "i32"), ("f16", "i32"), ("f16", "i64"),
                                   ("f32", "i32")])
@pytest.mark.parametrize("case", BWD_CASES, ids=lambda c: f"seed{c[0]}_F{c[3]}")
def test_segment_backward_typed(dt, it, case):
    """The gradient is stored in src's type: for sum and max it is the oracle's gradient on
    the widened src rounded once to that type (bit-exact, torch rounds to nearest even as
    the library does); for mean it is within one rounding of the type (plus the fp32
    reciprocal's error) of the exact quotient."""
    seed, nnz, S, F, dist, values, ef = case
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    t, wide = stored(p["src"], dt)
    s, i = t.to(DEV), ids(p["index"], it)
    g = np.random.default_rng(seed).standard_normal((S, F)).astype(np.float32)
    gd = torch.from_numpy(g).to(DEV)
    for op in OPS:
        say(f"typed segment backward {dt}/{it} seed={seed} F={F} {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.segment_reduce(wide, p["index"], S, op),
                                       geot.segment_reduce(s, i, S, op), f"{dt}/{it} seed={seed}")
        got = geot.segment_reduce_backward(gd, i, op, s if op == "max" else None,
                                           up(out), dtype=DT[dt])
        assert got.dtype == DT[dt] and got.shape == (nnz, F)
        ref = oracle.segment_reduce_backward(g, p["index"], op, wide, out)
        if op in ("sum", "max"):
            assert torch.equal(got.cpu(), torch.from_numpy(np.ascontiguousarray(ref)).to(DT[dt])), \
                f"{dt}/{it} seed={seed} {op}"
        else:
            err = np.abs(got.cpu().float().numpy().astype(np.float64) - ref.astype(np.float64))
            lim = (HALF_ULP[dt] + 1e-6) * np.abs(ref.astype(np.float64)) + HALF_SUBNORMAL[dt] + 1e-30
            assert np.all(err <= lim), f"{dt}/{it} seed={seed} mean: worst {float(np.max(err - lim))}"


# fp32 bit patterns around the roundings to bf16 and binary16: ties (to the even neighbour),
# neighbours of ties, the largest finite values and the ties past them (to infinity), fp32
# subnormals (bf16 keeps fp32's exponent range, binary16 rounds them to zero or its own
# subnormals), signed zeros, infinities and NaNs
SPECIAL_BITS = [
    0x00000000, 0x80000000, 0x3F808000, 0x3F818000, 0x3F808001, 0x3F807FFF, 0xBF808000,
    0x3F801000, 0x3F803000, 0x3F801001, 0xBF803000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F7F7FFF,
    0x7F7F8000, 0x477FE000, 0x477FF000, 0x477FEFFF, 0xC77FF000, 0x00000001, 0x00008000,
    0x00018000, 0x007FFFFF, 0x80018000, 0x33000000, 0x33C00000, 0x387FC000, 0x387FE000,
    0x7F800000, 0xFF800000, 0x7FC00000, 0x7F800001, 0xFFC00001, 0x40490FDB, 0xBDCCCCCD,
]


def rne16_bits(a, dt):
    """16-bit patterns of fp32 array `a` rounded to nearest even (NaN entries unspecified)."""
    if dt == "f16":
        with np.errstate(over="ignore"):
            return a.astype(np.float16).view(np.uint16)
    u = a.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("F", [32, 12, 6, 3], ids=lambda f: f"F{f}")
def test_segment_backward_rounds_like_torch(dt, F):
    """Gradients narrowed to 16-bit storage round to nearest even, bit for bit, on the values
    where a rounding can go wrong (ties, overflow, subnormals, signed zeros, infinities; NaN
    stays NaN), through the 8-, 4-, 2- and 1-wide stores of sum and max. The expected bits
    come from the definition: binary16 by numpy's conversion; bf16, the upper half of an fp32
    pattern, by rounding the pattern as an integer to a multiple of 2^16, ties to the even
    multiple (for a finite value the patterns order like the magnitudes, and the carry out of
    the largest finite bf16 lands on infinity's pattern)."""
    rng = np.random.default_rng(80 + F)
    S, nnz = 97, 5000
    index = np.sort(rng.integers(0, S, nnz)).astype(np.int64)
    special = np.array(SPECIAL_BITS, dtype=np.uint32).view(np.float32)
    g = special[rng.integers(0, special.size, (S, F))]
    gd = torch.from_numpy(g).to(DEV)
    t, wide = stored(rng.standard_normal((nnz, F)).astype(np.float32), dt)
    i = ids(index, "i32")
    for op in ("sum", "max"):
        say(f"special-value rounding {dt} F={F} {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.segment_reduce(wide, index, S, op),
                                       geot.segment_reduce(t.to(DEV), i, S, op), f"{dt} F={F}")
        got = geot.segment_reduce_backward(gd, i, op, t.to(DEV) if op == "max" else None, up(out),
                                           dtype=DT[dt]).cpu()
        exact = np.ascontiguousarray(oracle.segment_reduce_backward(g, index, op, wide, out), dtype=np.float32)
        nan = np.isnan(exact)
        rb = rne16_bits(exact, dt)
        gb = got.view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(np.isnan(got.float().numpy()), nan), f"{dt} F={F} {op}: NaN positions"
        bad = (gb != rb) & ~nan
        if bad.any():
            r, c = [int(v[0]) for v in np.nonzero(bad)]
            raise AssertionError(f"{dt} F={F} {op}: {int(bad.sum())} values differ; first at ({r}, {c}): "
                                 f"fp32 {hex(int(exact[r, c:c + 1].view(np.uint32)[0]))} -> "
                                 f"{hex(int(gb[r, c]))}, expected {hex(int(rb[r, c]))}")


def test_segment_backward_typed_through_autograd():
    """A bf16 src with int32 ids: autograd's gradient is bf16 and equals the fp32 gradient of
    the widened src rounded once."""
    p = random_problem(45, 30000, 1200, 16, "zipf", "normal", 0.1)
    t, wide = stored(p["src"], "bf16")
    from paper_2404_03019_amd.autograd import segment_reduce as ag_segment_reduce
    for op in OPS:
        x = t.to(DEV).requires_grad_(True)
        out = ag_segment_reduce(x, ids(p["index"], "i32"), 1200, op)
        g = torch.randn(out.shape, device=DEV, generator=torch.Generator(device=DEV).manual_seed(7))
        out.backward(g)
        assert x.grad.dtype == torch.bfloat16
        xf = torch.from_numpy(wide).to(DEV).requires_grad_(True)
        outf = ag_segment_reduce(xf, ids(p["index"], "i64"), 1200, op)
        outf.backward(g)
        # both paths form the same fp32 values (mean: the same products); bf16 rounds them once
        assert torch.equal(x.grad, xf.grad.to(torch.bfloat16)), op


GS_BWD_CASES = [
    # seed, nnz, R, n_x, F, dist, values, weighted
    (51, 20000, 1200, 900, 32, "zipf", "normal", True),     # 8-wide 16-bit vectors
    (52, 15000, 800, 2000, 3, "lognormal", "normal", True),  # 1-wide
    (53, 10000, 500, 700, 12, "uniform", "int", False),      # 4-wide; ties under max
    (54, 8000, 300, 400, 6, "one_heavy", "int", True),       # 2-wide
]


@pytest.mark.parametrize("dt,it", [("bf16", "i32"), ("bf16", "i64"), ("f16", "i32"), ("f32", "i32")])
@pytest.mark.parametrize("case", GS_BWD_CASES, ids=lambda c: f"seed{c[0]}_F{c[4]}")
def test_gather_backward_typed(dt, it, case):
    """16-bit X and int32 ids: the gradients (fp32) equal the oracle's on the widened X within
    the fp32 bound, max routing to the same recipients."""
    seed, nnz, R, nx, F, dist, values, weighted = case
    q = random_gather_problem(seed, nnz, R, nx, F, dist, values, weighted, 0.05)
    t, wide = stored(q["X"], dt)
    X = t.to(DEV)
    col, row = ids(q["col"], it), ids(q["index"], it)
    w = torch.from_numpy(q["weight"]).to(DEV) if q["weight"] is not None else None
    g = np.random.default_rng(seed).standard_normal((R, F)).astype(np.float32)
    for op in OPS:
        say(f"typed gather backward {dt}/{it} seed={seed} F={F} {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.gather_scatter(wide, q["col"], q["weight"], q["index"], R, op),
                                       geot.gather_scatter(X, col, w, row, R, op), f"{dt}/{it} seed={seed}")
        gx, gw = geot.gather_scatter_backward(X, col, w, row, torch.from_numpy(g).to(DEV), op, up(out))
        assert gx.dtype == torch.float32
        rx, rw = oracle.gather_scatter_backward(wide, q["col"], q["weight"], q["index"], g, op, out)
        ax, aw = oracle.gather_scatter_backward(wide, q["col"], q["weight"], q["index"], g, op, out,
                                                absolute=True)
        for got, ref, terms, what in ((gx, rx, ax, "grad_X"), (gw, rw, aw, "grad_w")):
            if got is None:
                assert not weighted and what == "grad_w"
                continue
            err = np.abs(got.cpu().numpy().astype(np.float64) - ref.astype(np.float64))
            assert np.all(err <= 1e-5 * terms + 1e-6), f"{what} {dt}/{it} seed={seed} {op}"


@pytest.mark.parametrize("op", OPS)
def test_gather_autograd_bf16_int32(op):
    """The differentiable fused form over bf16 x and int32 ids, with a Graph (its int32 ids
    widened for the transposition) and without: x.grad keeps bf16 and equals, within one
    bf16 rounding, the gradient of the same expression on the widened x with int64 ids;
    the weight gradient meets the fp32 bound."""
    from paper_2404_03019_amd.autograd import Graph, gather_scatter
    q = random_gather_problem(56, 30000, 2000, 1500, 16, "zipf", "normal", True, 0.02)
    x16, wide = stored(q["X"], "bf16")
    t = torch.from_numpy(np.random.default_rng(57).standard_normal((2000, 16)).astype(np.float32)).to(DEV)
    grads = {}
    for name, xin, it in (("bf16", x16.to(DEV), "i32"), ("f32", torch.from_numpy(wide).to(DEV), "i64")):
        for use_graph in (False, True):
            x = xin.clone().requires_grad_(True)
            w = torch.from_numpy(q["weight"]).to(DEV).requires_grad_(True)
            col, row = ids(q["col"], it), ids(q["index"], it)
            graph = Graph(col, row, 2000, w, num_src=1500) if use_graph else None
            (gather_scatter(x, col, w, row, 2000, op, graph) * t).sum().backward()
            assert x.grad.dtype == xin.dtype
            grads[name, use_graph] = (x.grad.float(), w.grad)
    for use_graph in (False, True):
        xb, wb = grads["bf16", use_graph]
        xf, wf = grads["f32", use_graph]
        assert torch.allclose(xb, xf.to(torch.bfloat16).float(), rtol=2 ** -7, atol=1e-5), (op, use_graph)
        assert torch.allclose(wb, wf, rtol=1e-4, atol=1e-5), (op, use_graph)


def test_typed_backward_misaligned_and_empty():
    """Gradients over a bf16 X (and src) view that starts 2 bytes into its buffer, so only
    2-byte loads are allowed, F = 16; and empty edge lists with int32 ids."""
    q = random_gather_problem(58, 9000, 600, 700, 16, "zipf", "int", True, 0.05)
    t, wide = stored(q["X"], "bf16")
    buf = torch.empty(t.numel() + 1, dtype=torch.bfloat16, device=DEV)
    X = buf[1:].view(t.shape)
    X.copy_(t.to(DEV))
    assert X.data_ptr() % 4 == 2
    col, row = ids(q["col"], "i32"), ids(q["index"], "i32")
    w = torch.from_numpy(q["weight"]).to(DEV)
    g = np.random.default_rng(59).standard_normal((600, 16)).astype(np.float32)
    for op in OPS:
        say(f"misaligned bf16 gather backward {op}")
        out = None
        if op == "max":
            out = forward_for_gradient(oracle.gather_scatter(wide, q["col"], q["weight"], q["index"], 600, op),
                                       geot.gather_scatter(X, col, w, row, 600, op), "misaligned bf16")
        gx, gw = geot.gather_scatter_backward(X, col, w, row, torch.from_numpy(g).to(DEV), op, up(out))
        rx, rw = oracle.gather_scatter_backward(wide, q["col"], q["weight"], q["index"], g, op, out)
        ax, aw = oracle.gather_scatter_backward(wide, q["col"], q["weight"], q["index"], g, op, out,
                                                absolute=True)
        for got, ref, terms, what in ((gx, rx, ax, "grad_X"), (gw, rw, aw, "grad_w")):
            err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
            assert np.all(err <= 1e-5 * terms + 1e-6), f"misaligned {what} {op}"
    p = random_problem(60, 7000, 400, 16, "zipf", "int", 0.1)
    ts, sw = stored(p["src"], "bf16")
    sb = torch.empty(ts.numel() + 1, dtype=torch.bfloat16, device=DEV)
    src = sb[1:].view(ts.shape)
    src.copy_(ts.to(DEV))
    i32 = ids(p["index"], "i32")
    gs = np.random.default_rng(61).standard_normal((400, 16)).astype(np.float32)
    out = forward_for_gradient(oracle.segment_reduce(sw, p["index"], 400, "max"),
                               geot.segment_reduce(src, i32, 400, "max"), "misaligned bf16 segment")
    got = geot.segment_reduce_backward(torch.from_numpy(gs).to(DEV), i32, "max", src, up(out))
    ref = oracle.segment_reduce_backward(gs, p["index"], "max", sw, out)
    assert torch.equal(got.cpu(), torch.from_numpy(ref).to(torch.bfloat16)), "misaligned bf16 segment max"
    # no edges: grad_X is zero, grad_w empty; no rows: grad_src empty
    e32 = torch.empty(0, dtype=torch.int32, device=DEV)
    gx, gw = geot.gather_scatter_backward(X, e32, torch.empty(0, device=DEV), e32,
                                          torch.from_numpy(g).to(DEV), "sum")
    assert gx.shape == (700, 16) and torch.count_nonzero(gx).item() == 0 and gw.numel() == 0
    e = geot.segment_reduce_backward(torch.from_numpy(gs).to(DEV), e32, "mean", dtype=torch.bfloat16)
    assert e.shape == (0, 16) and e.dtype == torch.bfloat16
