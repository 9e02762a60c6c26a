"""Randomized parity sweep: seeded random problems of every form against the oracle.

Each case draws a segment reduction or a fused gather form with random sizes (1 to about
1.5 M rows, log-uniform), width (1 to 512, ragged widths included), length distribution,
values, storage type (fp32, bf16, fp16), id type (int64, int32), op and, in most cases, a
random forced kernel choice (family, vector width, lanes, rows, load policy and tile order;
choices the library refuses as unsupported are skipped). For max, a third of the cases hold
NaN, infinities and signed zeros. Each case checks the forward against the oracle (max and
counts exact, sum and mean within 1e-5 * sum|terms| + 1e-6), the gradients (the segment
form in the storage type: sum and max exact, mean within one unit in the last place; the
fused form within the bound, infinities and NaN matching), and for fp32 / int64 inputs the
caller-workspace form, the no-allocation form, the call with index statistics, the max with
recorded recipients and its gradients, and the transposed edge list (as sorted triples).
This sweep found two defects that the fixed tests below name: the fp32 bound on long
same-signed chains, and the recipient of a run that starts at -inf.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import compare, oracle_gather, oracle_segment, say
from workloads import random_gather_problem, random_problem

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
FS = [1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 31, 32, 33, 63, 64, 65, 100, 127, 128, 129, 255, 256, 257, 300, 512]
DISTS = ["uniform", "zipf", "lognormal", "poisson", "fixed", "one_heavy"]
SPECIAL = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0], dtype=np.float32)
UNSUPPORTED = 5
CASES_PER_CHUNK = 40


def up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def close(got, ref, terms, what):
    """Within the bound, or equal (infinities) or both NaN."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    with np.errstate(invalid="ignore"):
        ok = same | (np.abs(got - ref) <= 1e-5 * np.asarray(terms) + 1e-6)
    assert ok.all(), f"{what}: {int((~ok).sum())} elements, first at {tuple(np.argwhere(~ok)[0])}"


def random_choice(g, dt, it):
    if g.random() < 0.4:
        return None
    c = dict(family="sp" if (g.random() < 0.2 and dt == "f32" and it == "i64") else "ep")
    if g.random() < 0.7:
        c["vec"] = int(g.choice([1, 2, 4, 8]))
    if g.random() < 0.7:
        c["lanes"] = int(g.choice([1, 2, 4, 8, 16, 32, 64]))
    if g.random() < 0.7:
        c["rows"] = int(g.choice([1, 2, 3, 5, 8, 17, 64, 300]))
    if g.random() < 0.3:
        c["flags"] = int(g.choice([1, 2, 4, 5, 6]))
    if c["family"] == "sp" and g.random() < 0.5:
        c["groups"] = int(g.choice([1, 2, 4, 8]))
    return c


def sprinkle(a, g):
    """A copy of `a` with about 2 % of its elements NaN, +-inf or +-0."""
    a = a.copy()
    flat = a.reshape(-1)
    k = max(1, flat.size // 50)
    flat[g.integers(0, flat.size, k)] = g.choice(SPECIAL, k)
    return a


def segment_case(seed, g, nnz, S, F, dist, values, ef, dt, it, op, ch):
    what = f"case {seed}: segment nnz={nnz} S={S} F={F} {dist}/{values} {dt}/{it} {op} choice={ch}"
    p = random_problem(seed, nnz, S, F, dist, values, ef)
    src = sprinkle(p["src"], g) if op == "max" and g.random() < 0.3 else p["src"]
    t = torch.from_numpy(src).to(DT[dt])
    wide = t.float().numpy()
    s = t.to(DEV)
    i = up(p["index"]).to(torch.int32 if it == "i32" else torch.int64)
    ref, terms = oracle_segment(wide, p["index"], S, op)
    try:
        got = geot.segment_reduce(s, i, S, op, choice=ch).cpu().numpy()
    except geot.GeotError as e:
        if e.status == UNSUPPORTED:
            return False
        raise
    compare(got, ref, op, terms, what)
    gout = np.random.default_rng(seed + 1).standard_normal((S, F)).astype(np.float32)
    rg = np.asarray(oracle.segment_reduce_backward(gout, p["index"], op, wide if op == "max" else None,
                                                   ref if op == "max" else None), dtype=np.float32)
    gs = geot.segment_reduce_backward(up(gout), i, op, s if op == "max" else None,
                                      up(ref) if op == "max" else None, dtype=DT[dt]).float().cpu().numpy()
    rgd = torch.from_numpy(rg).to(DT[dt]).float().numpy()   # the oracle's, rounded to the storage type
    if op == "mean":
        if dt == "f32":
            assert np.all(np.abs(gs.astype(np.float64) - rg) <= 1e-5 * np.abs(rg) + 1e-30), what + " mean gradient"
        else:   # one unit in the last place: the fp32 quotient rounds to the storage type once more
            m = torch.from_numpy(np.abs(rgd)).to(DT[dt])
            ulp = (torch.nextafter(m, torch.full_like(m, float("inf"))).float() - m.float()).numpy()
            assert np.all(np.abs(gs - rgd) <= ulp), what + " mean gradient"
    else:
        assert np.array_equal(gs, rgd), what + " gradient"
    if dt == "f32" and it == "i64":
        try:
            nb = geot.workspace_size(nnz, S, F, op, choice=ch)
            ws = torch.empty(nb + int(g.integers(0, 4096)), dtype=torch.uint8, device=DEV)
            compare(geot.segment_reduce_ws(s, i, S, op, ws, choice=ch).cpu().numpy(), ref, op, terms, what + " ws")
        except geot.GeotError as e:
            if e.status != UNSUPPORTED:
                raise
        try:
            o = torch.empty((S, F), device=DEV)
            compare(geot.segment_reduce_noalloc(s, i, S, op, o).cpu().numpy(), ref, op, terms, what + " noalloc")
        except geot.GeotError as e:   # beyond the static array
            if "workspace" not in e.detail:
                raise
        st = geot.index_stats(i, S)
        compare(geot.segment_reduce(s, i, S, op, stats=st).cpu().numpy(), ref, op, terms, what + " stats")
        if op == "max":
            out, arg = geot.segment_reduce_max_arg(s, i, S)
            compare(out.cpu().numpy(), ref, "max", None, what + " recording")
            ga = geot.segment_reduce_backward_max_arg(up(gout), i, arg).cpu().numpy()
            assert np.array_equal(ga.view(np.uint32), rg.view(np.uint32)), what + " gradient from recipients"
    return True


def gather_case(seed, g, nnz, S, F, dist, values, ef, dt, it, op, ch):
    nx = max(1, int(math.exp(g.uniform(0, math.log(3 * nnz + 2)))))
    if nx * F > 20_000_000:
        nx = max(1, 20_000_000 // F)
    weighted = g.random() < 0.7
    what = f"case {seed}: gather nnz={nnz} R={S} nx={nx} F={F} {dist} w={weighted} {dt}/{it} {op} choice={ch}"
    q = random_gather_problem(seed, nnz, S, nx, F, dist, "int" if values == "int" else "normal", weighted, ef)
    X, col, w, row = q["X"], q["col"], q["weight"], q["index"]
    if op == "max" and g.random() < 0.3:
        X = sprinkle(X, g)
    t = torch.from_numpy(X).to(DT[dt])
    wide = t.float().numpy()
    xi = t.to(DEV)
    ty = torch.int32 if it == "i32" else torch.int64
    ci, ri = up(col).to(ty), up(row).to(ty)
    wi = up(w) if w is not None else None
    ref, terms = oracle_gather(wide, col, w, row, S, op)
    try:
        got = geot.gather_scatter(xi, ci, wi, ri, S, op, choice=ch).cpu().numpy()
    except geot.GeotError as e:
        if e.status == UNSUPPORTED:
            return False
        raise
    compare(got, ref, op, terms, what)
    gout = np.random.default_rng(seed + 1).standard_normal((S, F)).astype(np.float32)
    o = np.ascontiguousarray(ref, dtype=np.float32) if op == "max" else None
    gx, gw = geot.gather_scatter_backward(xi, ci, wi, ri, up(gout), op, up(o) if o is not None else None)
    rx, rw = oracle.gather_scatter_backward(wide, col, w, row, gout, op, o)
    ax, aw = oracle.gather_scatter_backward(wide, col, w, row, gout, op, o, absolute=True)
    close(gx.cpu().numpy(), rx, ax, what + " grad_X")
    if gw is not None and rw is not None:
        close(gw.cpu().numpy(), rw, aw, what + " grad_w")
    if dt == "f32" and it == "i64":
        try:
            nb = geot.workspace_size(nnz, S, F, op, gather=True, weighted=w is not None, choice=ch)
            ws = torch.empty(nb + int(g.integers(0, 4096)), dtype=torch.uint8, device=DEV)
            compare(geot.gather_scatter_ws(xi, ci, wi, ri, S, op, ws, choice=ch).cpu().numpy(), ref, op, terms,
                    what + " ws")
        except geot.GeotError as e:
            if e.status != UNSUPPORTED:
                raise
        if op == "max":
            out, arg = geot.gather_scatter_max_arg(xi, ci, wi, ri, S)
            compare(out.cpu().numpy(), ref, "max", None, what + " recording")
            gx2, gw2 = geot.gather_scatter_backward_max_arg(xi, ci, wi, ri, up(gout), arg)
            close(gx2.cpu().numpy(), rx, ax, what + " grad_X from recipients")
            if gw2 is not None and rw is not None:
                close(gw2.cpu().numpy(), rw, aw, what + " grad_w from recipients")
        else:
            sc, rt, cf = (a.cpu().numpy() for a in geot.transpose_edges(ci, wi, ri, nx, S, op))
            coef = w.copy() if w is not None else np.ones(nnz, dtype=np.float32)
            if op == "mean":
                deg = np.bincount(row, minlength=S).astype(np.float32)
                coef = (coef / deg[row]).astype(np.float32)
            assert np.all(np.diff(sc) >= 0), what + " transposition sorted"
            want = np.lexsort((coef.view(np.uint32), row, col))
            got_ = np.lexsort((cf.view(np.uint32), rt, sc))
            assert np.array_equal(sc[got_], col[want]) and np.array_equal(rt[got_], row[want]) and \
                np.array_equal(cf[got_].view(np.uint32), coef[want].view(np.uint32)), what + " transposition"
    return True


@pytest.mark.parametrize("chunk", range(4))
def test_random_problems_against_the_oracle(chunk):
    ran = 0
    for case in range(CASES_PER_CHUNK):
        seed = 7_000_000 + chunk * 1000 + case
        g = np.random.default_rng(seed)
        gather = g.random() < 0.45
        nnz = int(math.exp(g.uniform(0, math.log(1_500_000))))
        S = max(1, int(math.exp(g.uniform(0, math.log(2 * nnz + 2)))))
        F = int(g.choice(FS))
        if nnz * F > 40_000_000:
            nnz = max(1, 40_000_000 // F)
        dist = str(g.choice(DISTS))
        values = str(g.choice(["normal", "int", "negative"]))
        ef = float(g.choice([0.0, 0.0, 0.1, 0.5]))
        dt = str(g.choice(["f32", "f32", "f32", "bf16", "f16"]))
        it = str(g.choice(["i64", "i32"]))
        op = str(g.choice(["sum", "mean", "max"]))
        ch = random_choice(g, dt, it)
        say(f"sweep case {seed}: {'gather' if gather else 'segment'} nnz={nnz} S={S} F={F} {dt}/{it} {op} {ch}")
        run = gather_case if gather else segment_case
        ran += run(seed, g, nnz, S, F, dist, values, ef, dt, it, op, ch)
    assert ran >= CASES_PER_CHUNK // 2
