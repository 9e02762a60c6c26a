"""GPU parity on the named workloads at their full sizes, with the selector's default
kernel choice (the launch configuration the bench times).

Every output element of every workload is compared with the oracle. The two large
power-law workloads use the multi-threaded oracle (the serial oracle's definitions
with segments split across host threads, pinned to it bit for bit by
``test_oracle_mt.py``), and on a sample of rows (the longest segments always
included) the serial oracle is run too and must agree with it bit for bit; the
power-law graph is also checked for per-feature conservation over all rows.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_03019_amd as geot
from gpu_util import compare, oracle_gather, oracle_segment, say
from workloads import make_config
from workloads.generators import C2_FEATURES

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def test_c1_zipf_small_full():
    c = make_config("c1_zipf_small")
    for op in ("sum", "mean", "max"):
        say(f"c1 {op}")
        got = geot.segment_reduce(up(c["src"]), up(c["index"]), c["num_segments"], op).cpu().numpy()
        ref, terms = oracle_segment(c["src"], c["index"], c["num_segments"], op)
        compare(got, ref, op, terms, f"c1 {op}")


def test_c1_literal_stress_full():
    c = make_config("c1_literal")
    for op in ("sum", "max"):
        got = geot.segment_reduce(up(c["src"]), up(c["index"]), c["num_segments"], op).cpu().numpy()
        ref, terms = oracle_segment(c["src"], c["index"], c["num_segments"], op)
        compare(got, ref, op, terms, f"c1-literal {op}")


@pytest.fixture(scope="module")
def c2():
    return make_config("c2_poisson_fsweep", F=256)


@pytest.mark.parametrize("F", C2_FEATURES)
def test_c2_feature_sweep_full(c2, F):
    src = np.ascontiguousarray(c2["src"][:, :F])
    idx = c2["index"]
    S = c2["num_segments"]
    s, i = up(src), up(idx)
    for op in ("sum", "mean", "max"):
        say(f"c2 F={F} {op}")
        got = geot.segment_reduce(s, i, S, op).cpu().numpy()
        ref, terms = oracle_segment(src, idx, S, op)
        compare(got, ref, op, terms, f"c2 F={F} {op}")


def test_c5_pointcloud_full():
    c = make_config("c5_pointcloud_knn")
    s, i = up(c["src"]), up(c["index"])
    for op in ("mean", "max", "sum"):
        say(f"c5 {op}")
        got = geot.segment_reduce(s, i, c["num_segments"], op).cpu().numpy()
        ref, terms = oracle_segment(c["src"], c["index"], c["num_segments"], op)
        compare(got, ref, op, terms, f"c5 {op}")


def _sample_segments(lengths, k, seed):
    rng = np.random.default_rng(seed)
    S = lengths.size
    picks = {0, S - 1, int(np.argmax(lengths)), int(np.argmin(lengths))}
    picks.update(int(x) for x in np.argsort(lengths)[-8:])  # the heaviest tail
    picks.update(int(x) for x in rng.choice(S, size=k, replace=False))
    return np.array(sorted(picks), dtype=np.int64)


def serial_agrees(ref_mt, rows_of, lengths, seed, what):
    """The serial oracle on sampled output rows equals the multi-threaded oracle's rows."""
    starts = np.concatenate([[0], np.cumsum(lengths)])
    for s in _sample_segments(lengths, 24, seed):
        a, b = int(starts[s]), int(starts[s + 1])
        one = rows_of(a, b)
        assert np.array_equal(one.view(np.uint32), ref_mt[s:s + 1].view(np.uint32)), f"{what}: row {s}"


def test_c3_powerlaw_graph_full():
    """All 232,965 x 32 outputs of the power-law graph reduction (114,615,892 rows)."""
    c = make_config("c3_powerlaw_graph")
    src, idx, S, L = c["src"], c["index"], c["num_segments"], c["lengths"]
    say("c3 generated")
    s = up(src)
    got = geot.segment_reduce(s, up(idx), S, "sum")
    # per-feature conservation over all 114,615,892 rows (fp64 totals)
    tot_in = s.sum(dim=0, dtype=torch.float64).cpu().numpy()
    tot_out = got.sum(dim=0, dtype=torch.float64).cpu().numpy()
    abs_in = s.abs().sum(dim=0, dtype=torch.float64).cpu().numpy()
    assert np.all(np.abs(tot_in - tot_out) <= 1e-5 * abs_in + 1e-6 * S), "c3 conservation"
    got = got.cpu().numpy()
    del s
    torch.cuda.empty_cache()
    say("c3 oracle")
    m = oracle.mt()
    ref = m.segment_reduce(src, idx, S, "sum")
    compare(got, ref, "sum", m.abs_term_sum(src, idx, S, "sum"), "c3 sum (every element)")
    z = lambda a, b: np.zeros(b - a, dtype=np.int64)
    serial_agrees(ref, lambda a, b: oracle.segment_reduce(src[a:b], z(a, b), 1, "sum"), L, 2, "c3")


def test_c4_spmm_full():
    """All 2,449,029 x 128 outputs of the SpMM workload (61,859,140 weighted edges)."""
    c = make_config("c4_spmm")
    X, col, w, row, R, L = c["X"], c["col"], c["weight"], c["index"], c["num_segments"], c["lengths"]
    say("c4 generated")
    got = geot.gather_scatter(up(X), up(col), up(w), up(row), R, "sum").cpu().numpy()
    torch.cuda.empty_cache()
    say("c4 oracle")
    m = oracle.mt()
    ref = m.gather_scatter(X, col, w, row, R, "sum")
    compare(got, ref, "sum", m.abs_term_sum(X, row, R, "sum", col, w), "c4 sum (every element)")
    z = lambda a, b: np.zeros(b - a, dtype=np.int64)
    serial_agrees(ref, lambda a, b: oracle.gather_scatter(X, col[a:b], w[a:b], z(a, b), 1, "sum"), L, 3, "c4")
