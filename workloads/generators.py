"""Seeded input generators for sorted segment reduction workloads.

The five named workloads stand in for the graph, mesh and point-cloud inputs of
the paper's evaluation (Table II graphs and GNN aggregation, Sections II-A/B and
V); the real datasets are not used. Every recipe is deterministic:

* segment lengths come from ``numpy.random.default_rng(seed)`` (PCG64), drawn
  in the order written below;
* large value arrays (src, X, col, weight) are drawn in ``CHUNK``-row pieces,
  piece ``k`` of array stream ``a`` from its own generator
  ``numpy.random.default_rng([seed, a, k])``; the pieces are independent, so
  they are filled by a thread pool and the result does not depend on the
  number of threads;
* fp32 values are drawn directly in fp32;
* segment lengths that must add up to a fixed total are rescaled with the
  largest-remainder rule ``lr_rescale``;
* the index lists segment ids in id order: ``repeat(arange(S), lengths)``.

Nothing here computes a reduction: these are inputs only.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np

CHUNK = 1 << 20

# name -> (seed, description). Sizes follow the workload definitions.
CONFIGS = {
    "c1_zipf_small": (0, "segment_reduce sum, src [65,536 x 32] U(-1,1), 4,096 segments, "
                         "finite Zipf(1.5) lengths, mean 16, 205 empty"),
    "c2_poisson_fsweep": (1, "segment_reduce sum/mean/max, src [2,000,000 x F] N(0,1), "
                             "100,000 segments, Poisson(20) lengths"),
    "c3_powerlaw_graph": (2, "segment_reduce sum, src [114,615,892 x 32] U(-1,1), "
                             "232,965 segments, lognormal(5.5, 1.2) lengths"),
    "c4_spmm": (3, "gather_scatter sum, X [2,449,029 x 128] N(0,1), 61,859,140 edges, "
                   "Zipf(2.0) row lengths, uniform col, w U(0,1)"),
    "c5_pointcloud_knn": (4, "segment_reduce mean/max, src [16,777,216 x 64] N(0,1), "
                             "1,048,576 segments of k=16"),
    "c1_literal": (0, "stress: unbounded Zipf(1.5) lengths rescaled to 65,536 rows"),
}

C2_FEATURES = (1, 2, 3, 4, 8, 15, 16, 32, 64, 128, 256)


# ----------------------------------------------------------------------------
# building blocks
# ----------------------------------------------------------------------------
def lr_rescale(weights, total: int) -> np.ndarray:
    """Largest-remainder rescale of non-negative ``weights`` to integers summing to ``total``.

    q = total * w / sum(w) in fp64; L = floor(q); the ``total - sum(L)`` entries
    with the largest fractional part q - L get one more, ties going to the lower
    position.
    """
    w = np.asarray(weights, dtype=np.float64)
    if w.ndim != 1 or w.size == 0:
        raise ValueError("weights must be a non-empty 1-D array")
    if total < 0:
        raise ValueError("total must be non-negative")
    sw = w.sum()
    if sw <= 0:
        raise ValueError("weights must have a positive sum")
    q = total * (w / sw)
    lengths = np.floor(q).astype(np.int64)
    rest = int(total - lengths.sum())
    if rest < 0 or rest > w.size:
        raise AssertionError("largest-remainder bookkeeping out of range")
    if rest:
        frac = q - lengths
        # primary key: larger fraction first; secondary: lower position first
        order = np.lexsort((np.arange(w.size), -frac))
        lengths[order[:rest]] += 1
    return lengths


def index_from_lengths(lengths) -> np.ndarray:
    """Sorted int64 segment index: segment s repeated lengths[s] times."""
    lengths = np.asarray(lengths, dtype=np.int64)
    return np.repeat(np.arange(lengths.size, dtype=np.int64), lengths)


def lengths_from_index(index, num_segments: int) -> np.ndarray:
    """Segment lengths of a sorted index (inverse of ``index_from_lengths``)."""
    return np.bincount(np.asarray(index, dtype=np.int64), minlength=num_segments).astype(np.int64)


_THREADS = max(1, min(16, os.cpu_count() or 1))


def _fill_chunks(out: np.ndarray, seed: int, stream: int, draw) -> np.ndarray:
    """Fill out[k*CHUNK:(k+1)*CHUNK] with draw(default_rng([seed, stream, k]), view) for every k."""
    n = out.shape[0]
    starts = list(range(0, n, CHUNK))

    def one(k):
        r0 = starts[k]
        draw(np.random.default_rng([seed, stream, k]), out[r0:min(n, r0 + CHUNK)])

    if len(starts) <= 1:
        for k in range(len(starts)):
            one(k)
    else:
        with cf.ThreadPoolExecutor(max_workers=_THREADS) as ex:
            list(ex.map(one, range(len(starts))))
    return out


def _draw_uniform(g, view):
    g.random(out=view, dtype=np.float32)
    view *= np.float32(2.0)
    view -= np.float32(1.0)


def _draw_normal(g, view):
    g.standard_normal(out=view, dtype=np.float32)


def values_uniform(seed: int, stream: int, rows: int, cols: int) -> np.ndarray:
    """U(-1, 1) fp32 as 2*u - 1 with u = random(dtype=float32) (exact in fp32)."""
    return _fill_chunks(np.empty((rows, cols), dtype=np.float32), seed, stream, _draw_uniform)


def values_normal(seed: int, stream: int, rows: int, cols: int) -> np.ndarray:
    """N(0, 1) fp32 drawn with standard_normal(dtype=float32)."""
    return _fill_chunks(np.empty((rows, cols), dtype=np.float32), seed, stream, _draw_normal)


# ----------------------------------------------------------------------------
# named workloads: lengths only (cheap) and full inputs
# ----------------------------------------------------------------------------
def _c1_lengths(rng) -> np.ndarray:
    S, total, n_empty = 4096, 65536, 205
    k = np.arange(1, S + 1, dtype=np.float64)
    p = k ** -1.5
    p /= p.sum()
    z = rng.choice(np.arange(1, S + 1), S, p=p)
    perm = rng.permutation(S)
    empty = np.zeros(S, dtype=bool)
    empty[perm[:n_empty]] = True
    nonempty = np.flatnonzero(~empty)
    lengths = np.zeros(S, dtype=np.int64)
    lengths[nonempty] = 1 + lr_rescale(z[nonempty], total - nonempty.size)
    return lengths


def config_lengths(name: str):
    """(rng positioned after the length draws, lengths) for a named workload."""
    seed = CONFIGS[name][0]
    rng = np.random.default_rng(seed)
    if name == "c1_zipf_small":
        return rng, _c1_lengths(rng)
    if name == "c1_literal":
        return rng, lr_rescale(rng.zipf(1.5, 4096), 65536)
    if name == "c2_poisson_fsweep":
        return rng, lr_rescale(rng.poisson(20, 100_000), 2_000_000)
    if name == "c3_powerlaw_graph":
        return rng, lr_rescale(rng.lognormal(5.5, 1.2, 232_965), 114_615_892)
    if name == "c4_spmm":
        return rng, lr_rescale(rng.zipf(2.0, 2_449_029), 61_859_140)
    if name == "c5_pointcloud_knn":
        return rng, np.full(1_048_576, 16, dtype=np.int64)
    raise KeyError(name)


def make_config(name: str, F: int | None = None) -> dict:
    """Full host inputs of a named workload.

    Returns a dict with ``kind`` ("segment_reduce" or "gather_scatter"), the
    arrays, ``num_segments`` (output rows), ``F`` and ``ops``.
    """
    _, lengths = config_lengths(name)
    S = int(lengths.size)
    nnz = int(lengths.sum())
    index = index_from_lengths(lengths)
    seed = CONFIGS[name][0]
    if name in ("c1_zipf_small", "c1_literal"):
        src = values_uniform(seed, 1, nnz, 32)
        return dict(kind="segment_reduce", src=src, index=index, num_segments=S, F=32,
                    lengths=lengths, ops=("sum",))
    if name == "c2_poisson_fsweep":
        full = values_normal(seed, 1, nnz, 256)
        F = 256 if F is None else int(F)
        if not 1 <= F <= 256:
            raise ValueError("F must be in 1..256 for the F sweep")
        src = full if F == 256 else np.ascontiguousarray(full[:, :F])
        return dict(kind="segment_reduce", src=src, index=index, num_segments=S, F=F,
                    lengths=lengths, ops=("sum", "mean", "max"))
    if name == "c3_powerlaw_graph":
        src = values_uniform(seed, 1, nnz, 32)
        return dict(kind="segment_reduce", src=src, index=index, num_segments=S, F=32,
                    lengths=lengths, ops=("sum",))
    if name == "c4_spmm":
        n_nodes = S
        col = _fill_chunks(np.empty(nnz, dtype=np.int64), seed, 2,
                           lambda g, v: v.__setitem__(slice(None), g.integers(0, n_nodes, v.size, dtype=np.int64)))
        w = _fill_chunks(np.empty(nnz, dtype=np.float32), seed, 3,
                         lambda g, v: g.random(out=v, dtype=np.float32))
        X = values_normal(seed, 1, n_nodes, 128)
        return dict(kind="gather_scatter", X=X, col=col, weight=w, index=index, num_segments=S,
                    F=128, lengths=lengths, ops=("sum",))
    if name == "c5_pointcloud_knn":
        src = values_normal(seed, 1, nnz, 64)
        return dict(kind="segment_reduce", src=src, index=index, num_segments=S, F=64,
                    lengths=lengths, ops=("mean", "max"))
    raise KeyError(name)


# ----------------------------------------------------------------------------
# generic random problems for tests
# ----------------------------------------------------------------------------
def _random_lengths(rng, S: int, nnz: int, dist: str, empty_frac: float) -> np.ndarray:
    if S <= 0:
        raise ValueError("S must be positive")
    if nnz == 0:
        return np.zeros(S, dtype=np.int64)
    if dist == "uniform":
        w = rng.random(S) + 0.05
    elif dist == "zipf":
        w = rng.zipf(1.8, S).astype(np.float64)
    elif dist == "lognormal":
        w = rng.lognormal(2.0, 1.5, S)
    elif dist == "poisson":
        w = rng.poisson(8, S).astype(np.float64) + 0.01
    elif dist == "fixed":
        w = np.ones(S)
    elif dist == "one_heavy":
        w = np.full(S, 1e-3)
        w[rng.integers(0, S)] = 1.0
    else:
        raise ValueError(dist)
    if empty_frac > 0:
        w = w * (rng.random(S) >= empty_frac)
        if w.sum() <= 0:
            w[rng.integers(0, S)] = 1.0
    return lr_rescale(w, nnz)


def _random_values(rng, rows: int, cols: int, values: str) -> np.ndarray:
    if values == "uniform":
        u = rng.random((rows, cols), dtype=np.float32)
        u *= np.float32(2.0)
        u -= np.float32(1.0)
        return u
    if values == "normal":
        return rng.standard_normal((rows, cols), dtype=np.float32)
    if values == "int":      # integers in [-8, 8]: every partial sum is exact in fp32
        return rng.integers(-8, 9, size=(rows, cols)).astype(np.float32)
    if values == "ternary":  # {-1, 0, 1}
        return rng.integers(-1, 2, size=(rows, cols)).astype(np.float32)
    if values == "positive":
        return rng.random((rows, cols), dtype=np.float32)
    if values == "negative":
        return -(rng.random((rows, cols), dtype=np.float32) + np.float32(0.5))
    raise ValueError(values)


def random_problem(seed: int, nnz: int, S: int, F: int, dist: str = "uniform",
                   values: str = "uniform", empty_frac: float = 0.0) -> dict:
    """A random segment_reduce input: src [nnz x F] fp32 and a sorted int64 index over S segments."""
    rng = np.random.default_rng(seed)
    lengths = _random_lengths(rng, S, nnz, dist, empty_frac)
    index = index_from_lengths(lengths)
    src = _random_values(rng, nnz, F, values)
    return dict(src=src, index=index, num_segments=S, F=F, lengths=lengths)


def random_gather_problem(seed: int, nnz: int, R: int, n_x: int, F: int, dist: str = "uniform",
                          values: str = "uniform", weighted: bool = True,
                          empty_frac: float = 0.0) -> dict:
    """A random gather_scatter input: X [n_x x F], col/weight per edge, sorted row ids over R rows."""
    rng = np.random.default_rng(seed)
    lengths = _random_lengths(rng, R, nnz, dist, empty_frac)
    index = index_from_lengths(lengths)
    col = rng.integers(0, n_x, nnz, dtype=np.int64)
    if weighted:
        if values == "int":
            weight = rng.integers(0, 4, nnz).astype(np.float32)
        else:
            weight = rng.random(nnz, dtype=np.float32)
    else:
        weight = None
    X = _random_values(rng, n_x, F, values)
    return dict(X=X, col=col, weight=weight, index=index, num_segments=R, F=F, lengths=lengths)
