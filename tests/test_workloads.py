"""Input recipes: largest-remainder rescale, index layout and the named workloads' length statistics.

The length statistics pinned here were obtained by an independent simulation
of the same recipes when the workloads were specified (Zipf / lognormal /
Poisson draws with numpy's PCG64), not by this module.
"""
import hashlib

import numpy as np
import pytest

from workloads import (config_lengths, index_from_lengths, lengths_from_index, lr_rescale,
                       make_config, random_gather_problem, random_problem)


def test_lr_rescale_total_and_ties():
    L = lr_rescale([1, 1, 1], 10)
    assert L.sum() == 10 and L.tolist() == [4, 3, 3]  # tie goes to the lower position
    L = lr_rescale([0.5, 0.25, 0.25], 7)
    assert L.tolist() == [3, 2, 2]  # q = [3.5, 1.75, 1.75]: the two largest remainders get +1
    rng = np.random.default_rng(0)
    for _ in range(20):
        w = rng.random(int(rng.integers(1, 500)))
        T = int(rng.integers(0, 10000))
        L = lr_rescale(w, T)
        assert L.sum() == T and L.min() >= 0
        q = T * w / w.sum()
        assert np.all(np.abs(L - q) < 1.0)


def test_index_layout_roundtrip():
    L = np.array([2, 0, 3, 0, 1])
    idx = index_from_lengths(L)
    assert idx.tolist() == [0, 0, 2, 2, 2, 4]
    assert lengths_from_index(idx, 5).tolist() == L.tolist()


@pytest.mark.parametrize("name,S,nnz,mx,p50,empty", [
    ("c1_zipf_small", 4096, 65536, 1221, 2, 205),
    ("c2_poisson_fsweep", 100000, 2000000, 46, 20, 0),
    ("c3_powerlaw_graph", 232965, 114615892, 87791, 241, 0),
    ("c4_spmm", 2449029, 61859140, 3466864, 3, 0),
    ("c5_pointcloud_knn", 1048576, 16777216, 16, 16, 0),
])
def test_named_length_statistics(name, S, nnz, mx, p50, empty):
    _, L = config_lengths(name)
    assert L.size == S and L.sum() == nnz
    assert L.max() == mx and np.median(L) == p50 and (L == 0).sum() == empty


def test_c1_literal_reading_is_degenerate():
    _, L = config_lengths("c1_literal")
    assert L.sum() == 65536 and L.max() > 0.99 * 65536


def test_c1_full_inputs_are_deterministic():
    a = make_config("c1_zipf_small")
    b = make_config("c1_zipf_small")
    assert a["src"].dtype == np.float32 and a["src"].shape == (65536, 32)
    assert np.array_equal(a["src"], b["src"]) and np.array_equal(a["index"], b["index"])
    assert a["src"].min() >= -1.0 and a["src"].max() < 1.0
    h = hashlib.sha256(a["index"].tobytes()).hexdigest()
    assert h == hashlib.sha256(index_from_lengths(a["lengths"]).tobytes()).hexdigest()


def test_random_problems_are_sorted_and_seeded():
    p = random_problem(5, 1000, 37, 3, "zipf", "int", 0.2)
    q = random_problem(5, 1000, 37, 3, "zipf", "int", 0.2)
    assert np.all(np.diff(p["index"]) >= 0) and p["index"].max() < 37
    assert np.array_equal(p["src"], q["src"])
    g = random_gather_problem(6, 500, 20, 30, 4, "lognormal", "normal", True, 0.1)
    assert g["col"].min() >= 0 and g["col"].max() < 30 and g["weight"].shape == (500,)
