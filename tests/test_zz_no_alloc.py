"""geot_segment_reduce_noalloc: the entry point that allocates nothing (its temporaries
live in the library's static per-GPU array) equals geot_segment_reduce bit for bit, and
the oracle to the usual bar, on two calls in a row, the second with a smaller input
(the array keeps the first call's contents; the second call clears what must start at
zero). A call too large for the array is refused before any device work.
"""
import numpy as np
import pytest
import torch

import paper_2404_03019_amd as geot
from gpu_util import bits_equal, compare, oracle_segment, say
from workloads import random_problem

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("op", ["sum", "mean", "max"])
def test_noalloc_matches_the_default_call_twice(op):
    # the first input has long runs of empty segments (the list in the array fills) and
    # many block-crossing segments; the second is smaller, with other runs
    first = random_problem(81, 2_000_000, 150_000, 24, "zipf", "normal", 0.4)
    second = random_problem(82, 30_000, 9_000, 24, "lognormal", "normal", 0.3)
    for k, p in enumerate((first, second)):
        src, idx, S = up(p["src"]), up(p["index"]), p["num_segments"]
        out = torch.full((S, 24), 3.0, device=DEV)
        say(f"noalloc {op} call {k} (nnz={idx.numel()})")
        geot.segment_reduce_noalloc(src, idx, S, op, out)
        want = geot.segment_reduce(src, idx, S, op).cpu().numpy()
        got = out.cpu().numpy()
        assert bits_equal(got, want), f"noalloc call {k} {op} differs from geot_segment_reduce"
        ref, terms = oracle_segment(p["src"], p["index"], S, op)
        compare(got, ref, op, terms, f"noalloc call {k} {op}")


def test_noalloc_refuses_inputs_beyond_its_array():
    """Temporary memory beyond the static array: refused on the host, out left untouched."""
    cap = geot.noalloc_scratch_bytes()
    assert cap == 128 << 20
    # 16 M rows of 256 floats: one block per 128 rows (64 lanes a row, 32 rows a group), two
    # partial rows of 256 floats per block, about 266 MiB of partials with aligned arrays
    n, S, F = 16_000_000, 10, 256
    assert geot.workspace_size(n, S, F, "sum") > 2 * cap
    src = torch.zeros((n, F), device=DEV)
    idx = torch.zeros(n, dtype=torch.int64, device=DEV)
    out = torch.full((S, F), 3.0, device=DEV)
    with pytest.raises(geot.GeotError, match="needs"):
        geot.segment_reduce_noalloc(src, idx, S, "sum", out)
    torch.cuda.synchronize()
    assert torch.all(out == 3.0)
