"""The caller-workspace forms (geot_segment_reduce_ws, geot_gather_scatter_ws) against
the oracle, on the small named workloads at full size and on random fused inputs.

Each call takes a workspace of exactly the bytes the *_workspace_size query returns
and must equal the oracle (max bit-exact, sum and mean within the bound) and the
default call bit for bit (same kernels, deterministic). A workspace one call fills is
reused by the next, of another shape; a too-small workspace is refused; a _ws call
captured in a HIP graph replays with new inputs.
"""
import numpy as np
import pytest
import torch

import paper_2404_03019_amd as geot
from gpu_util import bits_equal, compare, oracle_gather, oracle_segment, say
from workloads import make_config, random_gather_problem

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
OPS = ("sum", "mean", "max")


def up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def workspace(nbytes):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=DEV)


def check_segment(src, idx, S, ws, what, ops=OPS):
    s, i = up(src), up(idx)
    for op in ops:
        say(f"workspace {what} {op}")
        got = geot.segment_reduce_ws(s, i, S, op, ws)
        ref, terms = oracle_segment(src, idx, S, op)
        compare(got.cpu().numpy(), ref, op, terms, f"{what} {op} (workspace)")
        assert bits_equal(got.cpu().numpy(), geot.segment_reduce(s, i, S, op).cpu().numpy()), f"{what} {op}"


def test_named_workloads_through_one_workspace():
    """C1, the C2 feature sweep at F = 1, 15, 64, 256 and C5, one after another through one
    workspace sized for the largest of them (every call clears the workspace's list counters)."""
    c1 = make_config("c1_zipf_small")
    c2 = make_config("c2_poisson_fsweep", F=256)
    c5 = make_config("c5_pointcloud_knn")
    shapes = [(c1["index"].size, c1["num_segments"], 32), (c5["index"].size, c5["num_segments"], 64)]
    shapes += [(c2["index"].size, c2["num_segments"], F) for F in (1, 15, 64, 256)]
    need = max(geot.workspace_size(n, S, F, op) for n, S, F in shapes for op in OPS)
    ws = workspace(need)
    check_segment(c1["src"], c1["index"], c1["num_segments"], ws, "c1")
    for F in (1, 15, 64, 256):
        check_segment(np.ascontiguousarray(c2["src"][:, :F]), c2["index"], c2["num_segments"], ws, f"c2 F={F}")
    check_segment(c5["src"], c5["index"], c5["num_segments"], ws, "c5")


def test_exact_size_and_too_small():
    c = make_config("c1_zipf_small")
    s, i, S = up(c["src"]), up(c["index"]), c["num_segments"]
    need = geot.workspace_size(i.numel(), S, 32, "sum")
    out = geot.segment_reduce_ws(s, i, S, "sum", workspace(need))
    ref, terms = oracle_segment(c["src"], c["index"], S, "sum")
    compare(out.cpu().numpy(), ref, "sum", terms, "c1 exact workspace")
    with pytest.raises(geot.GeotError, match="needs"):
        geot.segment_reduce_ws(s, i, S, "sum", workspace(4096))
    # nothing to reduce: no workspace at all
    e = geot.segment_reduce_ws(s[:0], i[:0], S, "sum", None)
    assert torch.count_nonzero(e).item() == 0


@pytest.mark.parametrize("weighted", [True, False])
def test_gather_through_workspace(weighted):
    q = random_gather_problem(31, 40_000, 3000, 2500, 48, "zipf", "normal", weighted, 0.1)
    X, col, w, row, R = q["X"], q["col"], q["weight"], q["index"], q["num_segments"]
    choices = [None, dict(family="ep", rows=3), dict(family="ep", lanes=4, rows=9, flags=4), dict(family="sp")]
    need = max(geot.workspace_size(row.size, R, 48, op, gather=True, weighted=weighted, choice=ch)
               for op in OPS for ch in choices)
    ws = workspace(need)
    for op in OPS:
        ref, terms = oracle_gather(X, col, w, row, R, op)
        for ch in choices:
            say(f"workspace gather weighted={weighted} {op} {ch}")
            got = geot.gather_scatter_ws(up(X), up(col), up(w), up(row), R, op, ws, choice=ch)
            compare(got.cpu().numpy(), ref, op, terms, f"gather ws {op} {ch}")


def test_workspace_call_replays_in_a_graph():
    """A _ws call captured once (no warm-up call needed: it allocates nothing) and replayed
    with new inputs, long runs of empty segments included."""
    S, F, n = 200_000, 8, 3000
    rng = np.random.default_rng(74)
    src = torch.empty((n, F), device=DEV)
    idx = torch.empty(n, dtype=torch.int64, device=DEV)
    out = torch.empty((S, F), device=DEV)
    ws = workspace(geot.workspace_size(n, S, F, "sum"))
    st = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=st):
        geot.segment_reduce_ws(src, idx, S, "sum", ws, out=out)
    for k in range(3):
        i = np.sort(rng.integers(0, S, n)).astype(np.int64)
        v = rng.standard_normal((n, F)).astype(np.float32)
        idx.copy_(torch.from_numpy(i))
        src.copy_(torch.from_numpy(v))
        out.fill_(7.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say(f"workspace graph replay {k}")
        ref, terms = oracle_segment(v, i, S, "sum")
        compare(out.cpu().numpy(), ref, "sum", terms, f"ws replay {k}")
