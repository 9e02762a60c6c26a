"""Calls captured once in a HIP graph replay correctly: the library keeps no host-side
state that a replay would freeze (its gap list empties itself on the device).

Each graph is captured after one warm-up call on the capture stream (which
allocates the stream's temporary buffer), then replayed several times with new
input contents of the same shapes written by eager copies between replays; every
replay is checked against the oracle. The inputs have long runs of empty
segments, so every replay fills the gap list.
"""
import numpy as np
import pytest
import torch

import paper_2404_03019_amd as geot
from gpu_util import compare, forward_for_gradient, oracle_gather, oracle_segment, say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("op", ["sum", "mean", "max"])
def test_segment_reduce_replays(op):
    S, F, n = 200_000, 8, 3000
    rng = np.random.default_rng(70)
    src = torch.empty((n, F), device=DEV)
    idx = torch.empty(n, dtype=torch.int64, device=DEV)
    out = torch.empty((S, F), device=DEV)

    def refill():
        i = np.sort(rng.integers(0, S, n)).astype(np.int64)
        v = rng.standard_normal((n, F)).astype(np.float32)
        idx.copy_(torch.from_numpy(i))
        src.copy_(torch.from_numpy(v))
        torch.cuda.synchronize()
        return i, v

    st = torch.cuda.Stream()
    refill()
    with torch.cuda.stream(st):
        geot.segment_reduce(src, idx, S, op, out=out)
    st.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=st):
        geot.segment_reduce(src, idx, S, op, out=out)
    for k in range(4):
        i, v = refill()
        out.fill_(3.0)   # eager work between replays; the replay overwrites every row
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say(f"graph replay {k} segment_reduce {op}")
        ref, terms = oracle_segment(v, i, S, op)
        compare(out.cpu().numpy(), ref, op, terms, f"replay {k} {op}")


def test_gather_scatter_replays():
    R, nx, F, n = 150_000, 2000, 4, 2500
    rng = np.random.default_rng(71)
    X = torch.empty((nx, F), device=DEV)
    col = torch.empty(n, dtype=torch.int64, device=DEV)
    row = torch.empty(n, dtype=torch.int64, device=DEV)
    w = torch.empty(n, device=DEV)
    out = torch.empty((R, F), device=DEV)

    def refill():
        r = np.sort(rng.integers(0, R, n)).astype(np.int64)
        c = rng.integers(0, nx, n).astype(np.int64)
        x = rng.standard_normal((nx, F)).astype(np.float32)
        ww = rng.random(n, dtype=np.float32)
        for t, a in ((row, r), (col, c), (X, x), (w, ww)):
            t.copy_(torch.from_numpy(a))
        torch.cuda.synchronize()
        return x, c, ww, r

    st = torch.cuda.Stream()
    refill()
    with torch.cuda.stream(st):
        geot.gather_scatter(X, col, w, row, R, "max", out=out)
    st.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=st):
        geot.gather_scatter(X, col, w, row, R, "max", out=out)
    for k in range(4):
        x, c, ww, r = refill()
        g.replay()
        torch.cuda.synchronize()
        say(f"graph replay {k} gather_scatter max")
        ref, terms = oracle_gather(x, c, ww, r, R, "max")
        compare(out.cpu().numpy(), ref, "max", terms, f"gather replay {k}")


@pytest.mark.parametrize("op", ["sum", "mean", "max"])
@pytest.mark.parametrize("shape", [(3000, 200_000, 8), (600_000, 2000, 32)], ids=["ids", "offsets"])
def test_segment_backward_replays(op, shape):
    """The segment gradient captured once: with the ids read directly (few rows, long runs of
    empty segments through the gap list), and from 64 MB through the offsets pass and each
    block's first and last ids; max also through its recipient table."""
    import oracle
    n, S, F = shape
    rng = np.random.default_rng(72)
    src = torch.empty((n, F), device=DEV)
    idx = torch.empty(n, dtype=torch.int64, device=DEV)
    g = torch.empty((S, F), device=DEV)
    out = torch.empty((S, F), device=DEV)
    gs = torch.empty((n, F), device=DEV)

    def refill():
        i = np.sort(rng.integers(0, S, n)).astype(np.int64)
        v = rng.integers(-3, 4, (n, F)).astype(np.float32)   # integer values: max ties
        gg = rng.standard_normal((S, F)).astype(np.float32)
        idx.copy_(torch.from_numpy(i))
        src.copy_(torch.from_numpy(v))
        g.copy_(torch.from_numpy(gg))
        if op == "max":
            # the gradient is taken at the oracle's forward result, which the GPU forward must equal
            o = forward_for_gradient(oracle.segment_reduce(v, i, S, "max"),
                                     geot.segment_reduce(src, idx, S, "max"), "segment replay")
            out.copy_(torch.from_numpy(o))
        torch.cuda.synchronize()
        return i, v, gg

    def call():
        geot.segment_reduce_backward(g, idx, op, src if op == "max" else None, out if op == "max" else None,
                                     grad_src=gs)

    st = torch.cuda.Stream()
    refill()
    with torch.cuda.stream(st):
        call()
    st.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=st):
        call()
    for k in range(3):
        i, v, gg = refill()
        gs.fill_(5.0)   # eager work between replays; the replay overwrites every row
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        say(f"graph replay {k} segment backward {op} n={n}")
        ref = oracle.segment_reduce_backward(gg, i, op, v, out.cpu().numpy() if op == "max" else None)
        got = gs.cpu().numpy()
        if op == "mean":
            err = np.abs(got.astype(np.float64) - ref)
            assert np.all(err <= 1e-5 * np.abs(ref) + 1e-6), f"replay {k} mean"
        else:
            assert np.array_equal(got, ref), f"replay {k} {op}"


@pytest.mark.parametrize("shape", [(3000, 2000, 8, 40000), (30000, 300_000, 4, 1_200_000)],
                         ids=["direct", "radix"])
@pytest.mark.parametrize("op", ["sum", "mean", "max"])
def test_gather_backward_replays(op, shape):
    """Both gradients of the fused form captured once (temporaries from the stream-ordered
    pool, the transposition, the recipients for max) and replayed with new inputs: every
    replay within the fp32 bound of the oracle. 40,000 edges take the direct transposition,
    1,200,000 edges over 300,000 columns the radix partition (its counts, cursors and bin
    starts are rewritten by its own kernels on every replay)."""
    import oracle
    R, nx, F, n = shape
    rng = np.random.default_rng(73)
    X = torch.empty((nx, F), device=DEV)
    col = torch.empty(n, dtype=torch.int64, device=DEV)
    row = torch.empty(n, dtype=torch.int64, device=DEV)
    w = torch.empty(n, device=DEV)
    g = torch.empty((R, F), device=DEV)
    out = torch.empty((R, F), device=DEV)

    def refill():
        r = np.sort(rng.integers(0, R, n)).astype(np.int64)
        c = rng.integers(0, nx, n).astype(np.int64)
        x = rng.integers(-3, 4, (nx, F)).astype(np.float32)   # integer values: max ties
        ww = rng.integers(1, 4, n).astype(np.float32)
        gg = rng.standard_normal((R, F)).astype(np.float32)
        for t, a in ((row, r), (col, c), (X, x), (w, ww), (g, gg)):
            t.copy_(torch.from_numpy(a))
        if op == "max":
            o = forward_for_gradient(oracle.gather_scatter(x, c, ww, r, R, "max"),
                                     geot.gather_scatter(X, col, w, row, R, "max"), "gather replay")
            out.copy_(torch.from_numpy(o))
        torch.cuda.synchronize()
        return x, c, ww, r, gg

    def call():
        return geot.gather_scatter_backward(X, col, w, row, g, op, out if op == "max" else None)

    st = torch.cuda.Stream()
    refill()
    with torch.cuda.stream(st):
        call()
    st.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=st):
        gx, gw = call()
    for k in range(3):
        x, c, ww, r, gg = refill()
        graph.replay()
        torch.cuda.synchronize()
        say(f"graph replay {k} gather backward {op} n={n}")
        o = out.cpu().numpy() if op == "max" else None
        rx, rw = oracle.gather_scatter_backward(x, c, ww, r, gg, op, o)
        ax, aw = oracle.gather_scatter_backward(x, c, ww, r, gg, op, o, absolute=True)
        for got, ref, terms, what in ((gx, rx, ax, "grad_X"), (gw, rw, aw, "grad_w")):
            err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
            assert np.all(err <= 1e-5 * terms + 1e-6), f"replay {k} {op} {what}"


def test_two_graphs_of_different_sizes_on_one_stream():
    """A graph captured on a stream keeps the address of the stream's buffer. A later, larger
    call on that stream grows the buffer: the captured one is kept (not freed), so the first
    graph still replays correctly after a second, larger graph was captured on the same
    stream. Both graphs replay alternately with new inputs."""
    rng = np.random.default_rng(75)
    st = torch.cuda.Stream()
    cases = []
    for n, S, F in ((4000, 150_000, 4), (600_000, 90_000, 32)):   # the second needs a larger buffer
        src = torch.empty((n, F), device=DEV)
        idx = torch.empty(n, dtype=torch.int64, device=DEV)
        out = torch.empty((S, F), device=DEV)
        idx.copy_(torch.from_numpy(np.sort(rng.integers(0, S, n)).astype(np.int64)))
        src.copy_(torch.from_numpy(rng.standard_normal((n, F)).astype(np.float32)))
        torch.cuda.synchronize()
        with torch.cuda.stream(st):   # the warm-up call sizes the stream's buffer
            geot.segment_reduce(src, idx, S, "sum", out=out)
        st.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=st):
            geot.segment_reduce(src, idx, S, "sum", out=out)
        cases.append((g, src, idx, out, n, S, F))
    for k in range(2):
        for g, src, idx, out, n, S, F in cases:
            i = np.sort(rng.integers(0, S, n)).astype(np.int64)
            v = rng.standard_normal((n, F)).astype(np.float32)
            idx.copy_(torch.from_numpy(i))
            src.copy_(torch.from_numpy(v))
            out.fill_(5.0)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            say(f"two graphs: replay {k} of the n={n} graph")
            ref, terms = oracle_segment(v, i, S, "sum")
            compare(out.cpu().numpy(), ref, "sum", terms, f"graph n={n} replay {k}")
