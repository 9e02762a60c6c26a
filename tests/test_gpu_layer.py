"""A two-layer graph-convolution training step through the library's autograd wrappers,
against the same model written with plain torch index_add in fp64 on the CPU.

Bar: the loss within 1e-5 of the fp64 loss (relative, at least 1 in scale), and every
parameter gradient within 1e-5 * max|fp64 gradient| elementwise: the library's fp32 bound
(1e-5 relative) taken over the whole tensor. An elementwise relative bound does not apply
here: a weight gradient sums thousands of products of both signs, so its small entries are
the result of cancellation and carry the absolute error of the large ones. For scale, the
same model in fp32 with torch's CPU ops errs by up to 7e-6 of the largest gradient (the GIN
weights), and the library's fp32 step by about 1e-6."""
import numpy as np
import pytest
import torch

import paper_2404_03019_amd.autograd as ga
from workloads import random_gather_problem

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def close(got, ref, what):
    """|got - ref| <= 1e-5 * max|ref| elementwise (see the module docstring)."""
    err = (got.double().cpu() - ref).abs().max().item()
    scale = ref.abs().max().item()
    assert err <= 1e-5 * scale, (what, err, scale)


def gcn_norm(row, col, n):
    deg = np.bincount(row, minlength=n).astype(np.float64)
    return (1.0 / np.sqrt(np.maximum(deg[row], 1) * np.maximum(deg[col], 1))).astype(np.float32)


@pytest.mark.parametrize("reduce,cached,n,nnz,F", [("sum", False, 3000, 40000, 24), ("mean", False, 3000, 40000, 24),
                                                   ("max", False, 3000, 40000, 24), ("sum", True, 3000, 40000, 24),
                                                   ("mean", True, 3000, 40000, 24),
                                                   ("sum", False, 200_000, 1_500_000, 24),
                                                   ("sum", True, 200_000, 1_500_000, 24),
                                                   ("max", False, 200_000, 1_500_000, 24),
                                                   ("sum", True, 3000, 40000, 32), ("mean", False, 3000, 40000, 32),
                                                   ("sum", False, 3000, 40000, 60)])
def test_two_layer_training_step(reduce, cached, n, nnz, F):
    """cached: the layers take a Graph, whose transposed edge list serves the gradient. The
    graphs of 1,500,000 edges take the radix transposition (in the Graph's list and inside
    the gradient calls) and the recording max's gradients from recipients. The first layer
    aggregates before its transform (its input needs no gradient) at 24 -> 32 and 32 -> 32,
    and after it at 60 -> 32."""
    H, C = 32, 5
    q = random_gather_problem(301, nnz, n, n, F, "zipf", "normal", True, 0.0)
    row, col, X = q["index"], q["col"], q["X"]
    w = gcn_norm(row, col, n) if reduce == "sum" else None
    y = np.random.default_rng(302).integers(0, C, n)
    torch.manual_seed(303)
    m = torch.nn.ModuleList([ga.GraphConv(F, H, reduce), ga.GraphConv(H, C, reduce)])
    ref = [torch.nn.Linear(F, H, bias=False), torch.nn.Linear(H, C, bias=False)]
    for a, b in zip(m, ref):
        b.weight.data = a.lin.weight.data.clone()
    m = m.to(DEV)
    ref = [r.double() for r in ref]
    # library path on the GPU
    rt, ct = torch.from_numpy(row).to(DEV), torch.from_numpy(col).to(DEV)
    wt = torch.from_numpy(w).to(DEV) if w is not None else None
    if cached:
        g = ga.Graph(ct, rt, n, wt)
        h = torch.relu(m[0](torch.from_numpy(X).to(DEV), g))
        logits = m[1](h, g)
    else:
        h = torch.relu(m[0](torch.from_numpy(X).to(DEV), ct, rt, n, wt))
        logits = m[1](h, ct, rt, n, wt)
    loss = torch.nn.functional.cross_entropy(logits, torch.from_numpy(y).to(DEV))
    loss.backward()
    # reference: plain torch, fp64, CPU

    def agg(z):
        msg = z[torch.from_numpy(col)]
        if w is not None:
            msg = msg * torch.from_numpy(w).double()[:, None]
        idx = torch.from_numpy(row)[:, None].expand(-1, z.shape[1])
        tname = {"sum": "sum", "mean": "mean", "max": "amax"}[reduce]
        return torch.zeros(n, z.shape[1], dtype=torch.float64).scatter_reduce(0, idx, msg, tname,
                                                                               include_self=False)

    hr = torch.relu(agg(ref[0](torch.from_numpy(X).double())))
    lr = agg(ref[1](hr))
    loss_r = torch.nn.functional.cross_entropy(lr, torch.from_numpy(y))
    loss_r.backward()
    assert abs(loss.item() - loss_r.item()) <= 1e-5 * max(1.0, abs(loss_r.item()))
    for a, b in zip(m, ref):
        close(a.lin.weight.grad, b.weight.grad, reduce)


def test_graph_cache_follows_weight_updates():
    """A Graph rebuilds its transposed list when its weight tensor changes in place."""
    n = 500
    q = random_gather_problem(311, 6000, n, n, 4, "uniform", "normal", True, 0.0)
    ct, rt = torch.from_numpy(q["col"]).to(DEV), torch.from_numpy(q["index"]).to(DEV)
    w = torch.from_numpy(q["weight"]).to(DEV)
    g = ga.Graph(ct, rt, n, w)
    a = g.transposed("sum")[2].clone()
    assert g.transposed("sum")[2] is g.transposed("sum")[2]   # reused while unchanged
    w.mul_(2.0)
    b = g.transposed("sum")[2]
    assert torch.equal(torch.sort(b).values, torch.sort(2.0 * a).values)


@pytest.mark.parametrize("cached", [False, True])
def test_gin_training_step(cached):
    """Two GIN layers (learned eps) on an unweighted graph: loss and every parameter gradient
    against the same model with torch index_add in fp64 on the CPU."""
    n, F, H, C = 2500, 16, 24, 4
    q = random_gather_problem(321, 30000, n, n, F, "zipf", "normal", False, 0.05)
    row, col, X = q["index"], q["col"], q["X"]
    y = np.random.default_rng(322).integers(0, C, n)
    torch.manual_seed(323)
    m = torch.nn.ModuleList([ga.GINConv(F, H, eps=0.1, train_eps=True), ga.GINConv(H, C, train_eps=True)])
    ref = [ga.GINConv(F, H, eps=0.1, train_eps=True), ga.GINConv(H, C, train_eps=True)]
    for a, b in zip(m, ref):
        b.load_state_dict(a.state_dict())
    m = m.to(DEV)
    ref = [r.double() for r in ref]
    rt, ct = torch.from_numpy(row).to(DEV), torch.from_numpy(col).to(DEV)
    xt = torch.from_numpy(X).to(DEV)
    if cached:
        g = ga.Graph(ct, rt, n)
        logits = m[1](torch.relu(m[0](xt, g)), g)
    else:
        logits = m[1](torch.relu(m[0](xt, ct, rt, n)), ct, rt, n)
    loss = torch.nn.functional.cross_entropy(logits, torch.from_numpy(y).to(DEV))
    loss.backward()

    def layer(r, z):
        agg = torch.zeros(n, z.shape[1], dtype=torch.float64).index_add(0, torch.from_numpy(row),
                                                                        z[torch.from_numpy(col)])
        u = (1.0 + r.eps) * z + agg
        return r.lin2(torch.relu(r.lin1(u)))

    lr = layer(ref[1], torch.relu(layer(ref[0], torch.from_numpy(X).double())))
    loss_r = torch.nn.functional.cross_entropy(lr, torch.from_numpy(y))
    loss_r.backward()
    assert abs(loss.item() - loss_r.item()) <= 1e-5 * max(1.0, abs(loss_r.item()))
    for a, b in zip(m, ref):
        for (name, pa), pb in zip(a.named_parameters(), b.parameters()):
            close(pa.grad, pb.grad, (name, cached))
