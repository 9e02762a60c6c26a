"""Autograd and a message-passing layer on top of libgeot_hip.

The functions here are torch.autograd.Function wrappers: their forward calls
geot_segment_reduce / geot_gather_scatter and their backward calls
geot_segment_reduce_backward / geot_gather_scatter_backward. The only torch
arithmetic is in the layer's dense transform (a matrix product) and bias, as
in the GNN layers of the paper's end-to-end setting (Section V-F: message and
aggregation fused into one operator, update by a dense layer).
"""
from __future__ import annotations

import torch

from . import geot


# below this many rows (edges) the max records its recipients in the forward (32-bit numbers)
_ARG_ROWS = (1 << 32) - 1


class SegmentReduce(torch.autograd.Function):
    """out = segment_reduce(src, index, num_segments, reduce); differentiable in src.

    Max records each output element's recipient row in the forward (kept instead of src and
    out), so the backward is one pass that writes the gradient."""

    @staticmethod
    def forward(ctx, src, index, num_segments: int, reduce: str = "sum"):
        src = src.contiguous()
        ctx.reduce = reduce
        ctx.src_dtype = src.dtype
        ctx.recorded = reduce == "max" and index.numel() < _ARG_ROWS
        if ctx.recorded:
            out, arg = geot.segment_reduce_max_arg(src, index, num_segments)
            ctx.save_for_backward(index, arg)
        else:
            out = geot.segment_reduce(src, index, num_segments, reduce)
            if reduce == "max":
                ctx.save_for_backward(index, src, out)
            else:
                ctx.save_for_backward(index)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        grad_out = grad_out.contiguous()
        if ctx.recorded:
            index, arg = ctx.saved_tensors
            return geot.segment_reduce_backward_max_arg(grad_out, index, arg, ctx.src_dtype), None, None, None
        if ctx.reduce == "max":
            index, src, out = ctx.saved_tensors
        else:
            (index,) = ctx.saved_tensors
            src = out = None
        # the gradient is written in src's storage type, with src's ids (int64 or int32)
        g = geot.segment_reduce_backward(grad_out, index, ctx.reduce, src, out, dtype=ctx.src_dtype)
        return g, None, None, None


class Graph:
    """A static edge list: edge e goes from source node col[e] to destination
    row[e] (sorted), with an optional weight, over num_nodes destinations and
    num_src sources (default num_nodes).

    The same edges sorted by source (geot_transpose_edges) turn the gradient
    w.r.t. the source features of sum and mean into one forward gather. That
    copy is built on first use and kept while the weights are unchanged (it is
    rebuilt when an in-place update bumps the weight tensor's version).

    The destination ids' length statistics (geot_index_stats, one pass over the ids,
    synchronizing) are taken on the first forward and kept, so the selector of every
    gather over this graph also sees how evenly the edges spread over the rows
    (Section III-C: variance as a feature); they are refreshed when the ids are updated
    in place."""

    # kernel choice for the gather over the transposed list from 2^20 edges: one column tile and
    # 256 rows per row group (the library's tree is fit on forward gathers, whose gathered rows
    # repeat less; SpMM graph, 128 columns: 3.0 ms against 3.3 with the tree's choice)
    TRANSPOSED_GATHER = dict(family="ep", rows=256)

    def __init__(self, col, row, num_nodes: int, weight=None, num_src: int | None = None):
        self.col, self.row, self.weight = col, row, weight
        self.num_nodes = int(num_nodes)
        self.num_src = int(num_src if num_src is not None else num_nodes)
        self._transposed = {}
        self._stats = None
        self.gather_choice = self.TRANSPOSED_GATHER if row.numel() >= (1 << 20) else None

    def stats(self):
        """geot_index_stats of the destination ids (kept until the ids change in place)."""
        version = self.row._version
        if self._stats is None or self._stats[0] != version:
            self._stats = (version, geot.index_stats(self.row.long(), self.num_nodes) if self.row.numel() else None)
        return self._stats[1]

    def transposed(self, reduce: str):
        """(sorted_col, row_t, coef) for `reduce` in sum / mean."""
        version = self.weight._version if self.weight is not None else 0
        hit = self._transposed.get(reduce)
        if hit is None or hit[0] != version:
            w = self.weight.detach() if self.weight is not None else None
            # the transposition takes int64 ids: int32 ones are widened here, once per graph
            hit = (version, geot.transpose_edges(self.col.long(), w, self.row.long(), self.num_src, self.num_nodes,
                                                 reduce))
            self._transposed[reduce] = hit
        return hit[1]


class GatherScatter(torch.autograd.Function):
    """out = gather_scatter(x, col, weight, row, num_rows, reduce); differentiable in x and weight.
    With a Graph of the same edges, the gradient w.r.t. x of sum and mean is one forward
    gather over its cached transposed list."""

    @staticmethod
    def forward(ctx, x, col, weight, row, num_rows: int, reduce: str = "sum", graph=None):
        x = x.contiguous()
        ctx.recorded = reduce == "max" and row.numel() < _ARG_ROWS
        if ctx.recorded:   # max: each element's recipient edge, kept for the backward instead of out
            out, kept = geot.gather_scatter_max_arg(x, col, weight, row, num_rows)
        else:
            out = geot.gather_scatter(x, col, weight, row, num_rows, reduce,
                                      stats=graph.stats() if graph is not None else None)
            kept = out if reduce == "max" else torch.empty(0)
        ctx.reduce = reduce
        ctx.graph = graph
        ctx.save_for_backward(x, col, weight if weight is not None else torch.empty(0), row, kept)
        ctx.has_weight = weight is not None
        return out

    @staticmethod
    def backward(ctx, grad_out):
        x, col, weight, row, out = ctx.saved_tensors
        weight = weight if ctx.has_weight else None
        need_x = ctx.needs_input_grad[0]
        need_w = ctx.has_weight and ctx.needs_input_grad[2]
        grad_out = grad_out.contiguous()   # x keeps its storage type and the ids theirs
        gx = None
        if need_x and ctx.graph is not None and ctx.reduce in ("sum", "mean"):
            sorted_col, row_t, coef = ctx.graph.transposed(ctx.reduce)
            gx = geot.gather_scatter(grad_out, row_t, coef, sorted_col, x.shape[0], "sum",
                                     choice=ctx.graph.gather_choice)
            need_x = False
        if ctx.recorded:   # out holds the recipients the forward recorded
            gx2, gw = geot.gather_scatter_backward_max_arg(x, col, weight, row, grad_out, out,
                                                           need_x=need_x, need_weight=need_w)
        else:
            gx2, gw = geot.gather_scatter_backward(x, col, weight, row, grad_out, ctx.reduce,
                                                   out if ctx.reduce == "max" else None,
                                                   need_x=need_x, need_weight=need_w)
        gx = gx if gx is not None else gx2
        if gx is not None and gx.dtype != x.dtype:   # fp32 gradient of a 16-bit x: rounded once
            gx = gx.to(x.dtype)
        return gx, None, gw, None, None, None, None


def segment_reduce(src, index, num_segments, reduce="sum"):
    """Differentiable segment reduction (gradient w.r.t. src)."""
    return SegmentReduce.apply(src, index, num_segments, reduce)


def gather_scatter(x, col, weight, row, num_rows, reduce="sum", graph=None):
    """Differentiable fused gather-weight-scatter (gradients w.r.t. x and weight); `graph`
    (a Graph of the same edges) caches the transposed list for the gradient w.r.t. x."""
    return GatherScatter.apply(x, col, weight, row, num_rows, reduce, graph)


class RowsLinear(torch.autograd.Function):
    """y = x W^T for x with very many rows (one per graph node).

    The weight gradient gy^T x reduces over all the rows into a small
    (out x in) result. As one product it runs on only as many output tiles as
    that result has (MI355X, 2,449,029 x 128 rows: 3.7 ms); as a batched
    product over 4,096-row chunks, summed, it spreads over the chunks (0.8 ms).
    fp32 only; other types take the one product."""

    CHUNK = 4096

    @staticmethod
    def forward(ctx, x, weight):
        ctx.save_for_backward(x, weight)
        return torch.nn.functional.linear(x, weight)

    @staticmethod
    def backward(ctx, gy):
        x, weight = ctx.saved_tensors
        gy = gy.contiguous()
        gx = gy @ weight if ctx.needs_input_grad[0] else None
        gw = None
        if ctx.needs_input_grad[1]:
            c = RowsLinear.CHUNK
            n, nb = x.shape[0], x.shape[0] // RowsLinear.CHUNK
            if x.dtype != torch.float32 or nb < 2:
                gw = gy.t() @ x
            else:
                x = x.contiguous()
                a = gy[:nb * c].view(nb, c, gy.shape[1]).transpose(1, 2)
                b = x[:nb * c].view(nb, c, x.shape[1])
                gw = torch.bmm(a, b).sum(0)
                if nb * c < n:
                    gw = gw + gy[nb * c:].t() @ x[nb * c:]
        return gx, gw


class GraphConv(torch.nn.Module):
    """h' = aggregate_{e: row[e] = v} w_e * (h W)[col[e]] + b, with the aggregation fused (for sum
    and mean, which are linear, the aggregation runs first where that gathers fewer columns:
    where W widens the features, or where h needs no gradient and W does not narrow them to
    less than half).

    With w_e = 1 / sqrt(deg(row[e]) * deg(col[e])) and self-loops in the edge
    list this is a GCN layer; with reduce="mean" and no weights a GraphSAGE-style
    mean aggregation. The edge list is sorted by row (the destination).
    """

    def __init__(self, in_features: int, out_features: int, reduce: str = "sum", bias: bool = True):
        super().__init__()
        self.lin = torch.nn.Linear(in_features, out_features, bias=False)
        self.bias = torch.nn.Parameter(torch.zeros(out_features)) if bias else None
        self.reduce = reduce

    def _aggregate_first(self, h) -> bool:
        """Sum and mean are linear, so the aggregation may run before or after the transform; the
        order that gathers fewer columns in all is taken. With the gradient w.r.t. h (or none at
        all) both orders gather once per pass, of in_features columns if the aggregation runs
        first, else of out_features. With only the weight's gradient (h a constant input, such
        as the first layer's node features) the aggregation run first needs no gather in the
        backward (the weight gradient is agg(h)^T grad), while the transform run first gathers
        out_features columns again to form it (on the SpMM graph at 128 -> 128 a step saves
        the 2.9 ms gather)."""
        fi, fo = self.lin.in_features, self.lin.out_features
        weight_grad_only = torch.is_grad_enabled() and not h.requires_grad and self.lin.weight.requires_grad
        return fi < 2 * fo if weight_grad_only else fi < fo

    def forward(self, h, col, row=None, num_nodes: int | None = None, weight=None):
        """forward(h, graph) with a Graph, or forward(h, col, row, num_nodes, weight)."""
        graph = None
        if isinstance(col, Graph):
            graph = col
            col, row, num_nodes, weight = graph.col, graph.row, graph.num_nodes, graph.weight
        if self.reduce != "max" and self._aggregate_first(h):
            out = RowsLinear.apply(gather_scatter(h, col, weight, row, num_nodes, self.reduce, graph), self.lin.weight)
        else:
            out = gather_scatter(RowsLinear.apply(h, self.lin.weight), col, weight, row, num_nodes, self.reduce, graph)
        return out + self.bias if self.bias is not None else out


class GINConv(torch.nn.Module):
    """h' = MLP((1 + eps) * h + sum_{e: row[e] = v} h[col[e]]): a graph isomorphism network layer
    whose neighbour sum is one fused gather (no edge weights, no message tensor).

    The edge list is sorted by row (the destination) and sources and destinations are the same
    nodes. The MLP is Linear-ReLU-Linear with the node-count products of RowsLinear; where its
    first layer narrows the features it runs before the sum (the same map, since it is linear and
    the sum unweighted). eps is a learned scalar when train_eps, else a fixed one."""

    def __init__(self, in_features: int, out_features: int, hidden: int | None = None, eps: float = 0.0,
                 train_eps: bool = False):
        super().__init__()
        hidden = hidden or out_features
        self.lin1 = torch.nn.Linear(in_features, hidden)
        self.lin2 = torch.nn.Linear(hidden, out_features)
        e = torch.tensor([float(eps)])
        if train_eps:
            self.eps = torch.nn.Parameter(e)
        else:
            self.register_buffer("eps", e)

    def forward(self, h, col, row=None, num_nodes: int | None = None):
        """forward(h, graph) with a Graph (its weights are not used), or forward(h, col, row, num_nodes)."""
        graph = None
        if isinstance(col, Graph):
            graph = col
            col, row, num_nodes = graph.col, graph.row, graph.num_nodes
            if graph.weight is not None:   # the transposed list would carry the weights
                graph = None
        if h.shape[0] != num_nodes:
            raise ValueError("a GIN layer needs one feature row per node (sources = destinations)")
        if self.lin1.out_features < self.lin1.in_features:
            # the first linear map commutes with the (unweighted) neighbour sum: applied first, the
            # gather and its gradient move hidden columns instead of input ones
            h = RowsLinear.apply(h, self.lin1.weight)
            z = (1.0 + self.eps) * h + gather_scatter(h, col, None, row, num_nodes, "sum", graph) + self.lin1.bias
        else:
            z = (1.0 + self.eps) * h + gather_scatter(h, col, None, row, num_nodes, "sum", graph)
            z = RowsLinear.apply(z, self.lin1.weight) + self.lin1.bias
        z = torch.relu(z)
        return RowsLinear.apply(z, self.lin2.weight) + self.lin2.bias
