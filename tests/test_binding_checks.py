"""The Python binding rejects mismatched shapes before any library call (CPU only).

The C ABI sees raw pointers and sizes, not tensor shapes, so a shape mismatch that
reached it would turn into out-of-bounds device reads or writes. The binding
checks every size first (then that the tensors share one GPU); these tests use
CPU tensors, so reaching the device check proves the shapes passed, and a shape
error proves nothing was launched.
"""
import pytest
import torch

import paper_2404_03019_amd as geot


def f32(*shape):
    return torch.zeros(shape, dtype=torch.float32)


def i64(n):
    return torch.zeros(n, dtype=torch.int64)


def test_forward_shapes():
    with pytest.raises(ValueError, match="one entry per row"):
        geot.segment_reduce(f32(10, 4), i64(9), 3)
    with pytest.raises(ValueError, match="out must have shape"):
        geot.segment_reduce(f32(10, 4), i64(10), 3, out=f32(3, 5))
    with pytest.raises(ValueError, match="on the GPU"):
        geot.segment_reduce(f32(10, 4), i64(10), 3)
    with pytest.raises(ValueError, match="one entry per edge"):
        geot.gather_scatter(f32(5, 4), i64(10), None, i64(9), 3)
    with pytest.raises(ValueError, match="weight must have one entry per edge"):
        geot.gather_scatter(f32(5, 4), i64(10), f32(9), i64(10), 3)
    with pytest.raises(ValueError, match="out must have shape"):
        geot.gather_scatter(f32(5, 4), i64(10), f32(10), i64(10), 3, out=f32(4, 4))


def test_segment_backward_shapes():
    g = f32(3, 4)
    with pytest.raises(ValueError, match="grad_src must have shape"):
        geot.segment_reduce_backward(g, i64(10), "sum", grad_src=f32(10, 5))
    with pytest.raises(ValueError, match="grad_src must have shape"):
        geot.segment_reduce_backward(g, i64(10), "sum", grad_src=f32(11, 4))
    with pytest.raises(ValueError, match="src must have shape"):
        geot.segment_reduce_backward(g, i64(10), "max", src=f32(9, 4), out=f32(3, 4))
    with pytest.raises(ValueError, match="out must have shape"):
        geot.segment_reduce_backward(g, i64(10), "max", src=f32(10, 4), out=f32(2, 4))
    with pytest.raises(ValueError, match="max needs src and out"):
        geot.segment_reduce_backward(g, i64(10), "max", src=f32(10, 4))
    with pytest.raises(ValueError, match="unknown reduce"):
        geot.segment_reduce_backward(g, i64(10), "min")
    with pytest.raises(ValueError, match="on the GPU"):   # every shape agrees
        geot.segment_reduce_backward(g, i64(10), "max", src=f32(10, 4), out=f32(3, 4), grad_src=f32(10, 4))


def test_gather_backward_shapes():
    x, g = f32(6, 4), f32(3, 4)
    with pytest.raises(ValueError, match="x has 5 columns"):
        geot.gather_scatter_backward(f32(6, 5), i64(10), f32(10), i64(10), g)
    with pytest.raises(ValueError, match="one entry per edge"):
        geot.gather_scatter_backward(x, i64(11), f32(10), i64(10), g)
    with pytest.raises(ValueError, match="weight must have shape"):
        geot.gather_scatter_backward(x, i64(10), f32(9), i64(10), g)
    with pytest.raises(ValueError, match="out must have shape"):
        geot.gather_scatter_backward(x, i64(10), f32(10), i64(10), g, "max", out=f32(3, 5))
    with pytest.raises(ValueError, match="max needs out"):
        geot.gather_scatter_backward(x, i64(10), f32(10), i64(10), g, "max")
    with pytest.raises(ValueError, match="on the GPU"):
        geot.gather_scatter_backward(x, i64(10), f32(10), i64(10), g, "max", out=f32(3, 4))
