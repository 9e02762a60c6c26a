"""The order GraphConv gives its aggregation and transform (host logic, CPU): the one that
gathers fewer columns over the forward and backward passes it will run."""
import torch

import paper_2404_03019_amd.autograd as ga


def order(fi, fo, input_grad, reduce="sum", weight_grad=True, grad_enabled=True):
    layer = ga.GraphConv(fi, fo, reduce)
    layer.lin.weight.requires_grad_(weight_grad)
    h = torch.zeros(3, fi, requires_grad=input_grad)
    with torch.set_grad_enabled(grad_enabled):
        return layer._aggregate_first(h)


def test_with_the_input_gradient_the_narrower_side_is_gathered():
    # a gather of the in_features columns each pass if first, else of out_features
    assert order(64, 128, input_grad=True)
    assert not order(128, 128, input_grad=True)
    assert not order(128, 64, input_grad=True)


def test_with_only_the_weight_gradient_aggregation_first_saves_the_backward_gather():
    # first: one forward gather of fi columns; after: fo columns forward and again backward
    assert order(128, 128, input_grad=False)
    assert order(100, 64, input_grad=False)
    assert not order(128, 64, input_grad=False)   # 128 against 2 x 64: the transform first
    assert not order(200, 64, input_grad=False)


def test_without_gradients_only_the_forward_gather_counts():
    assert not order(128, 128, input_grad=False, grad_enabled=False)
    assert order(64, 128, input_grad=False, grad_enabled=False)
    assert not order(128, 128, input_grad=False, weight_grad=False)
