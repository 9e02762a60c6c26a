"""The layer's dense transform (autograd.RowsLinear) on the CPU: its value and both
gradients equal torch's own linear layer (exactly for the input gradient and in fp64;
to fp32 summation order for the chunked weight gradient), with and without remainder rows."""
import pytest
import torch

from paper_2404_03019_amd.autograd import RowsLinear


@pytest.mark.parametrize("n", [100, 2 * RowsLinear.CHUNK, 3 * RowsLinear.CHUNK + 17])
@pytest.mark.parametrize("dt", [torch.float32, torch.float64])
def test_rows_linear_matches_torch_linear(n, dt):
    g = torch.Generator().manual_seed(n)
    x = torch.randn(n, 24, dtype=dt, generator=g, requires_grad=True)
    w = torch.randn(10, 24, dtype=dt, generator=g, requires_grad=True)
    y = RowsLinear.apply(x, w)
    gy = torch.randn(y.shape, dtype=dt, generator=g)
    y.backward(gy)
    x2, w2 = x.detach().clone().requires_grad_(True), w.detach().clone().requires_grad_(True)
    y2 = torch.nn.functional.linear(x2, w2)
    y2.backward(gy)
    assert torch.equal(y, y2) and torch.equal(x.grad, x2.grad)
    if dt == torch.float64:
        assert torch.allclose(w.grad, w2.grad, rtol=1e-12, atol=1e-12)
    else:   # chunked sums: fp32 rounding of a different summation order
        assert torch.allclose(w.grad, w2.grad, rtol=1e-5, atol=1e-5 * float(w2.grad.abs().max()))
