"""GPU checks of the autograd layers: forward outputs and every gradient against the oracle on the
same inputs (products through the HIP kernels; sums within 1e-5 * sum|p| + 2^-126)."""
import numpy as np
import pytest

import oracle
from parity import assert_within_tolerance
from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MODELS = {"mitchell": oracle.MITCHELL, "exact_trunc": oracle.EXACT_TRUNC}


def _lut(model, m):
    from paper_2209_04161_amd import binding
    return binding.device_lut(binding.lut_build(m, model))


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


@pytest.mark.parametrize("model", ["mitchell", "exact_trunc"])
def test_am_linear_forward_and_gradients(model):
    from paper_2209_04161_amd import modules
    m = 7
    layer = modules.AMLinear(30, 20, _lut(model, m), m)
    x = torch.from_numpy(W.normal((16, 30), 1.0, 11)).cuda().requires_grad_(True)
    g = torch.from_numpy(W.normal((16, 20), 1.0, 12)).cuda()
    y = layer(x)
    y.backward(g)
    xh, wh, gh = _np(x), _np(layer.weight), _np(g)
    ref, S = oracle.gemm(MODELS[model], m, xh, wh)
    assert_within_tolerance(_np(y) - _np(layer.bias), ref, S, "linear fwd")
    ref, S = oracle.gemm(MODELS[model], m, gh, wh, False, True)
    assert_within_tolerance(_np(x.grad), ref, S, "linear dX")
    ref, S = oracle.gemm(MODELS[model], m, xh, gh, True, False)
    assert_within_tolerance(_np(layer.weight.grad), ref, S, "linear dW")
    np.testing.assert_allclose(_np(layer.bias.grad), gh.sum(0), rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("stride,padding", [(1, "same"), (2, "same"), (1, "valid"), (2, (1, 0, 2, 1))])
def test_am_conv2d_forward_and_gradients(stride, padding):
    from paper_2209_04161_amd import modules
    m = 7
    layer = modules.AMConv2d(5, 9, (3, 4), _lut("mitchell", m), m, stride=stride, padding=padding)
    x = torch.from_numpy(W.normal((3, 11, 13, 5), 1.0, 21)).cuda().requires_grad_(True)
    y = layer(x)
    g = torch.from_numpy(W.normal(tuple(y.shape), 1.0, 22)).cuda()
    y.backward(g)
    pt, pb, pl, pr = layer.pads(11, 13)
    d = dict(n=3, h=11, w=13, c_in=5, c_out=9, kh=3, kw=4, stride_h=stride, stride_w=stride,
             pad_top=pt, pad_bottom=pb, pad_left=pl, pad_right=pr)
    xh, wh, gh = _np(x), _np(layer.weight), _np(g)
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, m, d, xh, wh)
    assert_within_tolerance(_np(y) - _np(layer.bias), ref, S, "conv fwd")
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, m, d, gh, wh)
    assert_within_tolerance(_np(x.grad), ref, S, "conv dX")
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, m, d, xh, gh)
    assert_within_tolerance(_np(layer.weight.grad), ref, S, "conv dW")
    np.testing.assert_allclose(_np(layer.bias.grad), gh.sum((0, 1, 2)), rtol=1e-5, atol=1e-5)


def test_lenet5_training_step_with_the_layers():
    """One SGD step of a LeNet-5 built from the layers (batch 64, exact bfloat16-truncation
    multiplier): the loss is finite, every parameter gets a gradient, and the parameters move."""
    from paper_2209_04161_amd import modules
    m = 7
    lut = _lut("exact_trunc", m)
    F = torch.nn.functional
    torch.manual_seed(0)
    net = torch.nn.ModuleList([modules.AMConv2d(1, 6, 5, lut, m, padding="same"),
                               modules.AMConv2d(6, 16, 5, lut, m),
                               modules.AMLinear(400, 120, lut, m), modules.AMLinear(120, 84, lut, m),
                               modules.AMLinear(84, 10, lut, m)])
    x = torch.from_numpy(W.uniform((64, 28, 28, 1), 0.0, 1.0, 6000)).cuda()
    labels = torch.from_numpy(np.random.default_rng(6010).integers(0, 10, 64)).cuda()

    def pool(t):
        return F.max_pool2d(t.permute(0, 3, 1, 2), 2).permute(0, 2, 3, 1).contiguous()

    h = pool(torch.relu(net[0](x)))
    h = pool(torch.relu(net[1](h))).reshape(64, 400)
    h = torch.relu(net[2](h))
    h = torch.relu(net[3](h))
    loss = F.cross_entropy(net[4](h), labels)
    before = [p.detach().clone() for p in net.parameters()]
    loss.backward()
    assert torch.isfinite(loss).item()
    with torch.no_grad():
        for p in net.parameters():
            assert p.grad is not None and torch.isfinite(p.grad).all().item()
            p -= 0.1 * p.grad
    moved = [not torch.equal(b, p) for b, p in zip(before, net.parameters())]
    assert all(moved)
