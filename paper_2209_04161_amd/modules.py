"""PyTorch autograd layers over the C ABI: approximate-multiplier dense and 2-D convolution layers.

They play the part of the paper's AMDENSE and AMCONV2D layers (Sec. "ApproxTrain", Fig. of the
end-user's perspective): drop-in layers whose every multiply, forward and backward, is the
simulated approximate multiplier, with FP32 accumulation.

* Dense: Y = X W with W stored [in, out] (the Keras layout of the paper's layers);
  dW = X^T dY and dX = dY W^T (Sec. "AMDENSE"; the first operand of each product is the table's
  high index).
* Convolution: NHWC activations, HWIO weights; forward (Algorithm 3), weight gradient and
  preceding-layer gradient (Algorithm 4).

Bias additions are exact FP32 additions and run as ordinary torch ops; no multiply does.  The
layers only marshal tensors into the library's calls (`binding`): every product runs in the HIP
kernels, and a missing library raises.
"""
import torch

from . import binding


def _lut_check(lut, m_bits):
    if not (1 <= int(m_bits) <= 11):
        raise ValueError("m_bits must be in [1, 11]")
    if lut.dtype != torch.int32 or lut.numel() < (1 << (2 * int(m_bits))):
        raise ValueError("lut must be an int32 tensor of 2^(2M) entries (binding.device_lut)")


class _AMLinearFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w, lut, m_bits):
        x = x.contiguous()
        w = w.contiguous()
        ctx.save_for_backward(x, w, lut)
        ctx.m_bits = m_bits
        return binding.approx_gemm(x, w, lut, m_bits)

    @staticmethod
    def backward(ctx, dy):
        x, w, lut = ctx.saved_tensors
        dy = dy.contiguous()
        dx = dw = None
        if ctx.needs_input_grad[0]:
            dx = binding.approx_gemm(dy, w, lut, ctx.m_bits, trans_b=True)   # dY W^T
        if ctx.needs_input_grad[1]:
            dw = binding.approx_gemm(x, dy, lut, ctx.m_bits, trans_a=True)   # X^T dY
        return dx, dw, None, None


def am_linear(x, w, lut, m_bits):
    """Y = X W with approximate products; x [batch, in], w [in, out], float32 CUDA tensors."""
    return _AMLinearFn.apply(x, w, lut, m_bits)


def same_pads(size, k, s):
    """TF "SAME" padding of one spatial dimension: (before, after)."""
    out = (size + s - 1) // s
    total = max((out - 1) * s + k - size, 0)
    return total // 2, total - total // 2


class _AMConv2dFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w, lut, m_bits, stride, pads):
        x = x.contiguous()
        w = w.contiguous()
        n, h, wd, c_in = x.shape
        kh, kw, c_in_w, c_out = w.shape
        if c_in_w != c_in:
            raise ValueError("input channels of x and w differ")
        desc = dict(n=n, h=h, w=wd, c_in=c_in, c_out=c_out, kh=kh, kw=kw, stride_h=stride[0], stride_w=stride[1],
                    pad_top=pads[0], pad_bottom=pads[1], pad_left=pads[2], pad_right=pads[3])
        ctx.save_for_backward(x, w, lut)
        ctx.desc = desc
        ctx.m_bits = m_bits
        return binding.approx_conv2d_fwd(desc, x, w, lut, m_bits)

    @staticmethod
    def backward(ctx, dy):
        x, w, lut = ctx.saved_tensors
        dy = dy.contiguous()
        dx = dw = None
        if ctx.needs_input_grad[0]:
            dx = binding.approx_conv2d_bwd_data(ctx.desc, dy, w, lut, ctx.m_bits)
        if ctx.needs_input_grad[1]:
            dw = binding.approx_conv2d_bwd_weight(ctx.desc, x, dy, lut, ctx.m_bits)
        return dx, dw, None, None, None, None


def am_conv2d(x, w, lut, m_bits, stride=(1, 1), pads=(0, 0, 0, 0)):
    """Convolution with approximate products: x NHWC, w HWIO; pads (top, bottom, left, right)."""
    return _AMConv2dFn.apply(x, w, lut, m_bits, tuple(stride), tuple(pads))


class AMLinear(torch.nn.Module):
    """Dense layer y = x W + b with approximate products (W stored [in, out])."""

    def __init__(self, in_features, out_features, lut, m_bits, bias=True):
        super().__init__()
        _lut_check(lut, m_bits)
        self.m_bits = int(m_bits)
        self.register_buffer("lut", lut, persistent=False)
        self.weight = torch.nn.Parameter(torch.empty(in_features, out_features, device=lut.device))
        self.bias = torch.nn.Parameter(torch.zeros(out_features, device=lut.device)) if bias else None
        limit = (6.0 / (in_features + out_features)) ** 0.5  # Glorot uniform, as Keras initialises
        torch.nn.init.uniform_(self.weight, -limit, limit)

    def forward(self, x):
        y = am_linear(x, self.weight, self.lut, self.m_bits)
        return y + self.bias if self.bias is not None else y


class AMConv2d(torch.nn.Module):
    """2-D convolution with approximate products on NHWC tensors, HWIO weights.

    padding: "valid", "same" (TF's, possibly asymmetric), an int, or (top, bottom, left, right).
    """

    def __init__(self, in_channels, out_channels, kernel_size, lut, m_bits, stride=1, padding="valid", bias=True):
        super().__init__()
        _lut_check(lut, m_bits)
        kh, kw = (kernel_size, kernel_size) if isinstance(kernel_size, int) else tuple(kernel_size)
        self.stride = (stride, stride) if isinstance(stride, int) else tuple(stride)
        self.padding = padding
        self.m_bits = int(m_bits)
        self.register_buffer("lut", lut, persistent=False)
        self.weight = torch.nn.Parameter(torch.empty(kh, kw, in_channels, out_channels, device=lut.device))
        self.bias = torch.nn.Parameter(torch.zeros(out_channels, device=lut.device)) if bias else None
        fan_in, fan_out = kh * kw * in_channels, kh * kw * out_channels
        limit = (6.0 / (fan_in + fan_out)) ** 0.5
        torch.nn.init.uniform_(self.weight, -limit, limit)

    def pads(self, h, w):
        kh, kw = self.weight.shape[0], self.weight.shape[1]
        p = self.padding
        if p == "valid":
            return (0, 0, 0, 0)
        if p == "same":
            return same_pads(h, kh, self.stride[0]) + same_pads(w, kw, self.stride[1])
        if isinstance(p, int):
            return (p, p, p, p)
        return tuple(p)

    def forward(self, x):
        y = am_conv2d(x, self.weight, self.lut, self.m_bits, self.stride, self.pads(x.shape[1], x.shape[2]))
        return y + self.bias if self.bias is not None else y
