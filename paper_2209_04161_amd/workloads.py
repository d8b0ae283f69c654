"""Seeded synthetic inputs and workload shapes.

This module only draws random numbers and describes shapes; it holds none of the
approximate-multiplier arithmetic.  It is the one module both the HIP path's tests/bench and
the CPU oracle's tests take their inputs from, so that both sides see identical bits.

Distributions follow the layers the paper trains (Sec. "Experiment Setup": LeNet-5 on
MNIST-sized images, ResNet on CIFAR-10 / ImageNet-sized images); the datasets themselves are not
used: inputs are drawn with the same shapes and value ranges.
"""
import math

import numpy as np


def rng(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)


def uniform(shape, lo, hi, seed):
    return rng(seed).uniform(lo, hi, size=shape).astype(np.float32)


def normal(shape, std, seed):
    return (rng(seed).standard_normal(size=shape) * std).astype(np.float32)


def half_normal(shape, seed):
    """|N(0,1)|: post-ReLU-like activations."""
    return np.abs(rng(seed).standard_normal(size=shape)).astype(np.float32)


def he_normal(shape, fan_in, seed):
    return normal(shape, math.sqrt(2.0 / fan_in), seed)


def glorot_uniform(shape, fan_in, fan_out, seed):
    lim = math.sqrt(6.0 / (fan_in + fan_out))
    return uniform(shape, -lim, lim, seed)


def conv_desc(n, h, w, c_in, c_out, kh, kw, stride=1, pad=0, pads=None):
    """Convolution descriptor (NHWC activations, HWIO weights, explicit four-sided padding)."""
    if pads is None:
        pads = (pad, pad, pad, pad)
    pt, pb, pl, pr = pads
    return dict(n=n, h=h, w=w, c_in=c_in, c_out=c_out, kh=kh, kw=kw, stride_h=stride, stride_w=stride,
                pad_top=pt, pad_bottom=pb, pad_left=pl, pad_right=pr)


def conv_out_hw(p):
    oh = (p["h"] + p["pad_top"] + p["pad_bottom"] - p["kh"]) // p["stride_h"] + 1
    ow = (p["w"] + p["pad_left"] + p["pad_right"] - p["kw"]) // p["stride_w"] + 1
    return oh, ow


def conv_macs(p):
    """Nominal multiply count of one pass: N*OH*OW*CO*KH*KW*CI (same for all three passes)."""
    oh, ow = conv_out_hw(p)
    return p["n"] * oh * ow * p["c_out"] * p["kh"] * p["kw"] * p["c_in"]


# --- the workloads (model name, mantissa bits, shapes, seeds) -----------------------------

MITCHELL = "mitchell"
EXACT_TRUNC = "exact_trunc"

# single approx GEMM 64^3, uniform[-1,1], Mitchell M=7
GEMM_SMALL = dict(name="gemm_64", model=MITCHELL, m_bits=7, M=64, N=64, K=64)

# ResNet-style 3x3 conv, batch 128, 64->64 at 32x32, stride 1 pad 1, Mitchell M=7
RESNET_3X3 = dict(name="resnet_3x3_64_32x32_b128", model=MITCHELL, m_bits=7,
                  conv=conv_desc(128, 32, 32, 64, 64, 3, 3, 1, 1))

# ResNet-50-shaped layers, batch 32, Mitchell M=7
RESNET50_LAYERS = [
    dict(name="r50_stem_7x7s2_3to64_224", model=MITCHELL, m_bits=7, conv=conv_desc(32, 224, 224, 3, 64, 7, 7, 2, 3)),
    dict(name="r50_3x3_256to256_14", model=MITCHELL, m_bits=7, conv=conv_desc(32, 14, 14, 256, 256, 3, 3, 1, 1)),
    dict(name="r50_1x1_1024to256_14", model=MITCHELL, m_bits=7, conv=conv_desc(32, 14, 14, 1024, 256, 1, 1, 1, 0)),
]

# large approx GEMM 4096^3, normal(0,1), Mitchell with M=11 (2048-entry table rows) and M=7 (128-entry rows)
GEMM_LARGE = dict(name="gemm_4096", model=MITCHELL, m_bits=11, M=4096, N=4096, K=4096)

# LeNet-5 layer stack, batch 64, 1x28x28 in [0,1], exact bfloat16-truncation multiplier (M=7)
LENET5 = dict(name="lenet5_b64", model=EXACT_TRUNC, m_bits=7, batch=64,
              conv1=conv_desc(64, 28, 28, 1, 6, 5, 5, 1, 2),
              conv2=conv_desc(64, 14, 14, 6, 16, 5, 5, 1, 0),
              fc=[(400, 120), (120, 84), (84, 10)])


def gemm_inputs(M, N, K, dist="uniform", seed=0):
    if dist == "uniform":
        return uniform((M, K), -1.0, 1.0, seed), uniform((K, N), -1.0, 1.0, seed + 1)
    return normal((M, K), 1.0, seed), normal((K, N), 1.0, seed + 1)


def resnet_conv_inputs(p, seed=0, stem=False):
    """x: half-normal (uniform[0,1] image for the stem), w: He-normal, dy: N(0,1)."""
    oh, ow = conv_out_hw(p)
    xshape = (p["n"], p["h"], p["w"], p["c_in"])
    x = uniform(xshape, 0.0, 1.0, seed) if stem else half_normal(xshape, seed)
    w = he_normal((p["kh"], p["kw"], p["c_in"], p["c_out"]), p["kh"] * p["kw"] * p["c_in"], seed + 1)
    dy = normal((p["n"], oh, ow, p["c_out"]), 1.0, seed + 2)
    return x, w, dy
