"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Products are compared bit for bit (element-wise routine; GEMM/conv shapes whose every output
is a single product); sums within 1e-5 * sum|p| + 2^-126 per output.  Small shapes are compared
on every output; the full-size workloads on seeded samples of outputs that the oracle
computes one by one, in the same launch configuration the benchmark times.
"""
import json
import os

import numpy as np
import pytest

import oracle
from cases import mantissa_pairs_grid, outer_operands, random_bits, special_cross
from parity import assert_bits_equal, assert_within_tolerance
from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MODELS = {"mitchell": oracle.MITCHELL, "exact_trunc": oracle.EXACT_TRUNC}


@pytest.fixture(scope="module")
def B():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


_LUTS = {}


def dev_lut(B, model, m):
    key = (model, m)
    if key not in _LUTS:
        _LUTS[key] = B.device_lut(B.lut_build(m, model))
    return _LUTS[key]


def cuda(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


# ------------------------------------------------------------------ single products ------

@pytest.mark.parametrize("model", ["mitchell", "exact_trunc"])
@pytest.mark.parametrize("m", [1, 4, 7])
def test_mul_ew_every_mantissa_pair(B, model, m):
    a, b = mantissa_pairs_grid(m, seed=m)
    sa, sb = special_cross()
    a = np.concatenate([a, sa])
    b = np.concatenate([b, sb])
    got = host(B.approx_mul_ew(cuda(a), cuda(b), dev_lut(B, model, m), m))
    assert_bits_equal(got, oracle.mul(MODELS[model], m, a, b), "mul_ew %s M=%d" % (model, m))


@pytest.mark.parametrize("model", ["mitchell", "exact_trunc"])
@pytest.mark.parametrize("m", [8, 11])
def test_mul_ew_wide_tables_random_bits(B, model, m):
    a = random_bits(1 << 21, 100 + m)
    b = random_bits(1 << 21, 200 + m)
    sa, sb = special_cross()
    a = np.concatenate([a, sa])
    b = np.concatenate([b, sb])
    got = host(B.approx_mul_ew(cuda(a), cuda(b), dev_lut(B, model, m), m))
    assert_bits_equal(got, oracle.mul(MODELS[model], m, a, b), "mul_ew %s M=%d" % (model, m))


@pytest.mark.parametrize("m", [1, 5, 7, 9, 11])
def test_gemm_k1_products_bit_exact(B, m):
    """K = 1: every output is one product (sum starts at -0.0), through the full GEMM kernel."""
    a, b = outer_operands(m, seed=m)
    C = host(B.approx_gemm(cuda(a), cuda(b), dev_lut(B, "mitchell", m), m))
    want = oracle.mul(oracle.MITCHELL, m, np.repeat(a[:, 0], b.shape[1]), np.tile(b[0], a.shape[0]))
    assert_bits_equal(C, want, "gemm K=1 M=%d" % m)


def test_gemm_k1_special_values_bit_exact(B):
    from closed_forms import special_values
    s = special_values()
    a, b = s.reshape(-1, 1), s.reshape(1, -1)
    for m in (7, 11):
        C = host(B.approx_gemm(cuda(a), cuda(b), dev_lut(B, "exact_trunc", m), m))
        want = oracle.mul(oracle.EXACT_TRUNC, m, np.repeat(s, s.size), np.tile(s, s.size))
        assert_bits_equal(C, want, "gemm K=1 specials M=%d" % m)


def _window_vector(m, exps, rng):
    """Every M-bit mantissa field at each exponent and sign, plus +-0 and two denormals (read as
    zeros): finite non-zero values whose exponents keep every product in the normal range, the
    operands the table kernels' bf16 pair path takes."""
    k = np.arange(1 << m, dtype=np.uint32)
    parts = []
    for e in exps:
        for s in (0, 1):
            low = rng.integers(0, 1 << (23 - m), k.size, dtype=np.uint32)
            parts.append((np.uint32(s) << 31) | (np.uint32(e) << 23) | (k << (23 - m)) | low)
    parts.append(np.array([0x00000000, 0x80000000, 0x00000001, 0x80400000], np.uint32))
    return np.concatenate(parts).view(np.float32)


@pytest.mark.parametrize("m", [3, 7])
def test_gemm_k1_window_products_bit_exact(B, m):
    """K = 1 on operands inside the exponent window (Mitchell tables at M <= 7 take the bf16
    pair path there): every product bit for bit, signed zeros included."""
    rng = np.random.default_rng(70 + m)
    a = _window_vector(m, [127, 100, 150], rng).reshape(-1, 1)
    b = _window_vector(m, [127, 110, 140], rng).reshape(1, -1)
    C = host(B.approx_gemm(cuda(a), cuda(b), dev_lut(B, "mitchell", m), m))
    want = oracle.mul(oracle.MITCHELL, m, np.repeat(a[:, 0], b.shape[1]), np.tile(b[0], a.shape[0]))
    assert_bits_equal(C, want, "gemm K=1 window M=%d" % m)


@pytest.mark.parametrize("model,m", [("mitchell", 7), ("exact_trunc", 7), ("exact_trunc", 5)])
def test_gemm_large_tile_k1_window_products_bit_exact(B, model, m):
    """K = 1 at 4096 x 4096 inside the exponent window, a shape that takes the 8-wave 8-column
    tile: its bf16 pair path (Mitchell: 1-byte table) and its hi/lo path (exact truncation: 2-byte
    table; at M = 5 its rows hold 32 entries), every product bit for bit, signed zeros included."""
    rng = np.random.default_rng(91 + m)
    a = np.resize(_window_vector(m, list(range(100, 148, 3)), rng)[::-1], 4096).reshape(-1, 1)
    b = np.resize(_window_vector(m, list(range(110, 142, 2)), rng)[::-1], 4096).reshape(1, -1)
    C = host(B.approx_gemm(cuda(a), cuda(b), dev_lut(B, model, m), m))
    want = oracle.mul(MODELS[model], m, np.repeat(a[:, 0], b.shape[1]), np.tile(b[0], a.shape[0]))
    assert_bits_equal(C, want, "gemm 4096 x 4096 K=1 window %s" % model)


def test_gemm_large_tile_two_byte_table_sums(B):
    """The hi/lo path's sums (exact-truncation table, normal(0,1) operands) on the 8-wave
    8-column tile, every output against the oracle."""
    m = 7
    A, Bm = W.gemm_inputs(4096, 2048, 8, "normal", seed=5100)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "exact_trunc", m), m))
    ref, S = oracle.gemm(oracle.EXACT_TRUNC, m, A, Bm)
    assert_within_tolerance(C, ref, S, "gemm 4096 x 2048 x 8 exact_trunc")


@pytest.mark.parametrize("k", [2, 3, 41, 200])
def test_gemm_zero_sums_keep_their_sign(B, k):
    """Sums of signed zeros: -0 exactly when every product is -0 (the sum starts at -0.0), +0
    otherwise; the bf16 pair path rebuilds the sign of such sums in a second pass."""
    rng = np.random.default_rng(k)
    m = 7
    A = W.normal((70, k), 1.0, 80 + k)
    Bm = W.normal((k, 24), 1.0, 90 + k)
    A[:10] = 0.0                     # rows of +0
    A[10:14] = -0.0                  # rows of -0
    A[14, ::2] = 0.0                 # mixed row: zeros and values
    Bm[:, :6] = -np.abs(Bm[:, :6])   # columns of negative values
    Bm[:, 6:9] = np.abs(Bm[:, 6:9])  # columns of positive values
    Bm[:, 9] = -0.0
    Bm[rng.integers(0, k), 10] = 0.0
    Bm[:, 11] = -np.abs(Bm[:, 11])   # -0 products with the +0 rows up to the last step only
    Bm[-1, 11] = abs(Bm[-1, 11])
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "mitchell", m), m))
    ref, S = oracle.gemm(oracle.MITCHELL, m, A, Bm)
    zero = ref == 0.0
    assert zero.sum() >= 14 * 24
    assert_bits_equal(C[zero], ref[zero].astype(np.float32), "zero sums K=%d" % k)
    assert_within_tolerance(C, ref, S, "gemm zero rows K=%d" % k)


def test_conv_zero_sums_keep_their_sign(B):
    """Exactly-zero conv outputs carry the sign rule of R10 through the record layout and the
    bf16 path's sign pass, in all three passes.  No padded taps (the GPU's zero border would add
    signed zeros there, which the oracle skips): pad 0, and a 1x1 kernel for backward-data."""
    m = 7
    lut = dev_lut(B, "mitchell", m)

    def check(got, ref, S, what):
        zero = ref == 0.0
        assert zero.sum() > 0, what
        assert_bits_equal(got[zero], ref[zero].astype(np.float32), what + " zero outputs")
        assert_within_tolerance(got, ref, S, what)

    p = W.conv_desc(2, 6, 9, 7, 12, 3, 3, 1, 0)
    x = W.normal((2, 6, 9, 7), 1.0, 71)
    w = W.normal((3, 3, 7, 12), 1.0, 72)
    x[0] = 0.0                       # first image: +0 ...
    x[0, 2:4, 3:6, :] = -0.0         # ... with a block of -0
    w[..., :4] = -np.abs(w[..., :4])  # negative, positive and -0 output channels
    w[..., 4:8] = np.abs(w[..., 4:8])
    w[..., 8] = -0.0
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, m, p, x, w)
    check(y, ref, S, "fwd")

    p = W.conv_desc(2, 5, 7, 13, 9, 1, 1, 1, 0)
    dy = W.normal((2, 5, 7, 9), 1.0, 73)
    w = W.normal((1, 1, 13, 9), 1.0, 74)
    dy[1] = 0.0
    dy[1, :, :3, :] = -0.0
    w[0, 0, :5, :] = -np.abs(w[0, 0, :5, :])
    w[0, 0, 5:9, :] = np.abs(w[0, 0, 5:9, :])
    w[0, 0, 9, :] = -0.0
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, m, p, dy, w)
    check(dx, ref, S, "bwd_data")

    # few input channels and a 1 x 3 kernel: the pass runs unfolded along w and folds the sums
    # back (no padded taps either way)
    p = W.conv_desc(2, 5, 9, 3, 6, 1, 3, 1, 0)
    dy = W.normal((2, 5, 7, 6), 1.0, 77)
    w = W.normal((1, 3, 3, 6), 1.0, 78)
    dy[1] = 0.0
    dy[1, :, :2, :] = -0.0
    w[0, :, 0, :] = -np.abs(w[0, :, 0, :])
    w[0, :, 1, :] = np.abs(w[0, :, 1, :])
    w[0, 1:, 2, :] = -0.0
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, m, p, dy, w)
    check(dx, ref, S, "bwd_data unfolded")

    p = W.conv_desc(2, 6, 9, 5, 11, 3, 3, 1, 0)
    x = W.normal((2, 6, 9, 5), 1.0, 75)
    dy = W.normal((2, 4, 7, 11), 1.0, 76)
    x[..., 0] = 0.0                  # input channel 0: +0, channel 1: -0
    x[..., 1] = -0.0
    dy[..., :4] = -np.abs(dy[..., :4])
    dy[..., 4:8] = np.abs(dy[..., 4:8])
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, m))
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, m, p, x, dy)
    check(dw, ref, S, "bwd_weight")

    # forward taps in 2 channel chunks (32 channels): the sign pass walks every chunk
    p = W.conv_desc(1, 5, 6, 32, 10, 3, 3, 1, 0)
    x = W.normal((1, 5, 6, 32), 1.0, 79)
    w = W.normal((3, 3, 32, 10), 1.0, 80)
    x[0, :, :4, :] = -0.0            # windows of output columns 0, 1 see -0 only
    w[..., :4] = np.abs(w[..., :4])
    w[..., 4:8] = -np.abs(w[..., 4:8])
    w[..., 8] = -0.0
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, m, p, x, w)
    check(y, ref, S, "fwd in channel chunks")

    # backward-data taps in 4 output-channel chunks (64 channels), 1 x 1 kernel
    p = W.conv_desc(1, 4, 5, 6, 64, 1, 1, 1, 0)
    dy = W.normal((1, 4, 5, 64), 1.0, 81)
    w = W.normal((1, 1, 6, 64), 1.0, 82)
    dy[0, :2] = -0.0
    dy[0, 2, :2] = 0.0
    w[0, 0, :2, :] = np.abs(w[0, 0, :2, :])
    w[0, 0, 2:4, :] = -np.abs(w[0, 0, 2:4, :])
    w[0, 0, 4, :] = -0.0
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, m, p, dy, w)
    check(dx, ref, S, "bwd_data in channel chunks")
    assert np.signbit(ref[0, 0, 0, 0]) and not np.signbit(ref[0, 2, 0, 0])  # both zero signs occur


def test_conv_unfolded_padding_channel_is_neutral(B):
    """The w-unfolded forward pass pads an odd kw * c to whole channel pairs; the padding channel
    must add nothing, not even a zero sign, also in zero-padded image rows.  With x = +0 and
    negative weights every product, padded taps included, is -0, so every output is -0."""
    m = 7
    lut = dev_lut(B, "mitchell", m)
    p = W.conv_desc(2, 5, 7, 3, 4, 3, 3, 1, pads=(2, 1, 1, 1))   # kw * c = 9: one padding channel
    x = np.zeros((2, 5, 7, 3), dtype=np.float32)
    w = -np.abs(W.normal((3, 3, 3, 4), 1.0, 79))
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, m, p, x, w)
    assert (ref == 0.0).all() and np.signbit(ref).all()
    assert_bits_equal(y, ref.astype(np.float32), "unfolded forward, zero products")


def test_conv_single_product_shapes_bit_exact(B):
    """1x1 conv with one input channel (fwd), one output position (bwd_weight) and one output
    channel with a 1x1 kernel (bwd_data): every output is a single product."""
    m = 7
    lut = dev_lut(B, "mitchell", m)
    p = W.conv_desc(2, 5, 7, 1, 70, 1, 1, 1, 0)
    x = random_bits(2 * 5 * 7, 1).reshape(2, 5, 7, 1)
    w = random_bits(70, 2).reshape(1, 1, 1, 70)
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    want = oracle.mul(oracle.MITCHELL, m, np.repeat(x.reshape(-1), 70), np.tile(w.reshape(-1), 70))
    assert_bits_equal(y, want, "conv fwd 1x1 ci=1")
    # bwd_weight with a single output position: dw[kh,kw,ci,co] = amul(x[0,kh,kw,ci], dy[0,0,0,co])
    p = W.conv_desc(1, 3, 3, 5, 66, 3, 3, 1, 0)
    x = random_bits(45, 3).reshape(1, 3, 3, 5)
    dy = random_bits(66, 4).reshape(1, 1, 1, 66)
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, m))
    want = oracle.mul(oracle.MITCHELL, m, np.repeat(x.reshape(-1), 66), np.tile(dy.reshape(-1), 45))
    assert_bits_equal(dw, want, "conv bwd_weight single position")
    # bwd_data with 1x1 kernel, c_out = 1: dx[n,h,w,ci] = amul(dy[n,h,w,0], w[0,0,ci,0])
    p = W.conv_desc(2, 4, 6, 67, 1, 1, 1, 1, 0)
    dy = random_bits(48, 5).reshape(2, 4, 6, 1)
    w = random_bits(67, 6).reshape(1, 1, 67, 1)
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    want = oracle.mul(oracle.MITCHELL, m, np.repeat(dy.reshape(-1), 67), np.tile(w.reshape(-1), 48))
    assert_bits_equal(dx, want, "conv bwd_data 1x1 co=1")


# ------------------------------------------------------------------ GEMM sums ------------

GEMM_SHAPES = [(64, 64, 64), (1, 1, 1), (3, 17, 63), (65, 1000, 17), (130, 7, 300), (257, 129, 513),
               (700, 20, 33), (64, 16, 8192)]


@pytest.mark.parametrize("shape", GEMM_SHAPES)
@pytest.mark.parametrize("model,m", [("mitchell", 7), ("mitchell", 11), ("exact_trunc", 11)])
def test_gemm_matches_oracle(B, shape, model, m):
    """M = 11: Mitchell's table is sum-indexed (read from one g array), the exact truncated
    product's is not (rows staged per column and step)."""
    M, N, K = shape
    A = W.uniform((M, K), -1, 1, 1000 + M)
    Bm = W.uniform((K, N), -1, 1, 2000 + N)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, model, m), m))
    ref, S = oracle.gemm(MODELS[model], m, A, Bm)
    assert_within_tolerance(C, ref, S, "gemm %s %s M=%d" % (shape, model, m))


@pytest.mark.parametrize("ta,tb", [(True, False), (False, True), (True, True)])
@pytest.mark.parametrize("m", [3, 7, 8])
def test_gemm_transposes(B, ta, tb, m):
    M, N, K = 77, 45, 91
    A = W.normal((K, M) if ta else (M, K), 1.0, 31)
    Bm = W.normal((N, K) if tb else (K, N), 1.0, 32)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "exact_trunc", m), m, trans_a=ta, trans_b=tb))
    ref, S = oracle.gemm(oracle.EXACT_TRUNC, m, A, Bm, ta, tb)
    assert_within_tolerance(C, ref, S, "gemm trans %s %s" % (ta, tb))


def test_gemm_leading_dimension_canary_and_k0(B):
    """ldc > n: the padding columns of C keep their sentinel; k = 0 writes -0.0."""
    m = 7
    A = W.uniform((33, 20), -1, 1, 41)
    Bm = W.uniform((20, 10), -1, 1, 42)
    buf = torch.full((33, 17), 12345.0, dtype=torch.float32, device="cuda")
    out = buf[:, :10]
    B.lib()
    lut = dev_lut(B, "mitchell", m)
    B.approx_gemm(cuda(A), cuda(Bm), lut, m, out=out)
    got = host(buf)
    assert np.all(got[:, 10:] == 12345.0)
    ref, S = oracle.gemm(oracle.MITCHELL, m, A, Bm)
    assert_within_tolerance(got[:, :10], ref, S, "gemm ldc")
    z = B.approx_gemm(cuda(np.zeros((5, 0), np.float32)), cuda(np.zeros((0, 3), np.float32)), lut, m)
    assert np.all(host(z).view(np.uint32) == 0x80000000)


def test_gemm_deterministic(B):
    A = W.normal((300, 500), 1.0, 51)
    Bm = W.normal((500, 200), 1.0, 52)
    lut = dev_lut(B, "mitchell", 7)
    c1 = host(B.approx_gemm(cuda(A), cuda(Bm), lut, 7))
    c2 = host(B.approx_gemm(cuda(A), cuda(Bm), lut, 7))
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))


# ------------------------------------------------------------------ convolution ----------

CONV_CASES = [
    W.conv_desc(2, 7, 6, 3, 4, 3, 3, 1, 1),
    W.conv_desc(2, 9, 8, 2, 3, 3, 3, 2, 1),
    W.conv_desc(1, 11, 10, 3, 2, 5, 5, 2, pads=(2, 1, 0, 3)),
    W.conv_desc(3, 5, 5, 4, 2, 1, 1, 1, 0),
    W.conv_desc(2, 8, 9, 2, 3, 7, 7, 2, 3),
    W.conv_desc(1, 6, 6, 1, 2, 2, 3, 3, pads=(1, 0, 2, 1)),
    W.conv_desc(2, 13, 12, 20, 70, 3, 3, 1, 1),
    W.conv_desc(3, 10, 10, 65, 17, 3, 3, 2, 1),
    W.conv_desc(2, 9, 9, 16, 33, 1, 1, 2, 0),
    W.conv_desc(2, 28, 28, 1, 6, 5, 5, 1, 2),
    W.conv_desc(1, 9, 9, 3, 2, 1, 1, 2, 0),
    W.conv_desc(1, 16, 16, 3, 20, 7, 7, 2, 3),
    W.conv_desc(1, 6, 7, 2, 2, 3, 3, 3, pads=(0, 2, 1, 0)),
    W.conv_desc(2, 5, 4, 2, 3, 4, 4, 2, pads=(3, 3, 3, 3)),
    W.conv_desc(2, 5, 5, 300, 20, 3, 3, 1, 1),
    W.conv_desc(2, 6, 6, 24, 200, 3, 3, 2, 1),
    W.conv_desc(1, 3, 70, 130, 9, 3, 3, 1, 1),   # x rows pass through LDS in two channel chunks; backward
                                                 # weight: rows of 9100 elements, beyond its LDS row stage
    W.conv_desc(1, 3, 70, 9, 130, 3, 3, 1, 1),   # dy rows (backward data) likewise
    W.conv_desc(1, 3, 1100, 8, 5, 3, 3, 1, 1),   # few channels, but a row too long to unfold along w
    W.conv_desc(2, 7, 9, 5, 6, 1, 4, 1, 3, pads=(0, 0, 2, 1)),  # 1 x 4 kernel, unfolded into 20 channels
    dict(W.conv_desc(2, 8, 11, 3, 4, 3, 5, 1, 2), stride_w=2),   # unfolded with different strides
    W.conv_desc(2, 9, 7, 32, 10, 3, 3, 1, 1),    # forward taps in 2 channel chunks
    W.conv_desc(1, 6, 5, 64, 12, 3, 2, 2, pads=(1, 0, 0, 1)),   # 4 chunks, stride 2, asymmetric pads
    W.conv_desc(1, 3, 3, 256, 8, 3, 3, 1, 1),    # 4 chunks of 64 with a split reduction (9 rows)
    W.conv_desc(2, 7, 6, 10, 32, 3, 3, 1, 1),    # backward-data taps in 2 output-channel chunks
    W.conv_desc(1, 6, 5, 12, 64, 3, 2, 2, pads=(1, 0, 0, 1)),   # 4 chunks over stride phases
    W.conv_desc(1, 4, 4, 8, 256, 3, 3, 1, 1),    # 8 chunks of 32 with a split reduction (16 rows)
    W.conv_desc(2, 6, 9, 3, 32, 3, 3, 1, 1),     # unfolded backward data in 2 chunks
]


def _conv_inputs(p, seed):
    oh, ow = W.conv_out_hw(p)
    x = W.uniform((p["n"], p["h"], p["w"], p["c_in"]), -1, 1, seed)
    w = W.uniform((p["kh"], p["kw"], p["c_in"], p["c_out"]), -1, 1, seed + 1)
    dy = W.uniform((p["n"], oh, ow, p["c_out"]), -1, 1, seed + 2)
    return x, w, dy


@pytest.mark.parametrize("ci", range(len(CONV_CASES)))
@pytest.mark.parametrize("m", [7, 10])
def test_conv_passes_match_oracle(B, ci, m):
    p = CONV_CASES[ci]
    x, w, dy = _conv_inputs(p, 300 + ci)
    lut = dev_lut(B, "mitchell", m)
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, m, p, x, w)
    assert_within_tolerance(y, ref, S, "fwd %d" % ci)
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, m, p, dy, w)
    assert_within_tolerance(dx, ref, S, "bwd_data %d" % ci)
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, m))
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, m, p, x, dy)
    assert_within_tolerance(dw, ref, S, "bwd_weight %d" % ci)


def _random_conv_cases(count, seed):
    """Seeded random conv shapes: kernels 1..7, strides 1..3 (different in h and w), asymmetric pads
    0..3, channel counts on both sides of the w-unfolding thresholds, M in {3, 5, 7, 9}, both models."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        kh, kw = int(rng.integers(1, 8)), int(rng.integers(1, 8))
        sh, sw = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        pads = [int(rng.integers(0, 4)) for _ in range(4)]
        h, w = int(rng.integers(1, 14)), int(rng.integers(1, 14))
        if h + pads[0] + pads[1] < kh or w + pads[2] + pads[3] < kw:
            continue
        p = dict(n=int(rng.integers(1, 4)), h=h, w=w, c_in=int(rng.choice([1, 2, 3, 5, 7, 9, 15, 17, 33])),
                 c_out=int(rng.choice([1, 2, 3, 5, 8, 9, 16, 20, 40])), kh=kh, kw=kw, stride_h=sh, stride_w=sw,
                 pad_top=pads[0], pad_bottom=pads[1], pad_left=pads[2], pad_right=pads[3])
        cases.append((p, str(rng.choice(["mitchell", "exact_trunc"])), int(rng.choice([3, 5, 7, 9]))))
    return cases


RANDOM_CONV_CASES = _random_conv_cases(40, 20261202)


@pytest.mark.parametrize("ci", range(len(RANDOM_CONV_CASES)))
def test_conv_random_shapes_match_oracle(B, ci):
    p, model, m = RANDOM_CONV_CASES[ci]
    x, w, dy = _conv_inputs(p, 5000 + 3 * ci)
    lut = dev_lut(B, model, m)
    om = MODELS[model]
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    ref, S = oracle.conv2d_fwd(om, m, p, x, w)
    assert_within_tolerance(y, ref, S, "fwd %s" % p)
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    ref, S = oracle.conv2d_bwd_data(om, m, p, dy, w)
    assert_within_tolerance(dx, ref, S, "bwd_data %s" % p)
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, m))
    ref, S = oracle.conv2d_bwd_weight(om, m, p, x, dy)
    assert_within_tolerance(dw, ref, S, "bwd_weight %s" % p)


def test_operand_order_with_asymmetric_table(B):
    """A table from an asymmetric model (first operand truncated to M bits, second to M-1) pins
    the first operand of GEMM and of every convolution pass."""
    m = 5

    def asym(a, b):
        ua = np.float32(a).view(np.uint32) & np.uint32((0xFFFFFFFF << (23 - m)) & 0xFFFFFFFF)
        ub = np.float32(b).view(np.uint32) & np.uint32((0xFFFFFFFF << (24 - m)) & 0xFFFFFFFF)
        return float(ua.view(np.float32) * ub.view(np.float32))

    lut = B.device_lut(B.lut_build(m, asym))
    A = W.uniform((70, 40), -2, 2, 61)
    Bm = W.uniform((40, 30), -2, 2, 62)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), lut, m))
    ref, S = oracle.gemm(oracle.ASYM, m, A, Bm)
    assert_within_tolerance(C, ref, S, "gemm asym")
    p = CONV_CASES[1]
    x, w, dy = _conv_inputs(p, 63)
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
    ref, S = oracle.conv2d_fwd(oracle.ASYM, m, p, x, w)
    assert_within_tolerance(y, ref, S, "fwd asym")
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
    ref, S = oracle.conv2d_bwd_data(oracle.ASYM, m, p, dy, w)
    assert_within_tolerance(dx, ref, S, "bwd_data asym")
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, m))
    ref, S = oracle.conv2d_bwd_weight(oracle.ASYM, m, p, x, dy)
    assert_within_tolerance(dw, ref, S, "bwd_weight asym")


# ------------------------------------------------------------------ full-size workloads --

def _sample(total, count, seed):
    rng = np.random.default_rng(seed)
    idx = rng.choice(total, size=min(count, total), replace=False)
    return np.sort(np.concatenate([idx, [0, total - 1]]).astype(np.int64))


# Largest |gpu - oracle| / sum|p| of every full-size check, written as JSON to the path in
# AMSIM_PARITY_REPORT (when set) at the end of the module.
MAX_REL = {}


@pytest.fixture(scope="module", autouse=True)
def _parity_report():
    yield
    path = os.environ.get("AMSIM_PARITY_REPORT")
    if path and MAX_REL:
        with open(path, "w") as f:
            json.dump(MAX_REL, f, indent=1, sort_keys=True)


def _record(name, got, ref, S, what):
    rel = assert_within_tolerance(got, ref, S, what)
    MAX_REL[name] = {"max_err_over_sum_abs_products": rel, "outputs_compared": int(np.size(ref))}
    return rel


def _check_conv_full(B, p, m, seed, stem=False, samples=(2048, 2048, 512), relu=False, model="mitchell", name=None):
    """The three passes at full size.  samples: outputs compared per pass (seeded, plus the first
    and last), or None for every output."""
    x, w, dy = W.resnet_conv_inputs(p, seed=seed, stem=stem)
    if relu:  # post-ReLU activations: about half exact zeros
        x = np.maximum(W.normal(x.shape, 1.0, seed + 7), 0.0).astype(np.float32)
    lut = dev_lut(B, model, m)
    om = MODELS[model]
    name = name or "conv seed %d" % seed
    xd, wd, dyd = cuda(x), cuda(w), cuda(dy)

    def pick(out, i, s):
        return None if samples is None else _sample(out.size, samples[i], s)

    y = host(B.approx_conv2d_fwd(p, xd, wd, lut, m)).reshape(-1)
    idx = pick(y, 0, seed)
    ref, S = oracle.conv2d_fwd(om, m, p, x, w, idx=idx)
    _record(name + " fwd", y if idx is None else y[idx], ref, S, "fwd")
    dx = host(B.approx_conv2d_bwd_data(p, dyd, wd, lut, m)).reshape(-1)
    idx = pick(dx, 1, seed + 1)
    ref, S = oracle.conv2d_bwd_data(om, m, p, dy, w, idx=idx)
    _record(name + " bwd_data", dx if idx is None else dx[idx], ref, S, "bwd_data")
    dw = host(B.approx_conv2d_bwd_weight(p, xd, dyd, lut, m)).reshape(-1)
    idx = pick(dw, 2, seed + 2)
    ref, S = oracle.conv2d_bwd_weight(om, m, p, x, dy, idx=idx)
    _record(name + " bwd_weight", dw if idx is None else dw[idx], ref, S, "bwd_weight")
    return y


@pytest.mark.parametrize("pass_name", ["fwd", "bwd_data", "bwd_weight"])
def test_resnet_3x3_conv_full_size(B, pass_name):
    """ResNet 3x3 (batch 128, 64 -> 64 at 32x32) with the benchmark's inputs and launch: every
    output of the pass against the oracle (about 30 s of oracle time per pass on 16 threads)."""
    cfg = W.RESNET_3X3
    p, m = cfg["conv"], cfg["m_bits"]
    x, w, dy = W.resnet_conv_inputs(p, seed=3000)
    lut = dev_lut(B, "mitchell", m)
    if pass_name == "fwd":
        got = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, m))
        ref, S = oracle.conv2d_fwd(oracle.MITCHELL, m, p, x, w)
    elif pass_name == "bwd_data":
        got = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, m))
        ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, m, p, dy, w)
    else:
        got = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, m))
        ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, m, p, x, dy)
    _record("resnet 3x3 %s (all outputs)" % pass_name, got, ref, S, "resnet 3x3 " + pass_name)


def test_resnet_3x3_conv_full_size_two_byte_table(B):
    """ResNet 3x3 at full size with the exact-truncation table (2-byte entries): the forward and
    backward-data passes take the hi/lo path, backward-weight the exact path."""
    cfg = W.RESNET_3X3
    _check_conv_full(B, cfg["conv"], cfg["m_bits"], seed=3200, model="exact_trunc", name="resnet 3x3 exact_trunc")


def test_resnet_3x3_relu_input_full_size(B):
    """The same layer with x = ReLU(N(0,1)): half the first operands of forward and backward-weight
    are exact zeros."""
    cfg = W.RESNET_3X3
    _check_conv_full(B, cfg["conv"], cfg["m_bits"], seed=3100, relu=True, name="resnet 3x3 relu input")


@pytest.mark.parametrize("li", range(len(W.RESNET50_LAYERS)))
def test_resnet50_layers_full_size(B, li):
    cfg = W.RESNET50_LAYERS[li]
    _check_conv_full(B, cfg["conv"], cfg["m_bits"], seed=4000 + 10 * li, stem=(li == 0), samples=(1024, 1024, 256),
                     name=cfg["name"])


@pytest.mark.parametrize("m", [7, 11])
def test_gemm_4096_full_size(B, m):
    cfg = W.GEMM_LARGE
    A, Bm = W.gemm_inputs(cfg["M"], cfg["N"], cfg["K"], "normal", seed=5000)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "mitchell", m), m)).reshape(-1)
    idx = _sample(C.size, 1024, 5000 + m)
    ref, S = oracle.gemm(oracle.MITCHELL, m, A, Bm, idx=idx)
    _record("gemm 4096 M=%d" % m, C[idx], ref, S, "gemm 4096 M=%d" % m)


def test_conv_deterministic(B):
    p = W.RESNET_3X3["conv"]
    x, w, dy = W.resnet_conv_inputs(p, seed=3100)
    lut = dev_lut(B, "mitchell", 7)
    xd, wd, dyd = cuda(x), cuda(w), cuda(dy)
    for fn, args in ((B.approx_conv2d_fwd, (xd, wd)), (B.approx_conv2d_bwd_data, (dyd, wd)),
                     (B.approx_conv2d_bwd_weight, (xd, dyd))):
        r1 = host(fn(p, *args, lut, 7))
        r2 = host(fn(p, *args, lut, 7))
        assert np.array_equal(r1.view(np.uint32), r2.view(np.uint32))


def test_lenet5_stack_fwd_bwd(B):
    """LeNet-5 layer stack, batch 64, exact bfloat16-truncation multiplier (M = 7).  ReLU,
    max-pool and the loss gradient run as plain torch ops; every approximate layer call is
    checked against the oracle fed the same layer inputs."""
    cfg = W.LENET5
    m = cfg["m_bits"]
    lut = dev_lut(B, "exact_trunc", m)
    F = torch.nn.functional
    c1, c2 = cfg["conv1"], cfg["conv2"]
    bs = cfg["batch"]
    x0 = W.uniform((bs, 28, 28, 1), 0.0, 1.0, 6000)
    w1 = W.glorot_uniform((5, 5, 1, 6), 25 * 1, 25 * 6, 6001)
    w2 = W.glorot_uniform((5, 5, 6, 16), 25 * 6, 25 * 16, 6002)
    fcw = [W.glorot_uniform((i, o), i, o, 6003 + j) for j, (i, o) in enumerate(cfg["fc"])]
    labels = np.random.default_rng(6010).integers(0, 10, bs)

    def check(got_t, ref_S, what):
        got = host(got_t)
        assert_within_tolerance(got, ref_S[0], ref_S[1], what)

    def pool(t):  # NHWC 2x2 max-pool via torch
        return F.max_pool2d(t.permute(0, 3, 1, 2), 2).permute(0, 2, 3, 1).contiguous()

    X0 = cuda(x0)
    Y1 = B.approx_conv2d_fwd(c1, X0, cuda(w1), lut, m)
    check(Y1, oracle.conv2d_fwd(oracle.EXACT_TRUNC, m, c1, x0, w1), "conv1 fwd")
    A1 = torch.relu(Y1)
    P1 = pool(A1).requires_grad_(False)
    p1 = host(P1)
    Y2 = B.approx_conv2d_fwd(c2, P1, cuda(w2), lut, m)
    check(Y2, oracle.conv2d_fwd(oracle.EXACT_TRUNC, m, c2, p1, w2), "conv2 fwd")
    A2 = torch.relu(Y2)
    P2 = pool(A2)
    h = P2.reshape(bs, 400).contiguous()
    acts, pre = [h], []
    for j, wj in enumerate(fcw):
        hj = host(acts[-1])
        z = B.approx_gemm(acts[-1], cuda(wj), lut, m)
        check(z, oracle.gemm(oracle.EXACT_TRUNC, m, hj, wj), "fc%d fwd" % (j + 1))
        pre.append(z)
        acts.append(torch.relu(z).contiguous() if j < 2 else z)
    logits = acts[-1]
    g = (torch.softmax(logits, dim=1) - F.one_hot(torch.from_numpy(labels).cuda(), 10).float()) / bs
    g = g.contiguous()
    for j in (2, 1, 0):
        wj = fcw[j]
        aj = host(acts[j])
        gh = host(g)
        dW = B.approx_gemm(acts[j], g, lut, m, trans_a=True)
        check(dW, oracle.gemm(oracle.EXACT_TRUNC, m, aj, gh, True, False), "fc%d bwd_weight" % (j + 1))
        dX = B.approx_gemm(g, cuda(wj), lut, m, trans_b=True)
        check(dX, oracle.gemm(oracle.EXACT_TRUNC, m, gh, wj, False, True), "fc%d bwd_data" % (j + 1))
        g = dX if j == 0 else (dX * (pre[j - 1] > 0).float()).contiguous()
    # back through pool2 / relu2 into conv2
    P2g = g.reshape(bs, 5, 5, 16)
    A2r = A2.detach().clone().requires_grad_(True)
    pool(A2r).backward(P2g)
    dY2 = (A2r.grad * (Y2 > 0).float()).contiguous()
    dy2 = host(dY2)
    dW2 = B.approx_conv2d_bwd_weight(c2, P1, dY2, lut, m)
    check(dW2, oracle.conv2d_bwd_weight(oracle.EXACT_TRUNC, m, c2, p1, dy2), "conv2 bwd_weight")
    dP1 = B.approx_conv2d_bwd_data(c2, dY2, cuda(w2), lut, m)
    check(dP1, oracle.conv2d_bwd_data(oracle.EXACT_TRUNC, m, c2, dy2, w2), "conv2 bwd_data")
    A1r = A1.detach().clone().requires_grad_(True)
    pool(A1r).backward(dP1)
    dY1 = (A1r.grad * (Y1 > 0).float()).contiguous()
    dy1 = host(dY1)
    dW1 = B.approx_conv2d_bwd_weight(c1, X0, dY1, lut, m)
    check(dW1, oracle.conv2d_bwd_weight(oracle.EXACT_TRUNC, m, c1, x0, dy1), "conv1 bwd_weight")
    dX0 = B.approx_conv2d_bwd_data(c1, dY1, cuda(w1), lut, m)
    check(dX0, oracle.conv2d_bwd_data(oracle.EXACT_TRUNC, m, c1, dy1, w1), "conv1 bwd_data")


def test_kernel_timer_times_only_the_selected_kinds(B):
    """amsim_profile_start_kinds: the GEMM kernel is timed, a convolution pass in the same
    profiling window is not (and runs unbracketed); with every kind, both are."""
    A = cuda(W.normal((256, 128), 1.0, 91))
    Bm = cuda(W.normal((128, 64), 1.0, 92))
    p = W.conv_desc(2, 9, 9, 16, 16, 3, 3, 1, 1)
    oh, ow = W.conv_out_hw(p)
    x = cuda(W.normal((2, 9, 9, 16), 1.0, 93))
    w = cuda(W.normal((3, 3, 16, 16), 1.0, 94))
    lut = dev_lut(B, "mitchell", 7)
    for kinds, want in ((["gemm"], (1, 0)), (None, (1, 1))):
        B.amsim_profile_start(16, kinds=kinds)
        B.approx_gemm(A, Bm, lut, 7)
        B.approx_conv2d_fwd(p, x, w, lut, 7)
        torch.cuda.synchronize()
        B.amsim_profile_stop()
        got = (B.amsim_profile_read("gemm")[0], B.amsim_profile_read("conv_fwd")[0])
        assert got == want, (kinds, got)
        assert B.amsim_profile_read("gemm")[1] > 0.0
