"""GPU parity of the other multipliers the kernels simulate (through the _ex entry points):

* the native FP32 multiply in the same table kernels (the paper's "with native multiply" runs):
  single products bit for bit against the oracle's IEEE product, sums within the parity bar,
  for the GEMM and all three convolution passes;
* (1, e, m) formats with e < 8 (Sec. "AMSim"): the exponent cast bit for bit, single products
  bit for bit over every mantissa pair and an exponent grid around the format's zero and
  infinity limits, and sums of the GEMM and the convolution passes.
"""
import numpy as np
import pytest

import oracle
from cases import mantissa_pairs_grid, random_bits, special_cross
from parity import assert_bits_equal, assert_within_tolerance
from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def B():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


_LUTS = {}


def dev_lut(B, model, m):
    if (model, m) not in _LUTS:
        _LUTS[(model, m)] = B.device_lut(B.lut_build(m, model))
    return _LUTS[(model, m)]


MODELS = {"mitchell": oracle.MITCHELL, "exact_trunc": oracle.EXACT_TRUNC}


def cuda(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _normal_range(x):
    """Keeps operands whose products stay clear of FP32's denormal range (where the flush of a
    result that rounds to the smallest normal is the hardware's choice)."""
    x = np.asarray(x, np.float32).copy()
    u = x.view(np.uint32)
    e = (u >> 23) & 0xFF
    bad = (e > 0) & (e < 70) | (e > 190) & (e < 255)
    x[bad] = np.float32(1.5)
    return x


# ------------------------------------------------------------------ native multiply ------

def test_native_gemm_k1_products_bit_exact(B):
    a = _normal_range(random_bits(2048, 3)).reshape(-1, 1)
    b = _normal_range(random_bits(300, 4)).reshape(1, -1)
    sa, sb = special_cross()
    a = np.concatenate([a[:, 0], sa[:37]]).reshape(-1, 1)
    C = host(B.approx_gemm_ex(cuda(a), cuda(b), None, 7, multiply="native"))
    want = oracle.mul_ex(0, 7, np.repeat(a[:, 0], b.shape[1]), np.tile(b[0], a.shape[0]), native=True)
    assert_bits_equal(C, want, "native gemm K=1")


@pytest.mark.parametrize("shape", [(64, 64, 64), (257, 129, 513), (130, 7, 300), (4096, 512, 256)])
def test_native_gemm_sums(B, shape):
    M, N, K = shape
    A = W.normal((M, K), 1.0, 20 + M)
    Bm = W.normal((K, N), 1.0, 30 + N)
    C = host(B.approx_gemm_ex(cuda(A), cuda(Bm), None, 7, multiply="native")).reshape(-1)
    idx = None if M * N <= 300000 else np.sort(np.random.default_rng(M).choice(M * N, 20000, replace=False))
    ref, S = oracle.gemm(0, 7, A, Bm, idx=idx, native=True)
    assert_within_tolerance(C if idx is None else C[idx], ref, S, "native gemm %s" % (shape,))


@pytest.mark.parametrize("ta,tb", [(True, False), (False, True)])
def test_native_gemm_transposes(B, ta, tb):
    A = W.normal((91, 77) if ta else (77, 91), 1.0, 41)
    Bm = W.normal((45, 91) if tb else (91, 45), 1.0, 42)
    C = host(B.approx_gemm_ex(cuda(A), cuda(Bm), None, 7, trans_a=ta, trans_b=tb, multiply="native"))
    ref, S = oracle.gemm(0, 7, A, Bm, ta, tb, native=True)
    assert_within_tolerance(C, ref, S, "native gemm trans %s %s" % (ta, tb))


NATIVE_CONV = [
    W.conv_desc(2, 9, 8, 2, 3, 3, 3, 2, 1),
    W.conv_desc(2, 13, 12, 20, 70, 3, 3, 1, 1),
    W.conv_desc(1, 16, 16, 3, 20, 7, 7, 2, 3),      # w-unfolded forward and backward data
    W.conv_desc(2, 6, 6, 24, 200, 3, 3, 2, 1),
    W.conv_desc(2, 9, 7, 32, 10, 3, 3, 1, 1),       # forward taps in channel chunks
]


@pytest.mark.parametrize("ci", range(len(NATIVE_CONV)))
def test_native_conv_passes(B, ci):
    p = NATIVE_CONV[ci]
    oh, ow = W.conv_out_hw(p)
    x = W.normal((p["n"], p["h"], p["w"], p["c_in"]), 1.0, 60 + ci)
    w = W.normal((p["kh"], p["kw"], p["c_in"], p["c_out"]), 1.0, 61 + ci)
    dy = W.normal((p["n"], oh, ow, p["c_out"]), 1.0, 62 + ci)
    y = host(B.approx_conv2d_fwd_ex(p, cuda(x), cuda(w), None, 7, multiply="native"))
    ref, S = oracle.conv2d_fwd(0, 7, p, x, w, native=True)
    assert_within_tolerance(y, ref, S, "native fwd %d" % ci)
    dx = host(B.approx_conv2d_bwd_data_ex(p, cuda(dy), cuda(w), None, 7, multiply="native"))
    ref, S = oracle.conv2d_bwd_data(0, 7, p, dy, w, native=True)
    assert_within_tolerance(dx, ref, S, "native bwd_data %d" % ci)
    dw = host(B.approx_conv2d_bwd_weight_ex(p, cuda(x), cuda(dy), None, 7, multiply="native"))
    ref, S = oracle.conv2d_bwd_weight(0, 7, p, x, dy, native=True)
    assert_within_tolerance(dw, ref, S, "native bwd_weight %d" % ci)


def test_native_conv_single_products_bit_exact(B):
    p = W.conv_desc(2, 5, 7, 1, 70, 1, 1, 1, 0)
    x = _normal_range(random_bits(70, 5)).reshape(2, 5, 7, 1)
    w = _normal_range(random_bits(70, 6)).reshape(1, 1, 1, 70)
    y = host(B.approx_conv2d_fwd_ex(p, cuda(x), cuda(w), None, 7, multiply="native"))
    want = oracle.mul_ex(0, 7, np.repeat(x.reshape(-1), 70), np.tile(w.reshape(-1), 70), native=True)
    assert_bits_equal(y, want, "native conv fwd single products")


def test_native_resnet_3x3_sampled(B):
    cfg = W.RESNET_3X3
    p = cfg["conv"]
    x, w, dy = W.resnet_conv_inputs(p, seed=3000)
    xd, wd, dyd = cuda(x), cuda(w), cuda(dy)
    for name, fn, args, of in (
            ("fwd", B.approx_conv2d_fwd_ex, (xd, wd), lambda idx: oracle.conv2d_fwd(0, 7, p, x, w, idx=idx, native=True)),
            ("bwd_data", B.approx_conv2d_bwd_data_ex, (dyd, wd),
             lambda idx: oracle.conv2d_bwd_data(0, 7, p, dy, w, idx=idx, native=True)),
            ("bwd_weight", B.approx_conv2d_bwd_weight_ex, (xd, dyd),
             lambda idx: oracle.conv2d_bwd_weight(0, 7, p, x, dy, idx=idx, native=True))):
        got = host(fn(p, *args, None, 7, multiply="native")).reshape(-1)
        idx = np.sort(np.random.default_rng(len(name)).choice(got.size, 1024, replace=False))
        ref, S = of(idx)
        assert_within_tolerance(got[idx], ref, S, "native resnet 3x3 %s" % name)


# ------------------------------------------------------------------ (1, e, m) formats ----

def _format_grid(m, e, seed):
    """Every mantissa pair at exponent pairs around the format's zero and infinity limits (and
    outside its range, where the cast acts), both signs, plus the special-value cross product."""
    beta = (1 << (e - 1)) - 1
    c = 127
    exps = [(c, c), (c + beta, c), (c + beta, c + 1), (c - beta + 1, c - beta + 1), (c - beta + 1, c),
            (c - beta // 2, c - beta // 2), (c - beta // 2, c - (beta + 1) // 2), (c + beta // 2, c + beta // 2 + 1),
            (c + beta + 1, c - 3), (c - beta, c + 2), (c + beta // 2 + 1, c + beta // 2 + 1)]
    exps = [(min(max(ea, 1), 254), min(max(eb, 1), 254)) for ea, eb in exps]
    a, b = mantissa_pairs_grid(m, seed, exps=exps)
    sa, sb = special_cross()
    return np.concatenate([a, sa]), np.concatenate([b, sb])


@pytest.mark.parametrize("e,sat", [(2, False), (4, True), (5, False), (5, True), (7, False)])
def test_cast_exponent_bit_exact(B, e, sat):
    x = np.concatenate([random_bits(1 << 18, 90 + e), special_cross()[0]])
    for m in (3, 10):
        got = host(B.amsim_cast_exponent(cuda(x), e, "saturate" if sat else "inf", m))
        assert_bits_equal(got, oracle.cast(e, x, sat=sat, m_bits=m), "cast e=%d sat=%s m=%d" % (e, sat, m))


@pytest.mark.parametrize("model", ["mitchell", "exact_trunc"])
@pytest.mark.parametrize("e,sat,m", [(5, False, 7), (5, True, 4), (3, False, 5), (7, True, 7), (2, False, 3)])
def test_format_products_bit_exact(B, model, e, sat, m):
    a, b = _format_grid(m, e, seed=e * 10 + m)
    got = host(B.approx_mul_ew_ex(cuda(a), cuda(b), dev_lut(B, model, m), m, e_bits=e,
                                  exp_cast="saturate" if sat else "inf"))
    assert_bits_equal(got, oracle.mul_ex(MODELS[model], m, a, b, e_bits=e, sat=sat),
                      "mul_ew %s e=%d sat=%s M=%d" % (model, e, sat, m))


@pytest.mark.parametrize("e,sat,m", [(5, False, 7), (4, True, 5), (7, False, 10)])
def test_format_gemm_k1_products_bit_exact(B, e, sat, m):
    """K = 1 through the GEMM kernel: the decode's cast and the exact path's scaled products."""
    beta = (1 << (e - 1)) - 1
    rng = np.random.default_rng(e + m)
    n = 1 << m
    k = np.arange(n, dtype=np.uint32)
    if n > 256:
        k = np.sort(rng.choice(n, 256, replace=False)).astype(np.uint32)

    def vec(exps):
        parts = []
        for ex in exps:
            for s in (0, 1):
                low = rng.integers(0, 1 << (23 - m), k.size, dtype=np.uint32)
                parts.append((np.uint32(s) << 31) | (np.uint32(ex) << 23) | (k << (23 - m)) | low)
        return np.concatenate(parts).view(np.float32)

    c = 127
    a = vec([c, c + beta, c - beta + 1, c + beta + 2, c - beta - 1]).reshape(-1, 1)
    b = vec([c, c + 1, c - beta // 2, c - 2]).reshape(1, -1)
    opt = "saturate" if sat else "inf"
    C = host(B.approx_gemm_ex(cuda(a), cuda(b), dev_lut(B, "mitchell", m), m, e_bits=e, exp_cast=opt))
    want = oracle.mul_ex(oracle.MITCHELL, m, np.repeat(a[:, 0], b.shape[1]), np.tile(b[0], a.shape[0]), e_bits=e,
                         sat=sat)
    assert_bits_equal(C, want, "format gemm K=1 e=%d" % e)


@pytest.mark.parametrize("e,sat,model,m", [(5, False, "exact_trunc", 10), (5, True, "mitchell", 7),
                                           (4, False, "mitchell", 7), (7, False, "exact_trunc", 7),
                                           (5, True, "mitchell", 10)])
@pytest.mark.parametrize("shape", [(130, 70, 300), (4096, 256, 64)])
def test_format_gemm_sums(B, e, sat, model, m, shape):
    M, N, K = shape
    A = W.normal((M, K), 1.0, 3 * M + e)
    Bm = W.normal((K, N), 1.0, 5 * N + e)
    A[0, :4] = [1e6, -1e7, 3e-9, -2e-8]          # beyond the format's range on both sides
    opt = "saturate" if sat else "inf"
    C = host(B.approx_gemm_ex(cuda(A), cuda(Bm), dev_lut(B, model, m), m, e_bits=e, exp_cast=opt)).reshape(-1)
    idx = None if M * N <= 300000 else np.sort(np.random.default_rng(N).choice(M * N, 20000, replace=False))
    ref, S = oracle.gemm(MODELS[model], m, A, Bm, idx=idx, e_bits=e, sat=sat)
    assert_within_tolerance(C if idx is None else C[idx], ref, S, "format gemm e=%d %s %s" % (e, model, shape))


@pytest.mark.parametrize("e,sat", [(5, False), (4, True)])
@pytest.mark.parametrize("ci", [0, 1, 2])
def test_format_conv_passes(B, e, sat, ci):
    p = NATIVE_CONV[ci]
    oh, ow = W.conv_out_hw(p)
    x = W.normal((p["n"], p["h"], p["w"], p["c_in"]), 1.0, 70 + ci)
    w = W.normal((p["kh"], p["kw"], p["c_in"], p["c_out"]), 1.0, 71 + ci)
    dy = W.normal((p["n"], oh, ow, p["c_out"]), 1.0, 72 + ci)
    x.reshape(-1)[:2] = [4e5, -3e-9]
    lut = dev_lut(B, "mitchell", 7)
    opt = "saturate" if sat else "inf"
    kw = dict(e_bits=e, exp_cast=opt)
    om = dict(e_bits=e, sat=sat)
    y = host(B.approx_conv2d_fwd_ex(p, cuda(x), cuda(w), lut, 7, **kw))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, 7, p, x, w, **om)
    assert_within_tolerance(y, ref, S, "format fwd e=%d" % e)
    dx = host(B.approx_conv2d_bwd_data_ex(p, cuda(dy), cuda(w), lut, 7, **kw))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, 7, p, dy, w, **om)
    assert_within_tolerance(dx, ref, S, "format bwd_data e=%d" % e)
    dw = host(B.approx_conv2d_bwd_weight_ex(p, cuda(x), cuda(dy), lut, 7, **kw))
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, 7, p, x, dy, **om)
    assert_within_tolerance(dw, ref, S, "format bwd_weight e=%d" % e)


def test_options_rejected(B):
    x = cuda(np.ones((4, 4), np.float32))
    lut = dev_lut(B, "mitchell", 7)
    with pytest.raises(B.AmsimError):
        B.approx_gemm_ex(x, x, lut, 7, e_bits=1)
    with pytest.raises(B.AmsimError):
        B.approx_gemm_ex(x, x, lut, 7, e_bits=9)
    with pytest.raises(B.AmsimError):
        B.approx_gemm_ex(x, x, None, 7, multiply="native", e_bits=5)
