"""GPU checks of the direct-evaluation GEMM (no table): Mitchell's products computed from the
operands' bits must equal the oracle's bit for bit, sums must match within 1e-5 * sum|p| +
2^-126, and the native mode must match the FP32 products summed exactly."""
import numpy as np
import pytest

import oracle
from cases import outer_operands, random_bits
from parity import assert_bits_equal, assert_within_tolerance
from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _b():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


def cuda(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("m", [1, 5, 7, 11])
def test_direct_mitchell_products_bit_exact(m):
    B = _b()
    a, b = outer_operands(m, seed=40 + m)
    C = host(B.approx_gemm_direct(cuda(a), cuda(b), "mitchell", m))
    want = oracle.mul(oracle.MITCHELL, m, np.repeat(a[:, 0], b.shape[1]), np.tile(b[0], a.shape[0]))
    assert_bits_equal(C, want, "direct Mitchell K=1 M=%d" % m)


def test_direct_mitchell_special_values_bit_exact():
    from closed_forms import special_values
    B = _b()
    s = special_values()
    r = random_bits(300, 44)
    v = np.concatenate([s, r])
    for m in (3, 7, 11):
        C = host(B.approx_gemm_direct(cuda(v.reshape(-1, 1)), cuda(v.reshape(1, -1)), "mitchell", m))
        want = oracle.mul(oracle.MITCHELL, m, np.repeat(v, v.size), np.tile(v, v.size))
        assert_bits_equal(C, want, "direct Mitchell specials M=%d" % m)


@pytest.mark.parametrize("shape", [(64, 64, 64), (1, 1, 1), (65, 130, 17), (200, 70, 333), (3, 257, 1000)])
@pytest.mark.parametrize("m", [7, 11])
def test_direct_mitchell_gemm_matches_oracle(shape, m):
    B = _b()
    M, N, K = shape
    A = W.normal((M, K), 1.0, 50 + M)
    Bm = W.normal((K, N), 1.0, 60 + N)
    C = host(B.approx_gemm_direct(cuda(A), cuda(Bm), "mitchell", m))
    ref, S = oracle.gemm(oracle.MITCHELL, m, A, Bm)
    assert_within_tolerance(C, ref, S, "direct Mitchell %s M=%d" % (shape, m))


@pytest.mark.parametrize("shape", [(64, 64, 64), (65, 130, 17), (3, 257, 1000)])
def test_direct_native_gemm_matches_fp32_products(shape):
    B = _b()
    M, N, K = shape
    A = W.normal((M, K), 1.0, 70 + M)
    Bm = W.normal((K, N), 1.0, 80 + N)
    C = host(B.approx_gemm_direct(cuda(A), cuda(Bm), "native"))
    p = A[:, :, None] * Bm[None, :, :]          # float32 products, rounded once each
    ref = p.astype(np.float64).sum(1)
    S = np.abs(p).astype(np.float64).sum(1)
    assert_within_tolerance(C, ref, S, "direct native %s" % (shape,))


def test_direct_k0_and_leading_dimension():
    B = _b()
    A = torch.empty((5, 0), device="cuda")
    Bm = torch.empty((0, 6), device="cuda")
    C = host(B.approx_gemm_direct(A, Bm, "mitchell", 7))
    assert np.all(C == 0) and np.all(np.signbit(C))
    big = torch.full((5, 9), 7.0, device="cuda")
    out = big[:, :6]  # ldc 9 > n: the last 3 columns keep their sentinel
    a = W.normal((5, 4), 1.0, 90)
    b = W.normal((4, 6), 1.0, 91)
    B.approx_gemm_direct(cuda(a), cuda(b), "native", out=out)
    got = host(big)
    assert np.all(got[:, 6:] == 7.0)
    ref = (a[:, :, None] * b[None, :, :]).astype(np.float64).sum(1)
    np.testing.assert_allclose(got[:, :6], ref, rtol=1e-5, atol=1e-6)
