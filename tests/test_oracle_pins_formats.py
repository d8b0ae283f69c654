"""Pins of the oracle's other multipliers (CPU only): the native FP32 multiply, the exponent
cast of a (1, e, m) format and Algorithm 2 in that format's constants.

* Native: the IEEE single-precision product that numpy's float32 multiply computes, with
  denormal operands read as zero and denormal results flushed to zero around it.
* Cast (1, 5, 10), the IEEE binary16 layout: values binary16 represents pass unchanged, the
  range limits are binary16's largest finite value 65504 and smallest normal 2^-14, a value
  from 2^16 on becomes Inf (or 65504 when saturating), a binary16 denormal becomes zero.
* Products in (1, 5, 10): for operands whose exact product has at most 11 significant bits,
  the exact-truncation model equals numpy's binary16 product wherever both are normal, zero
  below binary16's normal range and Inf from 2^16 on; the boundary cases that Algorithm 2's
  order (zero test before the carry) decides are pinned one by one.
* e = 8 is Algorithm 2 itself: every product equals the FP32 oracle's on the whole grid.
"""
import numpy as np
import pytest

import oracle
from cases import mantissa_pairs_grid, random_bits, special_cross
from closed_forms import daz

F16_MAX = float(np.finfo(np.float16).max)    # 65504
F16_TINY = float(np.finfo(np.float16).tiny)  # 2^-14


def _ftz(x):
    x = np.asarray(x, dtype=np.float32)
    return np.where((x != 0) & (np.abs(x) < np.float32(2.0 ** -126)), np.copysign(np.float32(0.0), x), x)


def _same(got, want):
    got = np.asarray(got, np.float32).reshape(-1)
    want = np.asarray(want, np.float32).reshape(-1)
    ok = (got.view(np.uint32) == want.view(np.uint32)) | (np.isnan(got) & np.isnan(want))
    return ok


# ------------------------------------------------------------------ native multiply ------

def test_native_product_is_numpy_float32_product():
    a = random_bits(200000, 11)
    b = random_bits(200000, 12)
    sa, sb = special_cross()
    a = np.concatenate([a, sa])
    b = np.concatenate([b, sb])
    with np.errstate(over="ignore", invalid="ignore"):
        want = _ftz(daz(a) * daz(b))
    got = oracle.mul_ex(oracle.MITCHELL, 7, a, b, native=True)
    ok = _same(got, want)
    assert ok.all(), np.nonzero(~ok)[0][:5]


def test_native_product_rounds_to_nearest_even_and_overflows():
    one_ulp = np.float32(1.0) + np.float32(2.0 ** -23)
    # (1 + 2^-23)^2 = 1 + 2^-22 + 2^-46: rounds to 1 + 2^-22
    assert oracle.mul_native(float(one_ulp), float(one_ulp)) == float(np.float32(1.0) + np.float32(2.0 ** -22))
    big = float(np.finfo(np.float32).max)
    assert oracle.mul_native(big, 2.0) == np.inf
    assert oracle.mul_native(-big, 2.0) == -np.inf
    assert oracle.mul_native(2.0 ** -70, 2.0 ** -70) == 0.0          # below the normal range
    assert np.signbit(oracle.mul_native(-(2.0 ** -70), 2.0 ** -70))   # flushed to -0
    assert np.isnan(oracle.mul_native(0.0, np.inf))


def test_native_gemm_equals_sum_of_numpy_float32_products():
    rng = np.random.default_rng(5)
    A = rng.standard_normal((23, 37)).astype(np.float32)
    B = rng.standard_normal((37, 19)).astype(np.float32)
    C, S = oracle.gemm(oracle.MITCHELL, 7, A, B, native=True)
    prods = A[:, :, None] * B[None, :, :]          # float32 products, each rounded by numpy
    ref = prods.astype(np.float64).sum(axis=1)
    assert np.allclose(C, ref, rtol=0, atol=1e-12 * np.abs(prods).sum(axis=1).max() + 1e-30) or \
        np.all(np.abs(C - ref) <= np.abs(ref) * 2.0 ** -24 + 1e-30)
    assert np.allclose(S, np.abs(prods.astype(np.float64)).sum(axis=1))


# ------------------------------------------------------------------ exponent cast --------

def test_cast_1_5_10_keeps_binary16_values():
    rng = np.random.default_rng(21)
    h = rng.integers(0, 1 << 16, 200000, dtype=np.uint32).astype(np.uint16).view(np.float16)
    h = h[np.isfinite(h) & (np.abs(h) >= F16_TINY)]   # binary16 normals
    x = h.astype(np.float32)
    got = oracle.cast(5, x, m_bits=10)
    assert _same(got, x).all()
    assert _same(oracle.cast(5, x, sat=True, m_bits=10), x).all()


def test_cast_1_5_10_range_limits():
    big = np.float32(2.0 ** 16)
    below_big = np.nextafter(big, np.float32(0))        # exponent 15: in range
    tiny = np.float32(F16_TINY)
    below_tiny = np.nextafter(tiny, np.float32(0))      # a binary16 denormal
    x = np.array([F16_MAX, below_big, big, -big, 1e30, -1e30, tiny, below_tiny, -below_tiny, 1e-30,
                  np.inf, -np.inf, np.nan, 0.0, -0.0], np.float32)
    want_inf = np.array([F16_MAX, below_big, np.inf, -np.inf, np.inf, -np.inf, tiny, 0.0, -0.0, 0.0,
                         np.inf, -np.inf, np.nan, 0.0, -0.0], np.float32)
    want_sat = want_inf.copy()
    want_sat[[2, 4]] = F16_MAX
    want_sat[[3, 5]] = -F16_MAX
    assert _same(oracle.cast(5, x, m_bits=10), want_inf).all()
    assert _same(oracle.cast(5, x, sat=True, m_bits=10), want_sat).all()


def test_cast_largest_finite_value_per_mantissa_width():
    # (2 - 2^-m) * 2^beta, beta = 2^(e-1) - 1
    for e, m in [(2, 3), (4, 3), (5, 2), (5, 10), (7, 7)]:
        beta = (1 << (e - 1)) - 1
        got = oracle.cast(e, np.array([3.0e38], np.float32), sat=True, m_bits=m)[0]
        assert got == np.float32((2.0 - 2.0 ** -m) * 2.0 ** beta), (e, m)


def test_cast_e8_is_identity_on_normals():
    x = random_bits(300000, 31)
    fin = np.isfinite(x)
    got = oracle.cast(8, x, m_bits=7)
    assert _same(got[fin], daz(x)[fin]).all()


# ------------------------------------------------------------------ (1, e, m) products ---

def _f16_exact_operands(rng, n, sig_bits=4):
    """binary16 normals whose significands have sig_bits fraction bits (products then have at
    most 2 * (sig_bits + 1) significant bits, within binary16's 11)."""
    e = rng.integers(-14, 16, n)
    frac = rng.integers(0, 1 << sig_bits, n) / float(1 << sig_bits)
    s = np.where(rng.random(n) < 0.5, -1.0, 1.0)
    return (s * (1.0 + frac) * np.exp2(e)).astype(np.float32)


def test_product_1_5_10_equals_binary16_product():
    rng = np.random.default_rng(41)
    a = _f16_exact_operands(rng, 100000)
    b = _f16_exact_operands(rng, 100000)
    ua = np.floor(np.log2(np.abs(a.astype(np.float64)))).astype(int)
    ub = np.floor(np.log2(np.abs(b.astype(np.float64)))).astype(int)
    got = oracle.mul_ex(oracle.EXACT_TRUNC, 10, a, b, e_bits=5)
    with np.errstate(over="ignore"):
        p16 = (a.astype(np.float16) * b.astype(np.float16)).astype(np.float32)
    exact = a.astype(np.float64) * b.astype(np.float64)
    # away from the zero rule's boundary (ua + ub = -15, decided before the carry)
    normal = (ua + ub >= -14)
    assert _same(got[normal], p16[normal]).all()
    assert (np.abs(exact[normal & (np.abs(exact) >= 2.0 ** 16)]) >= 2.0 ** 16).all()
    deep = ua + ub <= -16            # binary16 denormal or zero; the format reads it as zero
    assert (got[deep] == 0).all() and (np.signbit(got[deep]) == np.signbit(exact[deep])).all()


@pytest.mark.parametrize("a,b,want", [
    (2.0 ** -7, 2.0 ** -7, 2.0 ** -14),              # smallest normal product
    (2.0 ** -7, 2.0 ** -8, 0.0),                     # Ea' + Eb' - beta = 0: zero
    (1.5 * 2.0 ** -8, 1.5 * 2.0 ** -7, 0.0),         # zero before the carry would make it normal
    (2.0 ** 7, 1.9375 * 2.0 ** 8, 1.9375 * 2.0 ** 15),  # largest exponent, no carry
    (2.0 ** 8, 2.0 ** 8, np.inf),                    # Ea' + Eb' - beta = 31 = 2^5 - 1
    (1.5 * 2.0 ** 7, 1.5 * 2.0 ** 8, np.inf),        # the carry lifts it to 31
    (-(2.0 ** 8), 2.0 ** 8, -np.inf),
    (2.0 ** 16, 2.0 ** -10, np.inf),                 # the operand casts to Inf first
    (2.0 ** -15, 2.0 ** 10, 0.0),                    # the operand casts to zero first
    (2.0 ** -15, np.inf, np.nan),                    # zero times Inf
])
def test_product_1_5_10_boundaries(a, b, want):
    got = oracle.mul_ex(oracle.EXACT_TRUNC, 10, np.array([a], np.float32), np.array([b], np.float32), e_bits=5)[0]
    assert _same([got], [want]).all(), (a, b, got, want)


def test_saturating_cast_feeds_the_product():
    got = oracle.mul_ex(oracle.EXACT_TRUNC, 10, np.array([1.0e6, -1.0e9], np.float32),
                        np.array([2.0 ** -12, 2.0 ** -13], np.float32), e_bits=5, sat=True)
    assert _same(got, np.array([F16_MAX * 2.0 ** -12, -F16_MAX * 2.0 ** -13], np.float32)).all()


@pytest.mark.parametrize("model", [oracle.MITCHELL, oracle.EXACT_TRUNC])
@pytest.mark.parametrize("m", [3, 7])
def test_e8_is_algorithm_2(model, m):
    a, b = mantissa_pairs_grid(m, seed=m + 50)
    sa, sb = special_cross()
    a = np.concatenate([a, sa, random_bits(50000, 7)])
    b = np.concatenate([b, sb, random_bits(50000, 8)])
    assert _same(oracle.mul_ex(model, m, a, b, e_bits=8), oracle.mul(model, m, a, b)).all()


@pytest.mark.parametrize("e", [3, 5, 7])
def test_narrow_format_equals_fp32_inside_its_range(e):
    """A product whose operands and result stay inside the format's range is the FP32 one."""
    beta = (1 << (e - 1)) - 1
    m = 7
    a, b = mantissa_pairs_grid(m, seed=e, exps=[(127, 127), (127 + beta // 2, 127 - beta // 2),
                                                (127 - beta // 2 + 1, 127)])
    assert _same(oracle.mul_ex(oracle.MITCHELL, m, a, b, e_bits=e), oracle.mul(oracle.MITCHELL, m, a, b)).all()


def test_format_gemm_equals_float64_matmul_of_binary16_values():
    rng = np.random.default_rng(77)
    A = (_f16_exact_operands(rng, 40 * 30) * np.float32(2.0 ** -4)).reshape(40, 30)
    B = (_f16_exact_operands(rng, 30 * 20) * np.float32(2.0 ** -4)).reshape(30, 20)
    A = np.clip(A, -255, 255).astype(np.float32)
    B = np.clip(B, -255, 255).astype(np.float32)
    A[np.abs(A) < 2.0 ** -6] = 0.0
    B[np.abs(B) < 2.0 ** -6] = 0.0
    C, S = oracle.gemm(oracle.EXACT_TRUNC, 10, A, B, e_bits=5)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    assert np.all(np.abs(C - ref) <= 1e-12 * S + np.abs(ref) * 2.0 ** -24)
