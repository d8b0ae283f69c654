"""GPU parity of the GEMM's vector shapes, a dense layer at batch 1 (Sec. "AMDENSE"; the paper's
mat-vec kernel, Sec. "Other Custom CUDA Kernels"):

* m == 1: the forward product y = x W and the input gradient dx = dy W^T of one sample;
* n == 1: the matrix-vector product W x with a column vector;
* k == 1: the weight gradient x^T dy of one sample, an outer product of single products.

These shapes run the vector kernels (one pass over the matrix, operands decoded where they are
read).  Sums are compared with the oracle on every output within the parity bar; k == 1 outputs,
single products, bit for bit.  The operands span the table models, M = 7 and 11, all transpose
layouts, k split across workgroups, special values and zero signs, the native multiply and a
(1, 5, m) format."""
import numpy as np
import pytest

import oracle
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
    if (model, m) not in _LUTS:
        _LUTS[(model, m)] = B.device_lut(B.lut_build(m, model))
    return _LUTS[(model, m)]


def stored(op, trans):
    """The array as stored for a transpose flag (op is the logical operand)."""
    return np.ascontiguousarray(op.T) if trans else np.ascontiguousarray(op)


def run(B, opA, opB, model="mitchell", m_bits=7, ta=False, tb=False, **mult):
    As, Bs = stored(opA, ta), stored(opB, tb)
    lut = dev_lut(B, model, m_bits)
    At, Bt = torch.from_numpy(As).cuda(), torch.from_numpy(Bs).cuda()
    if mult:
        C = B.approx_gemm_ex(At, Bt, lut, m_bits, trans_a=ta, trans_b=tb, **mult)
    else:
        C = B.approx_gemm(At, Bt, lut, m_bits, trans_a=ta, trans_b=tb)
    torch.cuda.synchronize()
    ref, S = oracle.gemm(MODELS[model], m_bits, As, Bs, transa=ta, transb=tb, **_orc(mult))
    return C.cpu().numpy(), ref, S


def _orc(mult):
    o = {}
    if mult.get("multiply") == "native":
        o["native"] = True
    if "e_bits" in mult:
        o["e_bits"] = mult["e_bits"]
    if mult.get("exp_cast") == "saturate":
        o["sat"] = True
    return o


ROW_SHAPES = [(1, 1, 2), (1, 5, 7), (1, 64, 31), (1, 65, 33), (1, 300, 784), (1, 100, 300), (1, 10, 100),
              (1, 1000, 2048), (1, 4097, 129), (1, 3, 40000)]


@pytest.mark.parametrize("shape", ROW_SHAPES)
@pytest.mark.parametrize("ta,tb", [(False, False), (True, True), (False, True)])
def test_row_vector_times_matrix(B, shape, ta, tb):
    m, n, k = shape
    a = W.normal((m, k), 1.0, 11 + k)
    b = W.normal((k, n), 0.05, 12 + n)
    C, ref, S = run(B, a, b, ta=ta, tb=tb)
    assert_within_tolerance(C, ref, S, what="m=1 %s ta=%d tb=%d" % (shape, ta, tb))


@pytest.mark.parametrize("shape", [(5, 1, 7), (64, 1, 31), (300, 1, 784), (4097, 1, 129), (2, 1, 40000)])
@pytest.mark.parametrize("ta,tb", [(False, False), (True, False), (False, True)])
def test_matrix_times_column_vector(B, shape, ta, tb):
    m, n, k = shape
    a = W.normal((m, k), 0.05, 21 + k)
    b = W.normal((k, n), 1.0, 22 + m)
    C, ref, S = run(B, a, b, ta=ta, tb=tb)
    assert_within_tolerance(C, ref, S, what="n=1 %s ta=%d tb=%d" % (shape, ta, tb))


@pytest.mark.parametrize("model,m_bits", [("exact_trunc", 7), ("mitchell", 11), ("mitchell", 3)])
def test_vector_shapes_other_tables(B, model, m_bits):
    a = W.normal((1, 2048), 1.0, 31)
    b = W.normal((2048, 257), 0.05, 32)
    C, ref, S = run(B, a, b, model=model, m_bits=m_bits)
    assert_within_tolerance(C, ref, S, what="m=1 %s M=%d" % (model, m_bits))
    C, ref, S = run(B, b.T.copy(), a.T.copy(), model=model, m_bits=m_bits)
    assert_within_tolerance(C, ref, S, what="n=1 %s M=%d" % (model, m_bits))


def _asym_lut(B, m):
    """The table of an asymmetric model: first operand truncated to M bits, second to M - 1."""
    def asym(a, b):
        ua = np.float32(a).view(np.uint32) & np.uint32((0xFFFFFFFF << (23 - m)) & 0xFFFFFFFF)
        ub = np.float32(b).view(np.uint32) & np.uint32((0xFFFFFFFF << (24 - m)) & 0xFFFFFFFF)
        return float(ua.view(np.float32) * ub.view(np.float32))
    return B.device_lut(B.lut_build(m, asym))


@pytest.mark.parametrize("shape", [(1, 70, 40), (70, 1, 40), (30, 20, 1)])
def test_vector_shapes_operand_order(B, shape):
    """op(A)'s element is the first operand (the table's high index) on every vector shape."""
    m_bits = 5
    m, n, k = shape
    lut = _asym_lut(B, m_bits)
    A = W.uniform((m, k), -2, 2, 91)
    Bm = W.uniform((k, n), -2, 2, 92)
    C = B.approx_gemm(torch.from_numpy(A).cuda(), torch.from_numpy(Bm).cuda(), lut, m_bits)
    torch.cuda.synchronize()
    ref, S = oracle.gemm(oracle.ASYM, m_bits, A, Bm)
    if k == 1:
        assert_bits_equal(C.cpu().numpy(), ref, "asym k=1")
    else:
        assert_within_tolerance(C.cpu().numpy(), ref, S, what="asym %s" % (shape,))
    # the swapped order gives other products (the check above can tell the two apart)
    swapped, _ = oracle.gemm(oracle.ASYM, m_bits, Bm.T.copy(), A.T.copy())
    assert not np.array_equal(swapped.T, ref)


@pytest.mark.parametrize("m,n", [(1, 1), (784, 300), (300, 100), (100, 10), (1, 4097), (4097, 1), (33, 65)])
@pytest.mark.parametrize("ta,tb", [(False, False), (True, True)])
def test_outer_product_is_bit_exact(B, m, n, ta, tb):
    a = W.normal((m, 1), 1.0, 41 + m)
    b = W.normal((1, n), 1.0, 42 + n)
    C, ref, _ = run(B, a, b, ta=ta, tb=tb)
    assert_bits_equal(C, ref, "k=1 outer product %dx%d" % (m, n))


def _specials(x, seed):
    x = x.copy()
    flat = x.reshape(-1)
    rng = np.random.default_rng(seed)
    idx = rng.choice(flat.size, size=min(flat.size, 12), replace=False)
    vals = [np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-40, 3e38, -3e38, 2.0 ** -100, 2.0 ** 100, 1.5 * 2.0 ** 126,
            -1.75 * 2.0 ** 127]
    for i, v in zip(idx, vals):
        flat[i] = np.float32(v)
    return x


@pytest.mark.parametrize("where", ["vector", "matrix"])
def test_vector_shapes_with_specials(B, where):
    a = W.normal((1, 300), 1.0, 51)
    b = W.normal((300, 70), 1.0, 52)
    if where == "vector":
        a = _specials(a, 53)
    else:
        b = _specials(b, 54)
    C, ref, S = run(B, a, b)
    assert_within_tolerance(C, ref, S, what="m=1 specials in the %s" % where)
    C, ref, S = run(B, b.T.copy(), a.T.copy())
    assert_within_tolerance(C, ref, S, what="n=1 specials in the %s" % where)
    C, ref, _ = run(B, a[:, :1].T.copy(), b[:1, :])
    assert_bits_equal(C, ref, "k=1 specials in the %s" % where)


def test_vector_sum_overflow_and_cancellation(B):
    # products that overflow the sum to +Inf in one column, cancel exactly to +0 in another,
    # and are all -0 in a third
    k = 200
    a = np.ones((1, k), np.float32)
    b = np.zeros((k, 3), np.float32)
    b[:, 0] = np.float32(2.0 ** 125)
    b[:100, 1] = 1.5
    b[100:, 1] = -1.5
    b[:, 2] = -0.0
    C, ref, S = run(B, a, b)
    assert np.isposinf(C[0, 0]) and np.isposinf(ref[0, 0])
    assert C[0, 1] == 0.0 and not np.signbit(C[0, 1]) and not np.signbit(ref[0, 1])
    assert C[0, 2] == 0.0 and np.signbit(C[0, 2]) and np.signbit(ref[0, 2])
    assert_within_tolerance(C, ref, S, what="overflow / cancellation")


def _normal_range(x):
    x = np.asarray(x, np.float32).copy()
    e = (x.view(np.uint32) >> 23) & 0xFF
    x[(e > 0) & (e < 70) | (e > 190) & (e < 255)] = np.float32(1.5)
    return x


@pytest.mark.parametrize("shape", [(1, 300, 784), (300, 1, 100), (40, 30, 1)])
def test_vector_shapes_native_multiply(B, shape):
    m, n, k = shape
    a = _normal_range(W.normal((m, k), 1.0, 61))
    b = _normal_range(W.normal((k, n), 1.0, 62))
    C, ref, S = run(B, a, b, multiply="native")
    if k == 1:
        assert_bits_equal(C, ref, "native k=1")
    else:
        assert_within_tolerance(C, ref, S, what="native %s" % (shape,))


@pytest.mark.parametrize("exp_cast", ["inf", "saturate"])
@pytest.mark.parametrize("shape", [(1, 200, 500), (200, 1, 64), (50, 60, 1)])
def test_vector_shapes_narrow_format(B, shape, exp_cast):
    m, n, k = shape
    # values around the (1, 5, m) format's limits: 2^-14 .. 2^15
    rng = np.random.default_rng(71)
    a = (rng.standard_normal((m, k)) * np.exp2(rng.integers(-16, 17, (m, k)))).astype(np.float32)
    b = (rng.standard_normal((k, n)) * np.exp2(rng.integers(-16, 17, (k, n)))).astype(np.float32)
    C, ref, S = run(B, a, b, e_bits=5, exp_cast=exp_cast)
    if k == 1:
        assert_bits_equal(C, ref, "e=5 k=1 %s" % exp_cast)
    else:
        assert_within_tolerance(C, ref, S, what="e=5 %s %s" % (shape, exp_cast))


def test_dense_layer_at_batch_one_matches_oracle(B):
    """LeNet-300-100's first layer at batch 1: forward, input gradient and weight gradient."""
    x = W.uniform((1, 784), 0.0, 1.0, 81)
    w = W.glorot_uniform((784, 300), 784, 300, 82)
    dy = W.normal((1, 300), 0.1, 83)
    y, ref, S = run(B, x, w)
    assert_within_tolerance(y, ref, S, what="fwd")
    dx, ref, S = run(B, dy, w.T.copy(), tb=True)
    assert_within_tolerance(dx, ref, S, what="input gradient")
    dw, ref, _ = run(B, x.T.copy(), dy, ta=True)
    assert_bits_equal(dw, ref, "weight gradient")
