"""GPU parity of the table kernels' exact path at K > 1, and of the choice between the paths.

The bf16 pair path (1-byte tables) and the hi/lo path (2-byte tables) run only while the
operands' exponents keep every product inside the normal range; Inf/NaN operands, or exponents
outside that window, send a call to the exact path, which implements Algorithm 2's zero and
overflow rules (zero test before the carry, Inf when the carry lifts the exponent to 255) and
IEEE Inf/NaN handling.  These tests run every such case through multi-step sums (several 8-step
slabs), including a product that overflows next to a large opposite-signed partial sum, NaN and
+-Inf inside sums, sums that overflow, and operands just inside and just outside each window
threshold, compared element by element with the oracle.
"""
import numpy as np
import pytest

import oracle
from parity import assert_within_tolerance
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


def cuda(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def with_exponent(x, field):
    """x with its exponent field replaced (sign and mantissa kept)."""
    u = np.atleast_1d(np.asarray(x, np.float32)).copy().view(np.uint32)
    r = ((u & np.uint32(0x807FFFFF)) | (np.uint32(field) << np.uint32(23))).view(np.float32)
    return r if np.ndim(x) else r[0]


def gemm_check(B, A, Bm, model="mitchell", m=7, what=""):
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, model, m), m))
    ref, S = oracle.gemm(MODELS[model], m, A, Bm)
    return assert_within_tolerance(C, ref, S, what)


@pytest.mark.parametrize("k", [2, 9, 17, 300, 4096])
def test_gemm_out_of_window_operands_multi_step(B, k):
    """One tiny operand (exponent field 2) among normal values: the window fails on its low
    side and the exact 1-byte path runs every slab of the sum."""
    A = W.normal((130, k), 1.0, 700 + k)
    Bm = W.normal((k, 24), 1.0, 800 + k)
    A[7, k // 2] = with_exponent(A[7, k // 2], 2)
    gemm_check(B, A, Bm, what="gemm tiny operand K=%d" % k)
    # a huge second operand (field 254): the window fails on its high side; products of it with
    # |a| >= 1 overflow to Inf and their sums too
    A = W.uniform((130, k), -1.0, 1.0, 710 + k)
    Bm = W.normal((k, 24), 1.0, 810 + k)
    Bm[k - 1, 3] = with_exponent(Bm[k - 1, 3], 254)
    gemm_check(B, A, Bm, what="gemm huge operand K=%d" % k)


@pytest.mark.parametrize("k", [2, 9, 300])
def test_gemm_overflowing_product_next_to_opposite_sum(B, k):
    """The product of 1.5 * 2^127 and 1.5 is Inf under Algorithm 2 (exponent 254 plus the carry);
    a partial sum of -2^127 must not absorb it: the output is +Inf."""
    A = np.zeros((64, k), np.float32)
    Bm = np.zeros((k, 16), np.float32)
    A[:, 0] = -(2.0 ** 127)
    A[:, k - 1] = 1.5 * 2.0 ** 127
    Bm[0, :] = 1.0
    Bm[k - 1, :] = 1.5
    if k > 2:
        A[:, 1:k - 1] = W.uniform((64, k - 2), -1.0, 1.0, 900 + k)
        Bm[1:k - 1, :] = W.uniform((k - 2, 16), -1.0, 1.0, 901 + k)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "mitchell", 7), 7))
    ref, S = oracle.gemm(oracle.MITCHELL, 7, A, Bm)
    assert np.all(ref == np.inf)
    assert_within_tolerance(C, ref, S, "overflow next to -2^127, K=%d" % k)


@pytest.mark.parametrize("k", [9, 64, 300])
def test_gemm_nan_and_infinities_in_sums(B, k):
    A = W.normal((70, k), 1.0, 950 + k)
    Bm = W.normal((k, 20), 1.0, 960 + k)
    A[3, k // 3] = np.nan                       # NaN in a row: the whole output row is NaN
    Bm[1, 5] = np.inf                            # +Inf and -Inf in one column: NaN where both count
    Bm[k - 2, 5] = -np.inf
    Bm[k // 2, 9] = np.inf                       # +Inf alone: +-Inf by the first operand's sign
    A[10, k // 2] = 0.0                          # Inf times zero: NaN
    gemm_check(B, A, Bm, what="gemm NaN/Inf K=%d" % k)
    # sums that overflow to Inf: products near 2^127, all positive
    A = np.abs(W.normal((70, k), 1.0, 970 + k)) * np.float32(2.0 ** 100)
    Bm = np.abs(W.normal((k, 20), 1.0, 971 + k)) * np.float32(2.0 ** 26)
    A = A.astype(np.float32)
    Bm = Bm.astype(np.float32)
    ref, _ = oracle.gemm(oracle.MITCHELL, 7, A, Bm)
    assert np.isinf(ref).any()
    gemm_check(B, A, Bm, what="gemm overflowing sums K=%d" % k)


def _window_operands(rng, shape, lo, hi):
    """Random operands whose finite exponent fields span exactly [lo, hi] (both attained)."""
    n = int(np.prod(shape))
    e = rng.integers(lo, hi + 1, n).astype(np.uint32)
    e[0], e[-1] = lo, hi
    mant = rng.integers(0, 1 << 23, n, dtype=np.uint32)
    sign = (rng.random(n) < 0.5).astype(np.uint32) << 31
    x = (sign | (e << 23) | mant).view(np.float32).reshape(shape)
    return rng.permutation(x.reshape(-1)).reshape(shape)


# (name, A's exponent range, B's exponent range): each threshold of the bf16 window on both sides
THRESHOLDS = [
    ("lo sum 128 (inside)", (64, 130), (64, 127)),
    ("lo sum 127 (outside)", (64, 130), (63, 127)),
    ("hi sum 380 (inside)", (120, 253), (100, 127)),
    ("hi sum 381 (outside)", (120, 254), (100, 127)),
    ("b hi 253 (inside)", (100, 127), (100, 253)),
    ("b hi 254 (outside)", (100, 126), (100, 254)),
]


@pytest.mark.parametrize("ti", range(len(THRESHOLDS)))
def test_gemm_window_thresholds_mitchell(B, ti):
    name, ra, rb = THRESHOLDS[ti]
    rng = np.random.default_rng(1000 + ti)
    A = _window_operands(rng, (4096, 17), *ra)
    Bm = _window_operands(rng, (17, 64), *rb)
    gemm_check(B, A, Bm, "mitchell", 7, "window %s" % name)
    # a small tile shape as well (other tile, same decision)
    gemm_check(B, A[:300], Bm[:, :24], "mitchell", 7, "window %s, small" % name)


# the hi/lo path's extra thresholds (2-byte tables): b_lo >= 16 and a_lo + b_lo >= 143
HL_THRESHOLDS = [
    ("b lo 16 (inside)", (127, 130), (16, 127)),
    ("b lo 15 (outside)", (128, 130), (15, 127)),
    ("lo sum 143 (inside)", (120, 130), (23, 127)),
    ("lo sum 142 (outside)", (120, 130), (22, 127)),
]


@pytest.mark.parametrize("ti", range(len(HL_THRESHOLDS)))
def test_gemm_window_thresholds_exact_trunc(B, ti):
    name, ra, rb = HL_THRESHOLDS[ti]
    rng = np.random.default_rng(1100 + ti)
    A = _window_operands(rng, (4096, 16), *ra)
    Bm = _window_operands(rng, (16, 4096), *rb)
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "exact_trunc", 7), 7)).reshape(-1)
    idx = np.sort(np.random.default_rng(1200 + ti).choice(C.size, 20000, replace=False))
    ref, S = oracle.gemm(oracle.EXACT_TRUNC, 7, A, Bm, idx=idx)
    assert_within_tolerance(C[idx], ref, S, "hi/lo window %s" % name)


# Calls of fewer than 2^27 products decide their path inside the table kernel; larger calls take it
# from a flags launch after the pre-pass.  Both decisions, on every threshold and special case,
# at both sizes: A is rows x 64, B 64 x cols.
SIZES = {"small": (300, 96), "large": (4096, 1024)}   # 1.8M and 268M products


def _sampled_gemm_check(B, A, Bm, model, what, seed):
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, model, 7), 7)).reshape(-1)
    idx = np.sort(np.random.default_rng(seed).choice(C.size, min(C.size, 20000), replace=False))
    ref, S = oracle.gemm(MODELS[model], 7, A, Bm, idx=idx)
    assert_within_tolerance(C[idx], ref, S, what)


@pytest.mark.parametrize("size", sorted(SIZES))
@pytest.mark.parametrize("case", [("mitchell",) + t for t in THRESHOLDS] + [("exact_trunc",) + t for t in HL_THRESHOLDS],
                         ids=lambda c: "%s %s" % (c[0], c[1]))
def test_window_thresholds_both_path_decisions(B, case, size):
    model, name, ra, rb = case
    rows, cols = SIZES[size]
    rng = np.random.default_rng(1400 + len(name) + rows)
    A = _window_operands(rng, (rows, 64), *ra)
    Bm = _window_operands(rng, (64, cols), *rb)
    _sampled_gemm_check(B, A, Bm, model, "%s window %s, %s call" % (model, name, size), 1500 + rows)


@pytest.mark.parametrize("size", sorted(SIZES))
@pytest.mark.parametrize("model", sorted(MODELS))
def test_special_operands_both_path_decisions(B, model, size):
    """NaN and +-Inf operands (no exponent window: the exact path, rounded products)."""
    rows, cols = SIZES[size]
    A = W.normal((rows, 64), 1.0, 1600 + rows)
    Bm = W.normal((64, cols), 1.0, 1601 + rows)
    A[3, 10] = np.nan
    Bm[5, 7] = np.inf
    Bm[40, 7] = -np.inf
    Bm[20, 9] = np.inf
    A[rows - 1, 20] = -np.inf
    _sampled_gemm_check(B, A, Bm, model, "%s NaN/Inf, %s call" % (model, size), 1602 + rows)


def _conv_case(seed, special):
    p = W.conv_desc(2, 9, 10, 12, 20, 3, 3, 1, 0)
    oh, ow = W.conv_out_hw(p)
    x = W.normal((2, 9, 10, 12), 1.0, seed)
    w = W.normal((3, 3, 12, 20), 1.0, seed + 1)
    dy = W.normal((2, oh, ow, 20), 1.0, seed + 2)
    if special == "tiny":
        x[0, 4, 5, 3] = with_exponent(x[0, 4, 5, 3], 2)
        dy[1, 2, 3, 7] = with_exponent(dy[1, 2, 3, 7], 2)
    elif special == "huge":
        w[1, 1, 4, 9] = with_exponent(w[1, 1, 4, 9], 254)
        dy[0, 3, 3, 2] = with_exponent(dy[0, 3, 3, 2], 254)
    elif special == "naninf":
        x[1, 5, 5, 2] = np.nan
        w[0, 2, 7, 11] = np.inf
        w[2, 0, 7, 11] = -np.inf
        dy[0, 1, 2, 4] = np.inf
        dy[1, 4, 4, 6] = -np.inf
    return p, x, w, dy


@pytest.mark.parametrize("special", ["tiny", "huge", "naninf"])
def test_conv_passes_exact_path_multi_step(B, special):
    p, x, w, dy = _conv_case(1300 + len(special), special)
    lut = dev_lut(B, "mitchell", 7)
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, 7))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, 7, p, x, w)
    assert_within_tolerance(y, ref, S, "fwd %s" % special)
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, 7))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, 7, p, dy, w)
    assert_within_tolerance(dx, ref, S, "bwd_data %s" % special)
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, 7))
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, 7, p, x, dy)
    assert_within_tolerance(dw, ref, S, "bwd_weight %s" % special)


@pytest.mark.parametrize("special", ["huge", "naninf"])
def test_conv_passes_exact_path_large_calls(B, special):
    """The exact path on calls of more than 2^27 products (path flags from their own launch), each
    pass on seeded sampled outputs: stride 2 and padding 1, 16 x 33 x 31 x 64 -> 64 channels."""
    p = W.conv_desc(16, 33, 31, 64, 64, 3, 3, 2, 1)
    oh, ow = W.conv_out_hw(p)
    x = W.normal((16, 33, 31, 64), 1.0, 1700)
    w = W.normal((3, 3, 64, 64), 1.0, 1701)
    dy = W.normal((16, oh, ow, 64), 1.0, 1702)
    assert W.conv_macs(p) > 2 ** 27
    if special == "huge":
        w[1, 1, 4, 9] = with_exponent(w[1, 1, 4, 9], 254)
        dy[0, 3, 3, 2] = with_exponent(dy[0, 3, 3, 2], 254)
        x[2, 7, 8, 5] = with_exponent(x[2, 7, 8, 5], 253)
    else:
        x[1, 5, 5, 2] = np.nan
        w[0, 2, 7, 11] = np.inf
        w[2, 0, 7, 11] = -np.inf
        dy[0, 1, 2, 4] = np.inf
        dy[1, 4, 4, 6] = -np.inf
    lut = dev_lut(B, "mitchell", 7)
    rng = np.random.default_rng(1703)
    for name, got, fn, a0, a1 in (
            ("fwd", B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, 7), oracle.conv2d_fwd, x, w),
            ("bwd_data", B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, 7), oracle.conv2d_bwd_data, dy, w),
            ("bwd_weight", B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, 7), oracle.conv2d_bwd_weight,
             x, dy)):
        got = host(got).reshape(-1)
        idx = np.sort(rng.choice(got.size, min(got.size, 3000), replace=False))
        ref, S = fn(oracle.MITCHELL, 7, p, a0, a1, idx=idx)
        assert_within_tolerance(got[idx], ref, S, "%s %s, large call" % (name, special))


def test_conv_overflowing_product_next_to_opposite_sum(B):
    """Forward pass with a 1x1 kernel and two input channels: x = (-2^127, 1.5 * 2^127) against
    w = (1, 1.5) gives -2^127 + Inf = +Inf at every output."""
    p = W.conv_desc(1, 4, 9, 2, 8, 1, 1, 1, 0)
    x = np.zeros((1, 4, 9, 2), np.float32)
    x[..., 0] = -(2.0 ** 127)
    x[..., 1] = 1.5 * 2.0 ** 127
    w = np.zeros((1, 1, 2, 8), np.float32)
    w[0, 0, 0, :] = 1.0
    w[0, 0, 1, :] = 1.5
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), dev_lut(B, "mitchell", 7), 7))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, 7, p, x, w)
    assert np.all(ref == np.inf)
    assert_within_tolerance(y, ref, S, "fwd overflow next to -2^127")


@pytest.mark.parametrize("m", [9, 11])
def test_wide_table_overflowing_product_next_to_opposite_sum(B, m):
    A = np.zeros((64, 4), np.float32)
    Bm = np.zeros((4, 16), np.float32)
    A[:, 0] = -(2.0 ** 127)
    A[:, 3] = 1.5 * 2.0 ** 127
    Bm[0, :] = 1.0
    Bm[3, :] = 1.5
    C = host(B.approx_gemm(cuda(A), cuda(Bm), dev_lut(B, "mitchell", m), m))
    ref, S = oracle.gemm(oracle.MITCHELL, m, A, Bm)
    assert np.all(ref == np.inf)
    assert_within_tolerance(C, ref, S, "wide table M=%d overflow" % m)


# ------------------------------------------------- zeros of the column matrix (reading R11)
# Algorithm 3 and 4 multiply the zeros their column matrices hold -- the zero border of x, the
# padding and the stride dilation of the error -- so an Inf or NaN weight at such a tap gives NaN,
# and such a product's sign counts in an exactly zero sum.  The kernels evaluate the border taps
# and the phases' padding; the taps between stride phases and the w-unfolded pass's unreached
# columns are added from per-channel flags.

BORDER_CASES = [
    ("pad 1", W.conv_desc(2, 7, 8, 9, 10, 3, 3, 1, 1)),
    ("stride 2", W.conv_desc(2, 9, 8, 12, 10, 3, 3, 2, 1)),
    ("stride 2x3, asymmetric pads", dict(W.conv_desc(1, 11, 10, 10, 6, 5, 5, 2, pads=(2, 1, 0, 3)), stride_w=3)),
    ("few channels, unfolded", W.conv_desc(2, 9, 10, 3, 6, 3, 4, 1, 1)),
    ("few channels, unfolded, stride 2", W.conv_desc(2, 11, 12, 2, 5, 5, 5, 2, 2)),
    # stride 1, pads within the kernel, 16 or more output channels: backward data on the forward route
    ("pad 1, backward data as forward", W.conv_desc(2, 7, 8, 9, 20, 3, 3, 1, 1)),
    ("asymmetric pads up to k - 1, backward data as forward", W.conv_desc(1, 8, 9, 6, 17, 4, 3, 1, pads=(3, 0, 1, 2))),
]


def _check_class_and_zero_signs(got, ref, S, what):
    zero = ref == 0.0
    if zero.any():
        from parity import assert_bits_equal
        assert_bits_equal(got[zero], ref[zero].astype(np.float32), what + " zero outputs")
    assert_within_tolerance(got, ref, S, what)


@pytest.mark.parametrize("ci", range(len(BORDER_CASES)))
def test_conv_border_products_inf_weights(B, ci):
    name, p = BORDER_CASES[ci]
    oh, ow = W.conv_out_hw(p)
    x = W.normal((p["n"], p["h"], p["w"], p["c_in"]), 1.0, 1400 + ci)
    w = W.normal((p["kh"], p["kw"], p["c_in"], p["c_out"]), 1.0, 1401 + ci)
    dy = W.normal((p["n"], oh, ow, p["c_out"]), 1.0, 1402 + ci)
    w[0, p["kw"] - 1, 1, 2] = np.inf      # a corner tap: padded for border outputs
    w[p["kh"] - 1, 0, 0, 3] = -np.inf
    w[p["kh"] // 2, p["kw"] // 2, p["c_in"] - 1, 0] = np.nan
    dy[0, 0, ow - 1, 1] = np.inf          # an error at the corner: its window holds padding of x
    lut = dev_lut(B, "mitchell", 7)
    y = host(B.approx_conv2d_fwd(p, cuda(x), cuda(w), lut, 7))
    ref, S = oracle.conv2d_fwd(oracle.MITCHELL, 7, p, x, w)
    assert np.isnan(ref).any()
    _check_class_and_zero_signs(y, ref, S, "fwd %s" % name)
    dx = host(B.approx_conv2d_bwd_data(p, cuda(dy), cuda(w), lut, 7))
    ref, S = oracle.conv2d_bwd_data(oracle.MITCHELL, 7, p, dy, w)
    _check_class_and_zero_signs(dx, ref, S, "bwd_data %s" % name)
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, 7))
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, 7, p, x, dy)
    _check_class_and_zero_signs(dw, ref, S, "bwd_weight %s" % name)


@pytest.mark.parametrize("ci", range(len(BORDER_CASES)))
@pytest.mark.parametrize("model", ["mitchell", "exact_trunc"])
def test_conv_border_products_zero_signs(B, ci, model):
    """Exactly-zero sums whose sign the border, padding and dilation zeros decide: inputs of +0 and
    -0 blocks against weights of one sign per output channel, a few taps of the other sign."""
    name, p = BORDER_CASES[ci]
    oh, ow = W.conv_out_hw(p)
    rng = np.random.default_rng(1500 + ci)
    x = W.normal((p["n"], p["h"], p["w"], p["c_in"]), 1.0, 1500 + ci)
    dy = W.normal((p["n"], oh, ow, p["c_out"]), 1.0, 1501 + ci)
    w = np.abs(W.normal((p["kh"], p["kw"], p["c_in"], p["c_out"]), 1.0, 1502 + ci))
    x[0] = 0.0
    x[0, :, : p["w"] // 2] = -0.0
    dy[0] = 0.0
    dy[0, : oh // 2] = -0.0
    w[..., ::2] *= -1                                 # negative and positive output channels
    w[0, 0, :, 1::4] *= -1                            # one tap of the other sign
    w[..., 3 % p["c_out"]] = -0.0
    lut = dev_lut(B, model, 7)
    om = MODELS[model]
    signs = set()
    for fn, of, args, oargs in (
            (B.approx_conv2d_fwd, oracle.conv2d_fwd, (cuda(x), cuda(w)), (x, w)),
            (B.approx_conv2d_bwd_data, oracle.conv2d_bwd_data, (cuda(dy), cuda(w)), (dy, w)),
            (B.approx_conv2d_bwd_weight, oracle.conv2d_bwd_weight, (cuda(x), cuda(dy)), (x, dy))):
        got = host(fn(p, *args, lut, 7))
        ref, S = of(om, 7, p, *oargs)
        zero = ref == 0.0
        signs |= set(np.signbit(ref[zero]).tolist())
        _check_class_and_zero_signs(got, ref, S, "%s %s" % (fn.__name__, name))
    assert signs == {True, False}


@pytest.mark.parametrize("pass_id", [0, 1, 2])
def test_exact_trunc_conv_passes_on_four_wave_tiles(B, pass_id):
    """The 2-byte (exact bfloat16-truncation) table on the hi/lo path in 4-wave tiles: the ResNet
    3x3 shape at batch 8, whose backward-weight pass (576 rows) takes a 4-wave, 8-column tile;
    seeded sampled outputs against the oracle."""
    p = W.conv_desc(8, 32, 32, 64, 64, 3, 3, 1, 1)
    x, w, dy = W.resnet_conv_inputs(p, seed=1800)
    lut = dev_lut(B, "exact_trunc", 7)
    rng = np.random.default_rng(1801 + pass_id)
    fn, ref_fn, a0, a1 = [(B.approx_conv2d_fwd, oracle.conv2d_fwd, x, w),
                          (B.approx_conv2d_bwd_data, oracle.conv2d_bwd_data, dy, w),
                          (B.approx_conv2d_bwd_weight, oracle.conv2d_bwd_weight, x, dy)][pass_id]
    got = host(fn(p, cuda(a0), cuda(a1), lut, 7)).reshape(-1)
    idx = np.sort(rng.choice(got.size, min(got.size, 4000), replace=False))
    ref, S = ref_fn(oracle.EXACT_TRUNC, 7, p, a0, a1, idx=idx)
    assert_within_tolerance(got[idx], ref, S, "exact_trunc pass %d" % pass_id)
