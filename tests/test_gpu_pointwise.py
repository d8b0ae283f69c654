"""GPU parity of 1 x 1 convolutions with stride 1 and no padding, which run as their GEMM.

Such a kernel's im2col matrix is the input itself (Algorithm 3) and there are no border or
dilation zeros, so each pass is a GEMM over the pixels with the pass's first operand first: the
library dispatches it to the GEMM path (tiled, or the vector kernels when a dimension is 1).
Every pass is compared with the oracle's convolution, for the table's products (M = 7 and 11),
the native multiply and a narrow format; the kernel timer still reports the pass; the
workspace query matches the GEMM's; and a pass too large for the GEMM's limits keeps the
convolution path.
"""
import numpy as np
import pytest

import oracle
from parity import assert_within_tolerance
from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

CASES = [
    W.conv_desc(3, 5, 7, 19, 13, 1, 1),      # ragged tiles
    W.conv_desc(2, 9, 11, 64, 40, 1, 1),
    W.conv_desc(1, 14, 14, 256, 72, 1, 1),   # reduction over many channels (splits)
    W.conv_desc(4, 3, 3, 5, 1, 1, 1),        # one output channel: forward is a vector product
    W.conv_desc(1, 1, 1, 33, 20, 1, 1),      # one pixel: backward weight is an outer product
    W.conv_desc(2, 4, 6, 1, 17, 1, 1),       # one input channel: forward is an outer product
]

MODES = [("mitchell", 7, {}), ("exact_trunc", 7, {}), ("mitchell", 11, {}), ("native", 7, {"multiply": "native"}),
         ("mitchell", 7, {"e_bits": 5, "exp_cast": "saturate"})]


@pytest.fixture(scope="module")
def B():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


def cuda(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _inputs(p, seed):
    x = W.normal((p["n"], p["h"], p["w"], p["c_in"]), 1.0, seed)
    w = W.normal((1, 1, p["c_in"], p["c_out"]), 0.5, seed + 1)
    dy = W.normal((p["n"], p["h"], p["w"], p["c_out"]), 1.0, seed + 2)
    return x, w, dy


@pytest.mark.parametrize("mi", range(len(MODES)), ids=[m[0] + str(m[1]) + ("_fmt" if "e_bits" in m[2] else "")
                                                        for m in MODES])
@pytest.mark.parametrize("ci", range(len(CASES)))
def test_pointwise_passes_match_the_oracle(B, ci, mi):
    p = CASES[ci]
    model, m, opts = MODES[mi]
    x, w, dy = _inputs(p, 900 + 7 * ci)
    native = opts.get("multiply") == "native"
    lut = None if native else B.device_lut(B.lut_build(m, model))
    mid = 0 if native else (oracle.MITCHELL if model == "mitchell" else oracle.EXACT_TRUNC)
    om = dict(native=True) if native else {}
    if "e_bits" in opts:
        om = dict(e_bits=opts["e_bits"], sat=opts["exp_cast"] == "saturate")
    for name, fn, ref_fn, a0, a1 in (("fwd", B.approx_conv2d_fwd_ex, oracle.conv2d_fwd, x, w),
                                     ("bwd_data", B.approx_conv2d_bwd_data_ex, oracle.conv2d_bwd_data, dy, w),
                                     ("bwd_weight", B.approx_conv2d_bwd_weight_ex, oracle.conv2d_bwd_weight, x, dy)):
        got = host(fn(p, cuda(a0), cuda(a1), lut, m, **opts))
        ref, S = ref_fn(mid, m, p, a0, a1, **om)
        assert_within_tolerance(got, ref, S, "pointwise %s case %d %s" % (name, ci, MODES[mi][0]))


def test_pointwise_timer_and_workspace(B):
    p = CASES[2]
    x, w, dy = _inputs(p, 950)
    lut = B.device_lut(B.lut_build(7, "mitchell"))
    npix = p["n"] * p["h"] * p["w"]
    # the workspace query is the GEMM's
    assert B.amsim_conv2d_workspace_size(p, 0, 7) == B.amsim_gemm_workspace_size(0, 0, npix, p["c_out"], p["c_in"], 7)
    assert B.amsim_conv2d_workspace_size(p, 1, 7) == B.amsim_gemm_workspace_size(0, 1, npix, p["c_in"], p["c_out"], 7)
    assert B.amsim_conv2d_workspace_size(p, 2, 7) == B.amsim_gemm_workspace_size(1, 0, p["c_in"], p["c_out"], npix, 7)
    xs, ws, dys = cuda(x), cuda(w), cuda(dy)
    B.approx_conv2d_fwd(p, xs, ws, lut, 7)
    torch.cuda.synchronize()
    B.amsim_profile_start(64)
    B.approx_conv2d_fwd(p, xs, ws, lut, 7)
    B.approx_conv2d_bwd_data(p, dys, ws, lut, 7)
    B.approx_conv2d_bwd_weight(p, xs, dys, lut, 7)
    torch.cuda.synchronize()
    B.amsim_profile_stop()
    for kind in ("conv_fwd", "conv_bwd_data", "conv_bwd_weight"):
        assert B.amsim_profile_read(kind)[0] == 1, kind
    assert B.amsim_profile_read("gemm")[0] == 0


def test_pointwise_beyond_the_gemm_limits_keeps_the_convolution_path(B):
    """Backward weight over 2 195 200 pixels: the GEMM's decoded first operand would pass 2^29
    words (pixels x 256 padded rows), so the pass runs as a convolution."""
    p = W.conv_desc(700, 56, 56, 4, 3, 1, 1)
    x, w, dy = _inputs(p, 960)
    lut = B.device_lut(B.lut_build(7, "mitchell"))
    npix = p["n"] * p["h"] * p["w"]
    assert B.amsim_conv2d_workspace_size(p, 2, 7) != B.amsim_gemm_workspace_size(1, 0, 4, 3, npix, 7)
    dw = host(B.approx_conv2d_bwd_weight(p, cuda(x), cuda(dy), lut, 7)).reshape(-1)
    ref, S = oracle.conv2d_bwd_weight(oracle.MITCHELL, 7, p, x, dy)
    assert_within_tolerance(dw, ref.reshape(-1), S.reshape(-1), "pointwise bwd_weight beyond the GEMM limits")
