"""GPU test: calls on two streams at once, each with its own workspace, give the results the same
calls give one at a time.  A call keeps all its state -- decoded operands, table rows, exponent
statistics, path flags, partial sums -- in its workspace; only the optional kernel timer is
shared (and locked).  The two streams run different shapes and multipliers, so that a shared
flag or table would show up as a wrong path or wrong products."""
import numpy as np
import pytest

from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def B():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


def _bits(t):
    return t.cpu().numpy().view(np.uint32).copy()


def test_two_streams_match_serial_calls(B):
    lut_m = B.device_lut(B.lut_build(7, "mitchell"))
    lut_e = B.device_lut(B.lut_build(7, "exact_trunc"))
    lut_11 = B.device_lut(B.lut_build(11, "mitchell"))
    rng = np.random.default_rng(77)
    A1 = torch.from_numpy(rng.normal(0, 1, (1024, 768)).astype(np.float32)).cuda()
    B1 = torch.from_numpy(rng.normal(0, 1, (768, 512)).astype(np.float32)).cuda()
    # out of the bf16 window: the exact path on this stream while the other runs the pair path
    A2 = torch.from_numpy((rng.normal(0, 1, (700, 300)) * 2.0 ** 120).astype(np.float32)).cuda()
    B2 = torch.from_numpy((rng.normal(0, 1, (300, 260)) * 2.0 ** 10).astype(np.float32)).cuda()
    cv = W.conv_desc(8, 20, 18, 32, 48, 3, 3, 2, 1)
    oh, ow = W.conv_out_hw(cv)
    x = torch.from_numpy(rng.normal(0, 1, (8, 20, 18, 32)).astype(np.float32)).cuda()
    w = torch.from_numpy(rng.normal(0, 0.2, (3, 3, 32, 48)).astype(np.float32)).cuda()
    dy = torch.from_numpy(rng.normal(0, 1, (8, oh, ow, 48)).astype(np.float32)).cuda()
    A3, B3 = A1[:, :300].contiguous(), B1[:300, :64].contiguous()

    def work_a():
        return [B.approx_gemm(A1, B1, lut_m, 7), B.approx_conv2d_bwd_data(cv, dy, w, lut_e, 7),
                B.approx_gemm(A3, B3, lut_11, 11)]

    def work_b():
        return [B.approx_gemm(A2, B2, lut_m, 7), B.approx_conv2d_fwd(cv, x, w, lut_m, 7),
                B.approx_conv2d_bwd_weight(cv, x, dy, lut_e, 7)]

    ref_a = [_bits(t) for t in work_a()]
    ref_b = [_bits(t) for t in work_b()]
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()  # default priority
    for rep in range(3):
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            got_a = work_a()
        with torch.cuda.stream(s2):
            got_b = work_b()
        torch.cuda.synchronize()
        for i, (g, r) in enumerate(zip(got_a, ref_a)):
            assert np.array_equal(_bits(g), r), "stream 1, call %d, repetition %d" % (i, rep)
        for i, (g, r) in enumerate(zip(got_b, ref_b)):
            assert np.array_equal(_bits(g), r), "stream 2, call %d, repetition %d" % (i, rep)
