"""GPU test: the library's calls can be captured into a HIP graph (torch.cuda.CUDAGraph) and
replayed.  Every call only enqueues kernels on the caller's stream (no host synchronisation, no
allocation inside the library; workspaces and outputs come from torch, inside the capture from
its graph pool), so a captured sequence -- tiled GEMMs, the three convolution passes with padding,
stride and the few-channel unfolded paths, the vector GEMMs -- replays to the same bits as eager
calls, also after its inputs are overwritten with new values between replays.  Each replay is
followed by eager work and a synchronisation before its results are read."""
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


def _inputs(seed):
    rng = np.random.default_rng(seed)
    c1 = W.conv_desc(8, 28, 28, 1, 6, 5, 5, 1, 2)            # few channels: unfolded passes
    c2 = W.conv_desc(8, 14, 14, 6, 16, 5, 5, 1, 0)
    c3 = dict(W.conv_desc(4, 15, 13, 12, 20, 3, 3, 2, 1), stride_w=3)  # strides, padding
    x1 = rng.uniform(0, 1, (8, 28, 28, 1)).astype(np.float32)
    w1 = rng.normal(0, 0.3, (5, 5, 1, 6)).astype(np.float32)
    x2 = rng.uniform(0, 1, (8, 14, 14, 6)).astype(np.float32)
    w2 = rng.normal(0, 0.1, (5, 5, 6, 16)).astype(np.float32)
    oh, ow = W.conv_out_hw(c2)
    dy2 = rng.normal(0, 1, (8, oh, ow, 16)).astype(np.float32)
    oh1, ow1 = W.conv_out_hw(c1)
    dy1 = rng.normal(0, 1, (8, oh1, ow1, 6)).astype(np.float32)
    x3 = rng.normal(0, 1, (4, 15, 13, 12)).astype(np.float32)
    w3 = rng.normal(0, 0.2, (3, 3, 12, 20)).astype(np.float32)
    oh3, ow3 = W.conv_out_hw(c3)
    dy3 = rng.normal(0, 1, (4, oh3, ow3, 20)).astype(np.float32)
    a = rng.normal(0, 1, (130, 400)).astype(np.float32)
    wf = rng.normal(0, 0.05, (400, 120)).astype(np.float32)
    g = rng.normal(0, 1, (130, 120)).astype(np.float32)
    v = rng.normal(0, 1, (1, 400)).astype(np.float32)
    descs = (c1, c2, c3)
    tensors = dict(x1=x1, w1=w1, x2=x2, w2=w2, dy2=dy2, dy1=dy1, x3=x3, w3=w3, dy3=dy3, a=a, wf=wf, g=g, v=v)
    return descs, tensors


def _sequence(B, descs, T, lut, m):
    c1, c2, c3 = descs
    return [
        B.approx_conv2d_fwd(c1, T["x1"], T["w1"], lut, m),
        B.approx_conv2d_bwd_weight(c1, T["x1"], T["dy1"], lut, m),
        B.approx_conv2d_bwd_data(c1, T["dy1"], T["w1"], lut, m),
        B.approx_conv2d_fwd(c2, T["x2"], T["w2"], lut, m),
        B.approx_conv2d_bwd_data(c2, T["dy2"], T["w2"], lut, m),
        B.approx_conv2d_bwd_weight(c2, T["x2"], T["dy2"], lut, m),
        B.approx_conv2d_fwd(c3, T["x3"], T["w3"], lut, m),
        B.approx_conv2d_bwd_data(c3, T["dy3"], T["w3"], lut, m),
        B.approx_conv2d_bwd_weight(c3, T["x3"], T["dy3"], lut, m),
        B.approx_gemm(T["a"], T["wf"], lut, m),
        B.approx_gemm(T["a"], T["g"], lut, m, trans_a=True),
        B.approx_gemm(T["g"], T["wf"], lut, m, trans_b=True),
        B.approx_gemm(T["v"], T["wf"], lut, m),                 # vector path, m = 1
        B.approx_gemm(T["a"], T["v"], lut, m, trans_b=True),   # vector path, n = 1
    ]


def _bits(ts):
    torch.cuda.synchronize()
    return [t.cpu().numpy().view(np.uint32).copy() for t in ts]


@pytest.mark.parametrize("model,m", [("mitchell", 7), ("exact_trunc", 7), ("mitchell", 10)])
def test_captured_sequence_replays_to_eager_bits(B, model, m):
    lut = B.device_lut(B.lut_build(m, model))
    descs, host = _inputs(11)
    T = {k: torch.from_numpy(v).cuda() for k, v in host.items()}
    eager = _bits(_sequence(B, descs, T, lut, m))          # also the warm-up before capture
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        outs = _sequence(B, descs, T, lut, m)
    for replay in range(3):
        graph.replay()
        torch.cuda.synchronize()
        _ = torch.ones(1000, device="cuda").sum().item()   # eager work between replays
        got = _bits(outs)
        for i, (g, e) in enumerate(zip(got, eager)):
            assert np.array_equal(g, e), "replay %d, call %d differs from the eager result" % (replay, i)
    # new input values in the captured tensors: the replay computes them, with nothing left over
    # from the capture (statistics, flags, table preparation all run again)
    _, host2 = _inputs(12)
    for k, v in host2.items():
        T[k].copy_(torch.from_numpy(v))
    eager2 = _bits(_sequence(B, descs, T, lut, m))
    graph.replay()
    got2 = _bits(outs)
    for i, (g, e) in enumerate(zip(got2, eager2)):
        assert np.array_equal(g, e), "replay on new inputs, call %d differs from the eager result" % i
    # values outside the bf16 window switch the path inside the replay (flags set on the device)
    T["a"].copy_(torch.from_numpy(host2["a"] * np.float32(2.0 ** 100)))
    eager3 = _bits(_sequence(B, descs, T, lut, m))
    graph.replay()
    got3 = _bits(outs)
    for i, (g, e) in enumerate(zip(got3, eager3)):
        assert np.array_equal(g, e), "replay with large operands, call %d differs from the eager result" % i
