"""Writes stay inside the caller's buffers.

Every convolution pass writes its result into the middle of a larger buffer whose two guard
regions hold a sentinel pattern, with a workspace that is an exact-size view of a larger
allocation whose tail holds another pattern.  After the call both guards must be unchanged, and
the result must equal bit for bit the result of an ordinary call (the library is deterministic).
The shapes take every route a pass has: direct and split reductions, the forward and the
stride-phase backward-data kernels, the w-unfolded forward and backward-data passes, pointwise
passes run as GEMMs, and the wide sum-indexed table.
"""
import numpy as np
import pytest

from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GUARD = 4096            # floats on each side of the result
SENTINEL = 0x7FA5A5A5   # a NaN payload no pass writes
WS_GUARD = 65536        # bytes after the workspace
WS_BYTE = 0x5A

CASES = [
    ("3x3 pad 1 (backward data on the forward kernel)", W.conv_desc(2, 9, 9, 32, 24, 3, 3, 1, 1), 7),
    ("stride 2 (backward data by stride phases)", W.conv_desc(2, 11, 10, 12, 20, 3, 3, 2, 1), 7),
    ("few channels (unfolded passes)", W.conv_desc(2, 12, 13, 3, 6, 5, 5, 1, 2), 7),
    ("long reduction, few outputs (split reductions)", W.conv_desc(8, 30, 30, 4, 4, 3, 3, 1, 1), 7),
    ("pointwise (GEMM route)", W.conv_desc(2, 7, 9, 40, 24, 1, 1), 7),
    ("wide sum-indexed table", W.conv_desc(2, 9, 9, 32, 24, 3, 3, 1, 1), 11),
]


@pytest.fixture(scope="module")
def B():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


def _guarded(shape):
    n = int(np.prod(shape))
    buf = torch.empty(n + 2 * GUARD, dtype=torch.int32, device="cuda")
    buf.fill_(SENTINEL)  # below 2^31: the same bits as an int32
    return buf, buf[GUARD:GUARD + n].view(torch.float32).view(shape)


def _guarded_workspace(nbytes):
    buf = torch.full((nbytes + WS_GUARD,), WS_BYTE, dtype=torch.uint8, device="cuda")
    return buf, buf[:nbytes]


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_conv_passes_write_only_their_results(B, ci):
    name, p, m = CASES[ci]
    oh, ow = W.conv_out_hw(p)
    x = torch.from_numpy(W.normal((p["n"], p["h"], p["w"], p["c_in"]), 1.0, 60 + ci)).cuda()
    w = torch.from_numpy(W.normal((p["kh"], p["kw"], p["c_in"], p["c_out"]), 1.0, 61 + ci)).cuda()
    dy = torch.from_numpy(W.normal((p["n"], oh, ow, p["c_out"]), 1.0, 62 + ci)).cuda()
    lut = B.device_lut(B.lut_build(m, "mitchell"))
    passes = [
        ("fwd", B.approx_conv2d_fwd, (x, w), (p["n"], oh, ow, p["c_out"]), B.AMSIM_CONV_FWD),
        ("bwd_data", B.approx_conv2d_bwd_data, (dy, w), (p["n"], p["h"], p["w"], p["c_in"]), B.AMSIM_CONV_BWD_DATA),
        ("bwd_weight", B.approx_conv2d_bwd_weight, (x, dy), (p["kh"], p["kw"], p["c_in"], p["c_out"]),
         B.AMSIM_CONV_BWD_WEIGHT),
    ]
    sentinel = np.int32(np.uint32(SENTINEL).view(np.int32))
    for pname, fn, args, shape, pass_id in passes:
        ref = fn(p, *args, lut, m)
        buf, out = _guarded(shape)
        nbytes = B.amsim_conv2d_workspace_size(p, pass_id, m)
        wbuf, ws = _guarded_workspace(nbytes)
        fn(p, *args, lut, m, out=out, workspace=ws)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        what = "%s %s" % (name, pname)
        assert np.all(b[:GUARD] == sentinel), what + ": a write before the result"
        assert np.all(b[-GUARD:] == sentinel), what + ": a write after the result"
        assert np.array_equal(b[GUARD:-GUARD], ref.cpu().numpy().view(np.int32).reshape(-1)), what + ": result differs"
        tail = wbuf[nbytes:].cpu().numpy()
        assert np.all(tail == WS_BYTE), what + ": a write past the workspace (%d bytes)" % nbytes


GEMM_CASES = [
    ("tiled", (300, 130, 257), 7),
    ("split reduction", (64, 24, 20000), 7),
    ("vector, m = 1", (1, 3000, 700), 7),
    ("vector, n = 1", (3000, 1, 700), 7),
    ("outer product, k = 1", (300, 200, 1), 7),
    ("wide sum-indexed table", (200, 72, 300), 11),
]


@pytest.mark.parametrize("gi", range(len(GEMM_CASES)))
def test_gemm_writes_only_its_result(B, gi):
    name, (m, n, k), mb = GEMM_CASES[gi]
    A = torch.from_numpy(W.normal((m, k), 1.0, 80 + gi)).cuda()
    Bm = torch.from_numpy(W.normal((k, n), 1.0, 81 + gi)).cuda()
    lut = B.device_lut(B.lut_build(mb, "mitchell"))
    ref = B.approx_gemm(A, Bm, lut, mb)
    buf, out = _guarded((m, n))
    nbytes = B.amsim_gemm_workspace_size(0, 0, m, n, k, mb)
    wbuf, ws = _guarded_workspace(nbytes)
    B.approx_gemm(A, Bm, lut, mb, out=out, workspace=ws)
    torch.cuda.synchronize()
    b = buf.cpu().numpy()
    sentinel = np.int32(np.uint32(SENTINEL).view(np.int32))
    assert np.all(b[:GUARD] == sentinel) and np.all(b[-GUARD:] == sentinel), name + ": a write outside the result"
    assert np.array_equal(b[GUARD:-GUARD], ref.cpu().numpy().view(np.int32).reshape(-1)), name + ": result differs"
    assert np.all(wbuf[nbytes:].cpu().numpy() == WS_BYTE), name + ": a write past the workspace (%d bytes)" % nbytes
