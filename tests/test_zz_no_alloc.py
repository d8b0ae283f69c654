"""GPU tests of approx_gemm_noalloc, the GEMM entry point that brings no workspace (its workspace is
the library's fixed per-GPU scratch buffer).  Its results must equal approx_gemm's bit for bit on
the same inputs (the same plan and kernels run), over calls in a row of falling size (each call
finds the previous call's contents in the buffer), and a call too large for the buffer must be
refused before anything runs."""
import numpy as np
import pytest

import oracle
from parity import assert_within_tolerance
from paper_2209_04161_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def B():
    from paper_2209_04161_amd import binding
    binding.lib()
    return binding


def _operands(m, n, k, trans_a, trans_b, seed):
    A = W.normal((k, m) if trans_a else (m, k), 1.0, seed)
    Bm = W.normal((n, k) if trans_b else (k, n), 1.0, seed + 1)
    return A, Bm


def _bits(t):
    torch.cuda.synchronize()
    return t.cpu().numpy().view(np.uint32)


# Calls in a row, each smaller than the one before; the third changes the table's row length
# (M = 9: 512-entry rows), the middle ones the operand layouts; the last is a vector shape, whose
# kernel needs no scratch at all.
SEQUENCE = [
    (1000, 700, 900, 7, False, False),
    (130, 70, 45, 7, True, False),
    (33, 257, 129, 9, False, True),
    (3, 5, 2, 7, True, True),
    (1, 5, 3, 7, True, True),
]


def test_noalloc_matches_approx_gemm_on_calls_of_falling_size(B):
    luts = {m: B.device_lut(B.lut_build(m, "mitchell")) for m in (7, 9)}
    for i, (m, n, k, mb, ta, tb) in enumerate(SEQUENCE):
        ws = B.amsim_gemm_workspace_size(ta, tb, m, n, k, mb)
        assert ws <= B.AMSIM_NOALLOC_SCRATCH_BYTES and (ws > 0 or m == 1), (m, n, k, ws)
        A, Bm = _operands(m, n, k, ta, tb, 100 + 7 * i)
        At, Bt = torch.from_numpy(A).cuda(), torch.from_numpy(Bm).cuda()
        ref = B.approx_gemm(At, Bt, luts[mb], mb, trans_a=ta, trans_b=tb)
        out = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
        got = B.approx_gemm_noalloc(At, Bt, luts[mb], mb, out, trans_a=ta, trans_b=tb)
        assert got is out
        np.testing.assert_array_equal(_bits(out), _bits(ref), err_msg="call %d %s" % (i, (m, n, k, mb, ta, tb)))
        # and within the parity bar of the oracle (sampled outputs)
        rng = np.random.default_rng(i)
        idx = rng.choice(m * n, size=min(m * n, 300), replace=False)
        C_ref, S = oracle.gemm(oracle.MITCHELL, mb, A, Bm, transa=ta, transb=tb, idx=idx)
        assert_within_tolerance(out.cpu().numpy().reshape(-1)[idx], C_ref, S, what="noalloc call %d" % i)


def test_noalloc_twice_same_shape_is_deterministic(B):
    lut = B.device_lut(B.lut_build(7, "mitchell"))
    A, Bm = _operands(300, 200, 500, False, False, 5)
    At, Bt = torch.from_numpy(A).cuda(), torch.from_numpy(Bm).cuda()
    o1 = torch.empty((300, 200), dtype=torch.float32, device="cuda")
    o2 = torch.empty((300, 200), dtype=torch.float32, device="cuda")
    B.approx_gemm_noalloc(At, Bt, lut, 7, o1)
    B.approx_gemm_noalloc(At, Bt, lut, 7, o2)
    np.testing.assert_array_equal(_bits(o1), _bits(o2))


def test_noalloc_k0_fills_negative_zero(B):
    lut = B.device_lut(B.lut_build(7, "mitchell"))
    At = torch.empty((4, 0), dtype=torch.float32, device="cuda")
    Bt = torch.empty((0, 6), dtype=torch.float32, device="cuda")
    out = torch.full((4, 6), 1.0, dtype=torch.float32, device="cuda")
    B.approx_gemm_noalloc(At, Bt, lut, 7, out)
    assert np.all(_bits(out) == np.uint32(0x80000000))


def test_noalloc_refuses_calls_beyond_the_buffer(B):
    lut = B.device_lut(B.lut_build(7, "mitchell"))
    m = n = k = 4096
    assert B.amsim_gemm_workspace_size(False, False, m, n, k, 7) > B.AMSIM_NOALLOC_SCRATCH_BYTES
    At = torch.zeros((m, k), dtype=torch.float32, device="cuda")
    Bt = torch.zeros((k, n), dtype=torch.float32, device="cuda")
    out = torch.full((m, n), 3.0, dtype=torch.float32, device="cuda")
    with pytest.raises(B.AmsimError) as e:
        B.approx_gemm_noalloc(At, Bt, lut, 7, out)
    assert e.value.status == B.AMSIM_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool(torch.all(out == 3.0))  # nothing ran
