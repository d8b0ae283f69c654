"""Sum-indexed wide tables: T[ka][kb] = g(ka + kb).

The table preparation checks every entry of a wide table (M = 8..11) for this property, and the
table kernels then read one array g of 2^(M+1) factors instead of staging a table row per column
and step; any other table keeps the row staging.  The cases run GEMMs over every mantissa pair of
an M = 8 table, built from Mitchell's (which is sum-indexed) with entries changed:
* a whole anti-diagonal changed alike, once below and once above s = 2^M - 1: still sum-indexed,
  and the changed products must come from the table, not from Mitchell's formula;
* a single entry changed off the entries g is read from: no longer sum-indexed, and that product
  must come from the changed entry.
Expected products follow Algorithm 2 for operands whose exponent sum stays in range: the product of
a and b is sign(a) sign(b) 2^(Ea + Eb - 254) v, where v = 2^carry * 1.mantissa is the entry's factor;
at the entries left unchanged this is checked against the oracle's Mitchell products too.
"""
import numpy as np
import pytest

import oracle
from parity import assert_bits_equal, assert_within_tolerance

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

M = 8
N = 1 << M


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


def _operands(seed):
    """a: every mantissa field ka (exponent fields 120..134, random signs and low bits); b likewise
    for kb."""
    rng = np.random.default_rng(seed)
    k = np.arange(N, dtype=np.uint32)

    def vec():
        e = rng.integers(120, 135, N).astype(np.uint32)
        s = rng.integers(0, 2, N).astype(np.uint32)
        low = rng.integers(0, 1 << (23 - M), N, dtype=np.uint32)
        return ((s << 31) | (e << 23) | (k << (23 - M)) | low).view(np.float32)

    return vec(), vec()


def _table_products(lut, a, b):
    """Products of a[i] and b[j] from table entry (ka(a[i]), kb(b[j])): sign * 2^(Ea + Eb - 254) * v."""
    ua, ub = a.view(np.uint32), b.view(np.uint32)
    ka = (ua >> (23 - M)) & (N - 1)
    kb = (ub >> (23 - M)) & (N - 1)
    ent = lut.reshape(N, N)[ka[:, None], kb[None, :]]
    v = ((ent & 0x00FFFFFF) + 0x3F800000).astype(np.uint32).view(np.float32).astype(np.float64)
    ea = ((ua >> 23) & 0xFF).astype(np.int64)
    eb = ((ub >> 23) & 0xFF).astype(np.int64)
    sign = np.where(((ua[:, None] ^ ub[None, :]) >> 31) != 0, -1.0, 1.0)
    return (sign * np.ldexp(v, (ea[:, None] + eb[None, :] - 254))).astype(np.float32)


def _changed_tables(B):
    base = B.lut_build(M, "mitchell")
    ka, kb = np.meshgrid(np.arange(N), np.arange(N), indexing="ij")
    s = (ka + kb).reshape(-1)
    diag = base.copy()
    diag[(s == 100) | (s == 400)] ^= np.uint32(0x100)   # still sum-indexed
    odd = base.copy()
    odd[3 * N + 5] ^= np.uint32(0x100)                    # (3, 5): not an entry g is read from
    return base, {"changed anti-diagonals": (diag, (s == 100) | (s == 400)),
                  "one changed entry": (odd, np.arange(N * N) == 3 * N + 5)}


@pytest.mark.parametrize("case", ["changed anti-diagonals", "one changed entry"])
def test_wide_table_products_come_from_the_table(B, case):
    base, tables = _changed_tables(B)
    lut, changed = tables[case]
    a, b = _operands(7)
    want = _table_products(lut, a, b)
    # the Algorithm 2 products above agree with the oracle's Mitchell products where the entries
    # are Mitchell's, and differ where they were changed
    mitchell = oracle.mul(oracle.MITCHELL, M, np.repeat(a, N), np.tile(b, N))
    assert np.array_equal(want.reshape(-1)[~changed].view(np.uint32), mitchell[~changed].view(np.uint32))
    assert not np.any(want.reshape(-1)[changed] == mitchell[changed])
    C = host(B.approx_gemm(cuda(a.reshape(N, 1)), cuda(b.reshape(1, N)), B.device_lut(lut), M))
    assert_bits_equal(C, want, "K = 1 GEMM, %s" % case)


@pytest.mark.parametrize("case", ["changed anti-diagonals", "one changed entry"])
def test_wide_table_sums_from_the_table(B, case):
    """K = 300 (several slabs of the sum-indexed body): sums of the table's products, within the
    sum tolerance of the oracle's comparisons."""
    base, tables = _changed_tables(B)
    lut, _ = tables[case]
    rng = np.random.default_rng(11)
    K = 300
    A = np.empty((N, K), np.float32)
    Bm = np.empty((K, 40), np.float32)
    for kk in range(K):
        a, b = _operands(100 + kk)
        A[:, kk] = a
        Bm[kk, :] = b[rng.permutation(N)[:40]]
    C = host(B.approx_gemm(cuda(A), cuda(Bm), B.device_lut(lut), M))
    ref = np.zeros((N, 40), np.float64)
    S = np.zeros((N, 40), np.float64)
    for kk in range(K):
        p = _table_products(lut, A[:, kk], Bm[kk, :]).astype(np.float64)
        ref += p
        S += np.abs(p)
    assert_within_tolerance(C, ref.astype(np.float32), S, "K = 300 GEMM, %s" % case)
