"""Independent derivations used to pin the oracle (test helpers, numpy only).

* Closed forms of the Algorithm 1 table for the two built-in multipliers, derived in integer
  arithmetic from the mathematics (not by calling any model).
* A bit-level mirror of Algorithm 2 (AMSim) that reads a table, with the readings of the
  paper's silent/garbled points spelled out (R1-R5 in the oracle header).
* Bit-truncation helpers (the (1,8,m) format conversion of Sec. "Experiment Setup").
"""
import numpy as np

E_MASK = np.uint32(0x7F800000)
S_MASK = np.uint32(0x80000000)
F_MASK = np.uint32(0x007FFFFF)


def mitchell_lut_closed_form(m):
    """Mitchell: operands 1.k and 1.j (k, j in units of 2^-M); log sum = (k + j) * 2^-M.

    If k + j < 2^M the product is 1 + (k+j)/2^M (no carry, mantissa (k+j) << (23-M)), otherwise
    it is 2 * (k+j)/2^M = 2 * (1 + (k+j-2^M)/2^M) (carry, mantissa (k+j-2^M) << (23-M)).
    """
    n = 1 << m
    k = np.arange(n, dtype=np.int64)[:, None]
    j = np.arange(n, dtype=np.int64)[None, :]
    s = k + j
    out = np.where(s < n, s << (23 - m), (1 << 23) | ((s - n) << (23 - m)))
    return out.astype(np.uint32).reshape(-1)


def exact_lut_closed_form(m):
    """Exact product of (1 + k/2^M)(1 + j/2^M) = p / 2^(2M) with p = (2^M + k)(2^M + j).

    p < 2^(2M+1): value in [1,2), mantissa (p - 2^(2M)) scaled to 23 bits = << (23 - 2M).
    Otherwise value in [2,4): carry, mantissa (p - 2^(2M+1)) << (22 - 2M).
    """
    n = 1 << m
    k = np.arange(n, dtype=np.int64)[:, None]
    j = np.arange(n, dtype=np.int64)[None, :]
    p = (n + k) * (n + j)
    lo = (p - (1 << (2 * m))) << (23 - 2 * m)
    hi = (1 << 23) | ((p - (1 << (2 * m + 1))) << (22 - 2 * m))
    out = np.where(p < (1 << (2 * m + 1)), lo, hi)
    return out.astype(np.uint32).reshape(-1)


def trunc_bits(x, m):
    """Keep sign, exponent and the top m mantissa bits of float32 values (bit truncation)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    mask = np.uint32((0xFFFFFFFF << (23 - m)) & 0xFFFFFFFF)
    return (u & mask).view(np.float32)


def daz(x):
    """Denormals read as signed zero (the operand reading of Algorithm 2's exponent test)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    zero_field = (u & E_MASK) == 0
    u[zero_field] &= S_MASK
    return u.view(np.float32)


def alg2_mirror(a, b, lut, m):
    """Algorithm 2 on float32 arrays a, b with mantissa table `lut` (uint32[2^(2M)]).

    Steps in the algorithm's order (masks per R2, index per R1/R2, sign XOR, exponent sum),
    then the special-value policy R3-R5.  Returns float32.
    """
    a = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    b = np.ascontiguousarray(b, dtype=np.float32).view(np.uint32)
    m_mask = np.uint32(((1 << m) - 1) << (23 - m))
    amnt = a & m_mask
    bmnt = b & m_mask
    index = (amnt >> np.uint32(23 - 2 * m)) + (bmnt >> np.uint32(23 - m))
    mntmult = lut[index.astype(np.int64)]
    carry = (mntmult & np.uint32(0x00800000)) >> np.uint32(23)
    mntmult = mntmult & np.uint32(0xFF7FFFFF) & F_MASK
    sign = (a ^ b) & S_MASK
    ea = ((a & E_MASK) >> np.uint32(23)).astype(np.int64)
    eb = ((b & E_MASK) >> np.uint32(23)).astype(np.int64)
    exp = ea + eb - 127
    fa = a & F_MASK
    fb = b & F_MASK
    nan_a = (ea == 255) & (fa != 0)
    nan_b = (eb == 255) & (fb != 0)
    inf_a = (ea == 255) & (fa == 0)
    inf_b = (eb == 255) & (fb == 0)
    zero_a = ea == 0
    zero_b = eb == 0

    out = np.empty(a.shape, dtype=np.uint32)
    normal_exp = exp + carry.astype(np.int64)
    normal = sign | (np.clip(normal_exp, 0, 255).astype(np.uint32) << np.uint32(23)) | mntmult
    out[:] = normal
    overflow_after_carry = normal_exp >= 255
    out[overflow_after_carry] = sign[overflow_after_carry] | np.uint32(0x7F800000)
    ovf = exp >= 255
    out[ovf] = sign[ovf] | np.uint32(0x7F800000)
    zero = (exp <= 0) | zero_a | zero_b
    out[zero] = sign[zero]
    inf = inf_a | inf_b
    out[inf] = sign[inf] | np.uint32(0x7F800000)
    nan = nan_a | nan_b | (inf_a & zero_b) | (inf_b & zero_a)
    out[nan] = np.uint32(0x7FC00000)
    return out.view(np.float32)


def special_values():
    """+-0, denormal extremes, FLT_MIN/MAX, +-Inf, NaN, +-1, +-1.5, powers of two."""
    f = np.float32
    base = [0.0, np.float32(1.4e-45), np.float32(1.1754942e-38), np.float32(1.1754944e-38),
            np.finfo(np.float32).max, np.inf, 1.0, 1.5, 1.9999999, 2.0 ** -63, 2.0 ** -64, 2.0 ** 63,
            2.0 ** 64, 2.0 ** 100, 2.0 ** -100, 3.0 * 2.0 ** 126, 1.75 * 2.0 ** -126, 0.3]
    vals = []
    for v in base:
        vals.append(f(v))
        vals.append(f(-v))
    vals.append(f(np.nan))
    return np.array(vals, dtype=np.float32)


def bits_equal_nan_class(x, y):
    """Element-wise bit equality, counting any NaN equal to any NaN."""
    x = np.asarray(x, dtype=np.float32)
    y = np.asarray(y, dtype=np.float32)
    both_nan = np.isnan(x) & np.isnan(y)
    same = x.view(np.uint32) == y.view(np.uint32)
    return same | both_nan
