"""Operand sets for exhaustive product checks (test helpers, numpy only)."""
import numpy as np

from closed_forms import special_values

# (Ea, Eb) biased exponent pairs around the zero/overflow limits of Algorithm 2
EXPONENT_PAIRS = [(127, 127), (1, 1), (1, 126), (63, 64), (64, 64), (64, 63), (126, 128), (200, 54),
                  (254, 1), (127, 253), (128, 253), (191, 190), (2, 125), (60, 66), (191, 191)]


def mantissa_pairs_grid(m, seed, exps=EXPONENT_PAIRS):
    """Every pair of top-M mantissa fields (random low bits) x exponent pairs x sign pairs."""
    rng = np.random.default_rng(seed)
    n = 1 << m
    k = np.arange(n, dtype=np.uint32)
    ka = np.repeat(k, n)
    kb = np.tile(k, n)
    A, B = [], []
    for ea, eb in exps:
        for sa in (0, 1):
            for sb in (0, 1):
                low_a = rng.integers(0, 1 << (23 - m), ka.size, dtype=np.uint32)
                low_b = rng.integers(0, 1 << (23 - m), kb.size, dtype=np.uint32)
                A.append((np.uint32(sa) << 31) | (np.uint32(ea) << 23) | (ka << (23 - m)) | low_a)
                B.append((np.uint32(sb) << 31) | (np.uint32(eb) << 23) | (kb << (23 - m)) | low_b)
    return np.concatenate(A).view(np.float32), np.concatenate(B).view(np.float32)


def special_cross():
    s = special_values()
    return np.repeat(s, s.size), np.tile(s, s.size)


def random_bits(n, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2 ** 32, n, dtype=np.uint64).astype(np.uint32).view(np.float32)


def outer_operands(m, seed):
    """Column/row operand vectors whose outer product covers every mantissa pair at several
    exponent/sign combinations: A is (rows x 1), B is (1 x cols)."""
    rng = np.random.default_rng(seed)
    n = 1 << m
    k = np.arange(n, dtype=np.uint32)
    if n > 256:  # wide tables: a random subset of mantissa fields per operand
        k = np.sort(rng.choice(n, 256, replace=False)).astype(np.uint32)

    def vec(exps):
        parts = []
        for e in exps:
            for s in (0, 1):
                low = rng.integers(0, 1 << (23 - m), k.size, dtype=np.uint32)
                parts.append((np.uint32(s) << 31) | (np.uint32(e) << 23) | (k << (23 - m)) | low)
        return np.concatenate(parts).view(np.float32)

    a = vec([127, 100, 160, 2, 250])
    b = vec([127, 150, 90, 126, 5])
    return a.reshape(-1, 1), b.reshape(1, -1)
