"""Parity bar shared by the GPU tests.

Products must be bit-exact (any NaN equals any NaN).  Sums may differ from the oracle's
(exactly rounded, double-accumulated) result by the FP32 accumulation-order error: per output
|gpu - oracle| <= 1e-5 * sum_k |product_k| + 2^-126 (the absolute floor covers denormal
partial sums that FP32 flushes to zero); Inf/NaN must match in class and sign.
"""
import numpy as np

REL_TOL = 1e-5
ABS_FLOOR = 2.0 ** -126


def assert_bits_equal(got, want, what=""):
    got = np.asarray(got, dtype=np.float32).reshape(-1)
    want = np.asarray(want, dtype=np.float32).reshape(-1)
    assert got.shape == want.shape
    same = (got.view(np.uint32) == want.view(np.uint32)) | (np.isnan(got) & np.isnan(want))
    if not same.all():
        bad = np.nonzero(~same)[0][:8]
        raise AssertionError("%s: %d of %d products differ, e.g. idx %s got %s want %s" % (
            what, int((~same).sum()), same.size, bad.tolist(), got[bad].view(np.uint32).tolist(),
            want[bad].view(np.uint32).tolist()))


def assert_within_tolerance(got, want, sabs, what=""):
    got = np.asarray(got, dtype=np.float32).reshape(-1)
    want = np.asarray(want, dtype=np.float32).reshape(-1)
    sabs = np.asarray(sabs, dtype=np.float64).reshape(-1)
    assert got.shape == want.shape == sabs.shape, (got.shape, want.shape, sabs.shape)
    fin_w = np.isfinite(want)
    fin_g = np.isfinite(got)
    cls = (fin_w == fin_g) & (np.isnan(want) == np.isnan(got))
    cls &= ~(np.isinf(want) & (got != want))
    err = np.abs(got.astype(np.float64) - want.astype(np.float64))
    tol = REL_TOL * sabs + ABS_FLOOR
    ok = cls & np.where(fin_w & fin_g, err <= tol, True)
    if not ok.all():
        bad = np.nonzero(~ok)[0][:8]
        raise AssertionError("%s: %d of %d outputs out of tolerance, e.g. idx %s got %s want %s sabs %s" % (
            what, int((~ok).sum()), ok.size, bad.tolist(), got[bad].tolist(), want[bad].tolist(),
            sabs[bad].tolist()))
    rel = np.where(sabs > 0, err / np.maximum(sabs, 1e-300), 0.0)
    return float(rel[fin_w & fin_g].max()) if (fin_w & fin_g).any() else 0.0
