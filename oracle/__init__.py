"""CPU oracle for the approximate-multiplier GEMM / convolution path (TEST INFRASTRUCTURE).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may import this
package.  It wraps ``amsim_oracle.c`` (plain C, double accumulation, direct model calls, no
lookup table) with numpy-facing helpers.  It imports nothing from the product package.
"""
import ctypes
import os

import numpy as np

from . import build_oracle

MITCHELL = 0      # Mitchell logarithmic multiplier on M-bit truncated operands
EXACT_TRUNC = 1   # exact product of M-bit truncated operands (bfloat16 truncation at M = 7)
ASYM = 2          # test model: first operand truncated to M bits, second to M-1, exact product

_lib = None


class OrcOpts(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int) for name in ("model", "m_bits", "e_bits", "sat", "native")]


def _opts(model_id, m_bits, e_bits=8, sat=False, native=False):
    return OrcOpts(int(model_id), int(m_bits), int(e_bits), int(bool(sat)), int(bool(native)))


class OrcConv(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int) for name in (
        "n", "h", "w", "c_in", "c_out", "kh", "kw", "stride_h", "stride_w",
        "pad_top", "pad_bottom", "pad_left", "pad_right")]


def lib():
    """Load liboracle.so, compiling it first if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(build_oracle.LIB):
        build_oracle.build()
    L = ctypes.CDLL(build_oracle.LIB)
    f32p = ctypes.POINTER(ctypes.c_float)
    f64p = ctypes.POINTER(ctypes.c_double)
    i64p = ctypes.POINTER(ctypes.c_int64)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    i64 = ctypes.c_int64
    L.orc_model.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_float]
    L.orc_model.restype = ctypes.c_float
    L.orc_mul.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_float]
    L.orc_mul.restype = ctypes.c_float
    L.orc_mul_array.argtypes = [ctypes.c_int, ctypes.c_int, i64, f32p, f32p, f32p]
    L.orc_mul_array.restype = None
    L.orc_lut.argtypes = [ctypes.c_int, ctypes.c_int, u32p]
    L.orc_lut.restype = ctypes.c_int
    L.orc_gemm.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, i64, i64, i64,
                           f32p, i64, f32p, i64, i64p, i64, f32p, f64p]
    L.orc_gemm.restype = None
    L.orc_conv2d.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(OrcConv),
                             f32p, f32p, i64p, i64, f32p, f64p]
    L.orc_conv2d.restype = ctypes.c_int
    op = ctypes.POINTER(OrcOpts)
    L.orc_mul_native.argtypes = [ctypes.c_float, ctypes.c_float]
    L.orc_mul_native.restype = ctypes.c_float
    L.orc_cast.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_float]
    L.orc_cast.restype = ctypes.c_float
    L.orc_mul_fmt.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_float]
    L.orc_mul_fmt.restype = ctypes.c_float
    L.orc_mul_ex_array.argtypes = [op, i64, f32p, f32p, f32p]
    L.orc_mul_ex_array.restype = None
    L.orc_cast_array.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, i64, f32p, f32p]
    L.orc_cast_array.restype = None
    L.orc_gemm_ex.argtypes = [op, ctypes.c_int, ctypes.c_int, i64, i64, i64, f32p, i64, f32p, i64, i64p, i64, f32p,
                              f64p]
    L.orc_gemm_ex.restype = None
    L.orc_conv2d_ex.argtypes = [op, ctypes.c_int, ctypes.POINTER(OrcConv), f32p, f32p, i64p, i64, f32p, f64p]
    L.orc_conv2d_ex.restype = ctypes.c_int
    L.orc_num_threads.argtypes = []
    L.orc_num_threads.restype = ctypes.c_int
    _lib = L
    return L


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def num_threads() -> int:
    return int(lib().orc_num_threads())


def mul(model: int, m_bits: int, a, b) -> np.ndarray:
    """Element-wise approximate product (AMSim semantics) of equal-shape float32 arrays."""
    a = _f32(a)
    b = _f32(b)
    assert a.shape == b.shape
    c = np.empty_like(a)
    lib().orc_mul_array(model, m_bits, a.size, _p(a, ctypes.c_float), _p(b, ctypes.c_float),
                        _p(c, ctypes.c_float))
    return c


def mul_ex(model_id: int, m_bits: int, a, b, e_bits=8, sat=False, native=False) -> np.ndarray:
    """Element-wise product of another multiplier: the table model through Algorithm 2 in a
    (1, e_bits, m) format (e_bits = 8: mul), or the native FP32 multiply (model ignored)."""
    a = _f32(a)
    b = _f32(b)
    assert a.shape == b.shape
    c = np.empty_like(a)
    o = _opts(model_id, m_bits, e_bits, sat, native)
    lib().orc_mul_ex_array(ctypes.byref(o), a.size, _p(a, ctypes.c_float), _p(b, ctypes.c_float),
                           _p(c, ctypes.c_float))
    return c


def cast(e_bits: int, x, sat=False, m_bits=7) -> np.ndarray:
    """The exponent-casting function of a (1, e_bits, m_bits) format, element-wise."""
    x = _f32(x)
    y = np.empty_like(x)
    lib().orc_cast_array(int(e_bits), int(bool(sat)), int(m_bits), x.size, _p(x, ctypes.c_float),
                         _p(y, ctypes.c_float))
    return y


def mul_native(a: float, b: float) -> float:
    return float(lib().orc_mul_native(a, b))


def model(model_id: int, m_bits: int, a: float, b: float) -> float:
    return float(lib().orc_model(model_id, m_bits, a, b))


def lut(model_id: int, m_bits: int) -> np.ndarray:
    """Algorithm 1 table: uint32[2^(2M)], entry k*2^M + j = carry << 23 | mantissa."""
    out = np.empty(1 << (2 * m_bits), dtype=np.uint32)
    rc = lib().orc_lut(model_id, m_bits, _p(out, ctypes.c_uint32))
    if rc != 0:
        raise ValueError("model not representable by a mantissa table")
    return out


def gemm(model_id, m_bits, A, B, transa=False, transb=False, idx=None, e_bits=8, sat=False, native=False):
    """C = op(A) @ op(B) with approximate products; returns (C float32, S float64 = sum |p|).

    A and B are 2-D float32 arrays as stored (op = transpose when the flag is set).  With
    ``idx`` (flat indices i*N + j) only those outputs are computed and returned as 1-D arrays.
    """
    A = _f32(A)
    B = _f32(B)
    M = A.shape[1] if transa else A.shape[0]
    K = A.shape[0] if transa else A.shape[1]
    Kb = B.shape[1] if transb else B.shape[0]
    N = B.shape[0] if transb else B.shape[1]
    assert K == Kb
    if idx is None:
        C = np.empty((M, N), np.float32)
        S = np.empty((M, N), np.float64)
        ip, n = None, 0
    else:
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        C = np.empty(idx.size, np.float32)
        S = np.empty(idx.size, np.float64)
        ip, n = _p(idx, ctypes.c_int64), idx.size
    o = _opts(model_id, m_bits, e_bits, sat, native)
    lib().orc_gemm_ex(ctypes.byref(o), int(transa), int(transb), M, N, K, _p(A, ctypes.c_float), A.shape[1],
                      _p(B, ctypes.c_float), B.shape[1], ip, n, _p(C, ctypes.c_float), _p(S, ctypes.c_double))
    return C, S


def conv_out_hw(p: dict):
    oh = (p["h"] + p["pad_top"] + p["pad_bottom"] - p["kh"]) // p["stride_h"] + 1
    ow = (p["w"] + p["pad_left"] + p["pad_right"] - p["kw"]) // p["stride_w"] + 1
    return oh, ow


def _conv(model_id, m_bits, pass_id, p, in0, in1, out_shape, idx, e_bits=8, sat=False, native=False):
    d = OrcConv(**{k: int(p[k]) for k, _ in OrcConv._fields_})
    in0 = _f32(in0)
    in1 = _f32(in1)
    if idx is None:
        out = np.empty(out_shape, np.float32)
        S = np.empty(out_shape, np.float64)
        ip, n = None, 0
    else:
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        out = np.empty(idx.size, np.float32)
        S = np.empty(idx.size, np.float64)
        ip, n = _p(idx, ctypes.c_int64), idx.size
    o = _opts(model_id, m_bits, e_bits, sat, native)
    rc = lib().orc_conv2d_ex(ctypes.byref(o), pass_id, ctypes.byref(d), _p(in0, ctypes.c_float),
                             _p(in1, ctypes.c_float), ip, n, _p(out, ctypes.c_float), _p(S, ctypes.c_double))
    assert rc == 0
    return out, S


def conv2d_fwd(model_id, m_bits, p, x, w, idx=None, **mult):
    """y[n,oh,ow,co] (NHWC) from x (NHWC) and w (HWIO); products amul(x, w).  mult: e_bits, sat,
    native, as for gemm."""
    oh, ow = conv_out_hw(p)
    return _conv(model_id, m_bits, 0, p, x, w, (p["n"], oh, ow, p["c_out"]), idx, **mult)


def conv2d_bwd_data(model_id, m_bits, p, dy, w, idx=None, **mult):
    """dx[n,h,w,ci] from dy (NHWC) and w (HWIO); products amul(dy, w)."""
    return _conv(model_id, m_bits, 1, p, dy, w, (p["n"], p["h"], p["w"], p["c_in"]), idx, **mult)


def conv2d_bwd_weight(model_id, m_bits, p, x, dy, idx=None, **mult):
    """dw[kh,kw,ci,co] (HWIO) from x and dy; products amul(x, dy)."""
    return _conv(model_id, m_bits, 2, p, x, dy, (p["kh"], p["kw"], p["c_in"], p["c_out"]), idx, **mult)
