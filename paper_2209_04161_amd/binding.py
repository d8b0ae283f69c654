"""Python binding of libamsim.so (argument marshalling only).

Every function here has the name of the C entry point it calls.  Tensors are torch tensors:
device memory comes from torch, the stream is torch's current stream, and the raw pointers go
through the C ABI.  All computation happens in the library's HIP kernels; if the library is
not built this module raises instead of computing anything another way.
"""
import ctypes
import os

import numpy as np

from . import build as _build

AMSIM_OK = 0
AMSIM_ERR_INVALID_ARG = -1
AMSIM_ERR_UNSUPPORTED = -2
AMSIM_ERR_MODEL = -3
AMSIM_ERR_WORKSPACE = -4
AMSIM_ERR_HIP = -5
AMSIM_ERR_IO = -6
AMSIM_ERR_SCRATCH = -7
AMSIM_NOALLOC_SCRATCH_BYTES = 64 << 20

AMSIM_CONV_FWD = 0
AMSIM_CONV_BWD_DATA = 1
AMSIM_CONV_BWD_WEIGHT = 2
AMSIM_DIRECT_NATIVE = 0
AMSIM_DIRECT_MITCHELL = 1

AMSIM_KERNEL_GEMM = 0
AMSIM_KERNEL_CONV_FWD = 1
AMSIM_KERNEL_CONV_BWD_DATA = 2
AMSIM_KERNEL_CONV_BWD_WEIGHT = 3
KERNEL_KINDS = {"gemm": 0, "conv_fwd": 1, "conv_bwd_data": 2, "conv_bwd_weight": 3,
                "gemm_native": 4, "conv_fwd_native": 5, "conv_bwd_data_native": 6, "conv_bwd_weight_native": 7}

AMSIM_MULTIPLY_TABLE = 0
AMSIM_MULTIPLY_NATIVE = 1
AMSIM_CAST_INF = 0
AMSIM_CAST_SATURATE = 1

MODEL_FN = ctypes.CFUNCTYPE(ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_void_p)


class AmsimError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, amsim_status_string(status), status))


class amsim_conv2d(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int) for name in (
        "n", "h", "w", "c_in", "c_out", "kh", "kw", "stride_h", "stride_w",
        "pad_top", "pad_bottom", "pad_left", "pad_right")]


class amsim_options(ctypes.Structure):
    _fields_ = [("multiply", ctypes.c_int), ("e_bits", ctypes.c_int), ("exp_cast", ctypes.c_int)]


def options(multiply="table", e_bits=8, exp_cast="inf") -> amsim_options:
    """The _ex calls' options: multiply "table" (AMSim) or "native"; e_bits of the (1, e, m)
    format; exp_cast "inf" or "saturate"."""
    mult = {"table": AMSIM_MULTIPLY_TABLE, "native": AMSIM_MULTIPLY_NATIVE}
    cast = {"inf": AMSIM_CAST_INF, "saturate": AMSIM_CAST_SATURATE}
    if multiply not in mult or exp_cast not in cast:
        raise ValueError("multiply must be 'table' or 'native', exp_cast 'inf' or 'saturate'")
    return amsim_options(mult[multiply], int(e_bits), cast[exp_cast])


_lib = None


def library_path() -> str:
    return _build.LIB


def lib():
    """Load the built library (no fallback: a missing library is an error)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError("libamsim.so is not built (%s); run __graft_entry__.build() or "
                           "python -m paper_2209_04161_amd.build" % path)
    L = ctypes.CDLL(path)
    vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    u32p = ctypes.POINTER(ctypes.c_uint32)
    szp = ctypes.POINTER(ctypes.c_size_t)
    cp = ctypes.POINTER(amsim_conv2d)
    op = ctypes.POINTER(amsim_options)
    sigs = {
        "amsim_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "amsim_version": ([], ctypes.c_int),
        "amsim_model_mitchell": ([ctypes.c_float, ctypes.c_float, vp], ctypes.c_float),
        "amsim_model_exact_trunc": ([ctypes.c_float, ctypes.c_float, vp], ctypes.c_float),
        "lut_build": ([ctypes.c_int, vp, vp, u32p, sz], ctypes.c_int),
        "lut_save": ([ctypes.c_char_p, ctypes.c_int, u32p, sz], ctypes.c_int),
        "lut_load": ([ctypes.c_char_p, ctypes.POINTER(ctypes.c_int), u32p, sz], ctypes.c_int),
        "amsim_gemm_workspace_size": ([ctypes.c_int, ctypes.c_int, i64, i64, i64, ctypes.c_int, szp], ctypes.c_int),
        "approx_gemm": ([ctypes.c_int, ctypes.c_int, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp, ctypes.c_int,
                         vp, sz, vp], ctypes.c_int),
        "amsim_conv2d_workspace_size": ([cp, ctypes.c_int, ctypes.c_int, szp], ctypes.c_int),
        "approx_conv2d_fwd": ([cp, vp, vp, vp, vp, ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_conv2d_bwd_data": ([cp, vp, vp, vp, vp, ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_conv2d_bwd_weight": ([cp, vp, vp, vp, vp, ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_mul_ew": ([i64, vp, vp, vp, vp, ctypes.c_int, vp], ctypes.c_int),
        "approx_gemm_noalloc": ([ctypes.c_int, ctypes.c_int, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp,
                                 ctypes.c_int, vp], ctypes.c_int),
        "approx_gemm_ex": ([op, ctypes.c_int, ctypes.c_int, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp,
                            ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_conv2d_fwd_ex": ([op, cp, vp, vp, vp, vp, ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_conv2d_bwd_data_ex": ([op, cp, vp, vp, vp, vp, ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_conv2d_bwd_weight_ex": ([op, cp, vp, vp, vp, vp, ctypes.c_int, vp, sz, vp], ctypes.c_int),
        "approx_mul_ew_ex": ([op, i64, vp, vp, vp, vp, ctypes.c_int, vp], ctypes.c_int),
        "amsim_cast_exponent": ([ctypes.c_int, ctypes.c_int, ctypes.c_int, i64, vp, vp, vp], ctypes.c_int),
        "approx_gemm_direct": ([ctypes.c_int, ctypes.c_int, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp],
                               ctypes.c_int),
        "amsim_profile_start": ([ctypes.c_int], ctypes.c_int),
        "amsim_profile_start_kinds": ([ctypes.c_int, ctypes.c_uint], ctypes.c_int),
        "amsim_profile_stop": ([], ctypes.c_int),
        "amsim_profile_read": ([ctypes.c_int, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)],
                               ctypes.c_int),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def amsim_status_string(status: int) -> str:
    return lib().amsim_status_string(int(status)).decode()


def _check(status, where):
    if status != AMSIM_OK:
        raise AmsimError(status, where)


# ------------------------------------------------------------------ tables ----------------

def _model_pointer(model):
    """Returns (function pointer as void*, keep-alive object)."""
    L = lib()
    if model in ("mitchell", "exact_trunc"):
        fn = getattr(L, "amsim_model_" + model)
        return ctypes.cast(fn, ctypes.c_void_p), fn
    if callable(model):
        cb = MODEL_FN(lambda a, b, ctx: float(model(a, b)))
        return ctypes.cast(cb, ctypes.c_void_p), cb
    raise ValueError("model must be 'mitchell', 'exact_trunc' or a callable (a, b) -> float")


def lut_build(m_bits: int, model="mitchell") -> np.ndarray:
    """Algorithm 1 on the host: uint32[2^(2M)] table for a built-in or Python-callable model."""
    n = 1 << (2 * int(m_bits)) if 1 <= int(m_bits) <= 11 else 0
    out = np.zeros(max(n, 1), dtype=np.uint32)
    fptr, keep = _model_pointer(model)
    ctx = ctypes.c_int(int(m_bits))
    status = lib().lut_build(int(m_bits), fptr, ctypes.cast(ctypes.byref(ctx), ctypes.c_void_p),
                             out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), out.size if n else 0)
    del keep
    _check(status, "lut_build")
    return out


def lut_save(path: str, m_bits: int, table: np.ndarray) -> None:
    table = np.ascontiguousarray(table, dtype=np.uint32)
    _check(lib().lut_save(os.fsencode(path), int(m_bits), table.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
                          table.size), "lut_save")


def lut_load(path: str):
    """Returns (m_bits, table)."""
    m = ctypes.c_int(0)
    _check(lib().lut_load(os.fsencode(path), ctypes.byref(m), None, 0), "lut_load")
    out = np.empty(1 << (2 * m.value), dtype=np.uint32)
    _check(lib().lut_load(os.fsencode(path), ctypes.byref(m), out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
                          out.size), "lut_load")
    return m.value, out


def model_value(model: str, m_bits: int, a: float, b: float) -> float:
    """Call a built-in functional model directly (host)."""
    ctx = ctypes.c_int(int(m_bits))
    fn = getattr(lib(), "amsim_model_" + model)
    return float(fn(a, b, ctypes.cast(ctypes.byref(ctx), ctypes.c_void_p)))


# ------------------------------------------------------------------ device calls ----------

def _torch():
    import torch
    return torch


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def device_lut(table: np.ndarray, device="cuda"):
    """Upload a table to the device as an int32 tensor holding the uint32 bits."""
    torch = _torch()
    return torch.from_numpy(np.ascontiguousarray(table, dtype=np.uint32).view(np.int32)).to(device)


def _check_f32(t, name, shape=None, device=None):
    torch = _torch()
    if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
        raise ValueError("%s must be a contiguous float32 CUDA tensor" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, the call needs %s" % (name, tuple(t.shape), tuple(shape)))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, the call's operands on %s" % (name, t.device, device))


def _check_lut(lut, m_bits, device=None, native=False):
    torch = _torch()
    if native and lut is None:
        return
    if lut.dtype not in (torch.int32,) or not lut.is_cuda or lut.numel() < (1 << (2 * m_bits)):
        raise ValueError("lut must be an int32 CUDA tensor of 2^(2M) entries")
    if device is not None and lut.device != device:
        raise ValueError("lut is on %s, the call's operands on %s" % (lut.device, device))


def _check_workspace(ws, nbytes, device):
    torch = _torch()
    if ws.dtype != torch.uint8 or not ws.is_cuda or not ws.is_contiguous() or ws.device != device:
        raise ValueError("workspace must be a contiguous uint8 CUDA tensor on %s" % device)
    if ws.numel() < nbytes:
        raise ValueError("workspace holds %d bytes, the call needs %d" % (ws.numel(), nbytes))


def amsim_gemm_workspace_size(trans_a, trans_b, m, n, k, m_bits) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().amsim_gemm_workspace_size(int(trans_a), int(trans_b), m, n, k, int(m_bits), ctypes.byref(b)),
           "amsim_gemm_workspace_size")
    return b.value


def _workspace(nbytes, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _gemm_args(A, B, lut, m_bits, trans_a, trans_b, out, workspace, native=False):
    torch = _torch()
    _check_f32(A, "A")
    _check_f32(B, "B", device=A.device)
    _check_lut(lut, m_bits, A.device, native)
    if A.dim() != 2 or B.dim() != 2:
        raise ValueError("A and B must be 2-D")
    m = A.shape[1] if trans_a else A.shape[0]
    k = A.shape[0] if trans_a else A.shape[1]
    kb = B.shape[1] if trans_b else B.shape[0]
    n = B.shape[0] if trans_b else B.shape[1]
    if k != kb:
        raise ValueError("inner dimensions differ")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    if (out.dtype != torch.float32 or out.device != A.device or out.dim() != 2 or tuple(out.shape) != (m, n)
            or (m > 0 and n > 1 and out.stride(1) != 1) or (m > 1 and out.stride(0) < n)):
        raise ValueError("out must be a float32 (%d, %d) tensor on %s with unit column stride" % (m, n, A.device))
    if workspace is not False:  # False: the call brings no workspace
        ws_bytes = amsim_gemm_workspace_size(trans_a, trans_b, m, n, k, m_bits if not native else 7)
        if workspace is None:
            workspace = _workspace(ws_bytes, A.device)
        _check_workspace(workspace, ws_bytes, A.device)
    ldc = out.stride(0) if m > 1 else n
    return m, n, k, out, ldc, workspace


def approx_gemm(A, B, lut, m_bits, trans_a=False, trans_b=False, out=None, workspace=None):
    """C = op(A) @ op(B) with approximate products (row-major float32 CUDA tensors)."""
    m, n, k, out, ldc, workspace = _gemm_args(A, B, lut, m_bits, trans_a, trans_b, out, workspace)
    _check(lib().approx_gemm(int(trans_a), int(trans_b), m, n, k, _ptr(A), A.shape[1], _ptr(B), B.shape[1],
                             _ptr(out), ldc, _ptr(lut), int(m_bits), _ptr(workspace), workspace.numel(), _stream()),
           "approx_gemm")
    return out


def approx_gemm_noalloc(A, B, lut, m_bits, out, trans_a=False, trans_b=False):
    """approx_gemm on the library's fixed per-GPU scratch buffer, for callers that cannot allocate:
    `out` is required and nothing is allocated.  Raises AmsimError (AMSIM_ERR_SCRATCH) when the
    call needs more than AMSIM_NOALLOC_SCRATCH_BYTES of workspace."""
    if out is None:
        raise ValueError("approx_gemm_noalloc: out is required (the call allocates nothing)")
    m, n, k, out, ldc, _ = _gemm_args(A, B, lut, m_bits, trans_a, trans_b, out, False)
    _check(lib().approx_gemm_noalloc(int(trans_a), int(trans_b), m, n, k, _ptr(A), A.shape[1], _ptr(B), B.shape[1],
                                     _ptr(out), ldc, _ptr(lut), int(m_bits), _stream()), "approx_gemm_noalloc")
    return out


def approx_gemm_ex(A, B, lut, m_bits, trans_a=False, trans_b=False, out=None, workspace=None, multiply="table",
                   e_bits=8, exp_cast="inf"):
    """approx_gemm with options (see options())."""
    opt = options(multiply, e_bits, exp_cast)
    native = multiply == "native"
    m, n, k, out, ldc, workspace = _gemm_args(A, B, lut, m_bits, trans_a, trans_b, out, workspace, native)
    _check(lib().approx_gemm_ex(ctypes.byref(opt), int(trans_a), int(trans_b), m, n, k, _ptr(A), A.shape[1], _ptr(B),
                                B.shape[1], _ptr(out), ldc, _ptr(lut), int(m_bits), _ptr(workspace),
                                workspace.numel(), _stream()), "approx_gemm_ex")
    return out


def approx_gemm_direct(A, B, mode, m_bits=7, out=None):
    """C = A @ B without a table: mode "native" (FP32 multiply) or "mitchell" (Mitchell's
    multiplier on the top m_bits mantissa bits, computed from the operands' bits)."""
    torch = _torch()
    _check_f32(A, "A")
    _check_f32(B, "B", device=A.device)
    modes = {"native": AMSIM_DIRECT_NATIVE, "mitchell": AMSIM_DIRECT_MITCHELL}
    if mode not in modes:
        raise ValueError("mode must be 'native' or 'mitchell'")
    m, k = A.shape
    if B.shape[0] != k:
        raise ValueError("inner dimensions differ")
    n = B.shape[1]
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    if (out.dtype != torch.float32 or out.device != A.device or tuple(out.shape) != (m, n)
            or (n > 1 and out.stride(1) != 1) or (m > 1 and out.stride(0) < n)):
        raise ValueError("out must be a float32 (%d, %d) tensor on %s with unit column stride" % (m, n, A.device))
    _check(lib().approx_gemm_direct(modes[mode], int(m_bits), m, n, k, _ptr(A), A.stride(0), _ptr(B), B.stride(0),
                                    _ptr(out), out.stride(0), _stream()), "approx_gemm_direct")
    return out


def conv_desc_struct(d: dict) -> amsim_conv2d:
    return amsim_conv2d(**{k: int(d[k]) for k, _ in amsim_conv2d._fields_})


def conv_out_hw(d):
    oh = (d["h"] + d["pad_top"] + d["pad_bottom"] - d["kh"]) // d["stride_h"] + 1
    ow = (d["w"] + d["pad_left"] + d["pad_right"] - d["kw"]) // d["stride_w"] + 1
    return oh, ow


def amsim_conv2d_workspace_size(desc: dict, pass_id: int, m_bits: int) -> int:
    b = ctypes.c_size_t(0)
    s = conv_desc_struct(desc)
    _check(lib().amsim_conv2d_workspace_size(ctypes.byref(s), int(pass_id), int(m_bits), ctypes.byref(b)),
           "amsim_conv2d_workspace_size")
    return b.value


def _conv_shapes(desc):
    oh, ow = conv_out_hw(desc)
    x = (desc["n"], desc["h"], desc["w"], desc["c_in"])
    w = (desc["kh"], desc["kw"], desc["c_in"], desc["c_out"])
    y = (desc["n"], oh, ow, desc["c_out"])
    return x, w, y


def _conv_call(fn_name, pass_id, desc, in0, in1, out, lut, m_bits, workspace, opt=None):
    native = opt is not None and opt.multiply == AMSIM_MULTIPLY_NATIVE
    s = conv_desc_struct(desc)
    ws_bytes = amsim_conv2d_workspace_size(desc, pass_id, m_bits if not native else 7)
    if workspace is None:
        workspace = _workspace(ws_bytes, in0.device)
    _check_workspace(workspace, ws_bytes, in0.device)
    if opt is None:
        fn = getattr(lib(), fn_name)
        status = fn(ctypes.byref(s), _ptr(in0), _ptr(in1), _ptr(out), _ptr(lut), int(m_bits), _ptr(workspace),
                    workspace.numel(), _stream())
    else:
        fn_name = fn_name + "_ex"
        fn = getattr(lib(), fn_name)
        status = fn(ctypes.byref(opt), ctypes.byref(s), _ptr(in0), _ptr(in1), _ptr(out), _ptr(lut), int(m_bits),
                    _ptr(workspace), workspace.numel(), _stream())
    _check(status, fn_name)
    return out


def _conv_pass(pass_id, desc, in0, in1, lut, m_bits, out, workspace, opt):
    torch = _torch()
    xs, ws_, ys = _conv_shapes(desc)
    shapes = {AMSIM_CONV_FWD: (("x", xs), ("w", ws_), ys), AMSIM_CONV_BWD_DATA: (("dy", ys), ("w", ws_), xs),
              AMSIM_CONV_BWD_WEIGHT: (("x", xs), ("dy", ys), ws_)}[pass_id]
    (n0, s0), (n1, s1), so = shapes
    native = opt is not None and opt.multiply == AMSIM_MULTIPLY_NATIVE
    _check_f32(in0, n0, s0)
    _check_f32(in1, n1, s1, in0.device)
    _check_lut(lut, m_bits, in0.device, native)
    if out is None:
        out = torch.empty(so, dtype=torch.float32, device=in0.device)
    _check_f32(out, "out", so, in0.device)
    name = {AMSIM_CONV_FWD: "approx_conv2d_fwd", AMSIM_CONV_BWD_DATA: "approx_conv2d_bwd_data",
            AMSIM_CONV_BWD_WEIGHT: "approx_conv2d_bwd_weight"}[pass_id]
    return _conv_call(name, pass_id, desc, in0, in1, out, lut, m_bits, workspace, opt)


def approx_conv2d_fwd(desc, x, w, lut, m_bits, out=None, workspace=None):
    """y (NHWC) from x (NHWC) and w (HWIO)."""
    return _conv_pass(AMSIM_CONV_FWD, desc, x, w, lut, m_bits, out, workspace, None)


def approx_conv2d_bwd_data(desc, dy, w, lut, m_bits, out=None, workspace=None):
    """dx (NHWC) from dy (NHWC) and w (HWIO)."""
    return _conv_pass(AMSIM_CONV_BWD_DATA, desc, dy, w, lut, m_bits, out, workspace, None)


def approx_conv2d_bwd_weight(desc, x, dy, lut, m_bits, out=None, workspace=None):
    """dw (HWIO) from x (NHWC) and dy (NHWC)."""
    return _conv_pass(AMSIM_CONV_BWD_WEIGHT, desc, x, dy, lut, m_bits, out, workspace, None)


def approx_conv2d_fwd_ex(desc, x, w, lut, m_bits, out=None, workspace=None, multiply="table", e_bits=8,
                         exp_cast="inf"):
    return _conv_pass(AMSIM_CONV_FWD, desc, x, w, lut, m_bits, out, workspace, options(multiply, e_bits, exp_cast))


def approx_conv2d_bwd_data_ex(desc, dy, w, lut, m_bits, out=None, workspace=None, multiply="table", e_bits=8,
                              exp_cast="inf"):
    return _conv_pass(AMSIM_CONV_BWD_DATA, desc, dy, w, lut, m_bits, out, workspace,
                      options(multiply, e_bits, exp_cast))


def approx_conv2d_bwd_weight_ex(desc, x, dy, lut, m_bits, out=None, workspace=None, multiply="table", e_bits=8,
                                exp_cast="inf"):
    return _conv_pass(AMSIM_CONV_BWD_WEIGHT, desc, x, dy, lut, m_bits, out, workspace,
                      options(multiply, e_bits, exp_cast))


def approx_mul_ew(a, b, lut, m_bits, out=None):
    torch = _torch()
    _check_f32(a, "a")
    _check_f32(b, "b", tuple(a.shape), a.device)
    _check_lut(lut, m_bits, a.device)
    if out is None:
        out = torch.empty_like(a)
    _check_f32(out, "out", tuple(a.shape), a.device)
    _check(lib().approx_mul_ew(a.numel(), _ptr(a), _ptr(b), _ptr(out), _ptr(lut), int(m_bits), _stream()),
           "approx_mul_ew")
    return out


def approx_mul_ew_ex(a, b, lut, m_bits, out=None, e_bits=8, exp_cast="inf"):
    torch = _torch()
    _check_f32(a, "a")
    _check_f32(b, "b", tuple(a.shape), a.device)
    _check_lut(lut, m_bits, a.device)
    if out is None:
        out = torch.empty_like(a)
    _check_f32(out, "out", tuple(a.shape), a.device)
    opt = options("table", e_bits, exp_cast)
    _check(lib().approx_mul_ew_ex(ctypes.byref(opt), a.numel(), _ptr(a), _ptr(b), _ptr(out), _ptr(lut), int(m_bits),
                                  _stream()), "approx_mul_ew_ex")
    return out


def amsim_cast_exponent(x, e_bits, exp_cast="inf", m_bits=7, out=None):
    """x cast to the (1, e_bits, m_bits) format's range, as FP32 values."""
    torch = _torch()
    _check_f32(x, "x")
    cast = {"inf": AMSIM_CAST_INF, "saturate": AMSIM_CAST_SATURATE}[exp_cast]
    if out is None:
        out = torch.empty_like(x)
    _check_f32(out, "out", tuple(x.shape), x.device)
    _check(lib().amsim_cast_exponent(int(e_bits), cast, int(m_bits), x.numel(), _ptr(x), _ptr(out), _stream()),
           "amsim_cast_exponent")
    return out


# ------------------------------------------------------------------ kernel timing --------

def amsim_profile_start(max_launches: int = 4096, kinds=None) -> None:
    """Start timing main-kernel launches; kinds: names or AMSIM_KERNEL_* values to time (default all)."""
    if kinds is None:
        _check(lib().amsim_profile_start(int(max_launches)), "amsim_profile_start")
        return
    mask = 0
    for k in kinds:
        mask |= 1 << (KERNEL_KINDS[k] if isinstance(k, str) else int(k))
    _check(lib().amsim_profile_start_kinds(int(max_launches), mask), "amsim_profile_start_kinds")


def amsim_profile_stop() -> None:
    _check(lib().amsim_profile_stop(), "amsim_profile_stop")


def amsim_profile_read(kind) -> tuple:
    """(launches, total_ms) of one main-kernel kind since the last amsim_profile_start."""
    if isinstance(kind, str):
        kind = KERNEL_KINDS[kind]
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0.0)
    _check(lib().amsim_profile_read(int(kind), ctypes.byref(n), ctypes.byref(ms)), "amsim_profile_read")
    return n.value, ms.value
