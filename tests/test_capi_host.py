"""Host-side checks of the C ABI (no GPU): the library loads, exports what include/amsim.h
declares, builds tables that match the oracle and the closed forms, validates arguments and
reads/writes table files.  No device entry point is called past its argument checks."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from closed_forms import exact_lut_closed_form, mitchell_lut_closed_form
from paper_2209_04161_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(binding.library_path()):
        from paper_2209_04161_amd import build
        build.build()
    return binding.lib()


def _declared_functions():
    with open(os.path.join(ROOT, "include", "amsim.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^(?:const\s+)?(?:int|float|void|char|size_t|uint32_t)\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert "approx_gemm" in names and "lut_build" in names and len(names) >= 14
    for n in names:
        assert hasattr(L, n), n


def test_status_strings(L):
    for code in (0, -1, -2, -3, -4, -5, -6, 7):
        assert isinstance(binding.amsim_status_string(code), str)


@pytest.mark.parametrize("m", list(range(1, 12)))
def test_lut_build_matches_closed_form_and_oracle(L, m):
    t_mit = binding.lut_build(m, "mitchell")
    t_ex = binding.lut_build(m, "exact_trunc")
    assert np.array_equal(t_mit, mitchell_lut_closed_form(m))
    assert np.array_equal(t_ex, exact_lut_closed_form(m))
    if m <= 9:
        assert np.array_equal(t_mit, oracle.lut(oracle.MITCHELL, m))
        assert np.array_equal(t_ex, oracle.lut(oracle.EXACT_TRUNC, m))


def test_lut_build_python_model_and_asymmetric_order(L):
    """A Python functional model goes through the same ABI; the first operand is the high index."""
    m = 4

    def asym(a, b):  # a truncated to M bits, b to M-1 bits, exact product
        ua = np.float32(a).view(np.uint32) & np.uint32((0xFFFFFFFF << (23 - m)) & 0xFFFFFFFF)
        ub = np.float32(b).view(np.uint32) & np.uint32((0xFFFFFFFF << (24 - m)) & 0xFFFFFFFF)
        return float(ua.view(np.float32) * ub.view(np.float32))

    t = binding.lut_build(m, asym)
    assert np.array_equal(t, oracle.lut(oracle.ASYM, m))


def test_lut_build_rejects_unrepresentable_models(L):
    with pytest.raises(binding.AmsimError) as e:
        binding.lut_build(5, lambda a, b: a * b * 0.25)   # exponent borrow: not a carry
    assert e.value.status == binding.AMSIM_ERR_MODEL
    with pytest.raises(binding.AmsimError) as e:
        binding.lut_build(5, lambda a, b: abs(a * b))      # sign not the XOR
    assert e.value.status == binding.AMSIM_ERR_MODEL

    def exp_dependent(a, b):  # mantissa depends on the exponent: not a table model
        p = np.float32(a) * np.float32(b)
        return float(p * np.float32(1.0625)) if abs(p) > 1e10 else float(p)
    with pytest.raises(binding.AmsimError) as e:
        binding.lut_build(3, exp_dependent)
    assert e.value.status == binding.AMSIM_ERR_MODEL


def test_lut_build_argument_errors(L):
    out = np.zeros(16, np.uint32)
    ctx = ctypes.c_int(2)
    p = out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))
    fn = ctypes.cast(L.amsim_model_mitchell, ctypes.c_void_p)
    assert L.lut_build(0, fn, ctypes.cast(ctypes.byref(ctx), ctypes.c_void_p), p, 16) == binding.AMSIM_ERR_UNSUPPORTED
    assert L.lut_build(12, fn, None, p, 16) == binding.AMSIM_ERR_UNSUPPORTED
    assert L.lut_build(2, None, None, p, 16) == binding.AMSIM_ERR_INVALID_ARG
    assert L.lut_build(2, fn, ctypes.cast(ctypes.byref(ctx), ctypes.c_void_p), None, 16) == binding.AMSIM_ERR_INVALID_ARG
    assert L.lut_build(2, fn, ctypes.cast(ctypes.byref(ctx), ctypes.c_void_p), p, 15) == binding.AMSIM_ERR_INVALID_ARG
    assert L.lut_build(2, fn, ctypes.cast(ctypes.byref(ctx), ctypes.c_void_p), p, 16) == binding.AMSIM_OK


def test_builtin_models_direct(L):
    assert binding.model_value("mitchell", 7, 1.5, 1.5) == 2.0
    assert binding.model_value("exact_trunc", 7, 1.5, 1.5) == 2.25
    assert binding.model_value("mitchell", 7, -3.0, 0.5) == -1.5


def test_lut_file_roundtrip(L, tmp_path):
    t = binding.lut_build(6, "mitchell")
    p = str(tmp_path / "mit6.amlt")
    binding.lut_save(p, 6, t)
    assert os.path.getsize(p) == 16 + 4 * (1 << 12)
    m, t2 = binding.lut_load(p)
    assert m == 6 and np.array_equal(t, t2)
    bad = str(tmp_path / "bad.amlt")
    with open(bad, "wb") as f:
        f.write(b"XXXX" + bytes(12))
    with pytest.raises(binding.AmsimError) as e:
        binding.lut_load(bad)
    assert e.value.status == binding.AMSIM_ERR_IO


def test_workspace_size_queries(L):
    assert binding.amsim_gemm_workspace_size(0, 0, 0, 5, 5, 7) == 0
    assert binding.amsim_gemm_workspace_size(0, 0, 64, 64, 64, 7) >= 65536 + 2 * 64 * 64 * 4
    assert binding.amsim_gemm_workspace_size(0, 0, 64, 64, 64, 11) >= 2 * 64 * 64 * 4
    d = dict(n=2, h=8, w=8, c_in=3, c_out=4, kh=3, kw=3, stride_h=1, stride_w=1,
             pad_top=1, pad_bottom=1, pad_left=1, pad_right=1)
    for p in (0, 1, 2):
        assert binding.amsim_conv2d_workspace_size(d, p, 7) > 0
    with pytest.raises(binding.AmsimError):
        binding.amsim_conv2d_workspace_size(d, 3, 7)
    with pytest.raises(binding.AmsimError):
        binding.amsim_conv2d_workspace_size(dict(d, kh=11), 0, 7)   # kernel larger than padded image
    # the width limit of the channel-inside-row decode (w and OW below 4096)
    # (this 1 x 1 pass runs as its GEMM, a one-step outer product that needs no workspace)
    wide = dict(d, n=1, h=1, w=4095, c_in=1, c_out=1, kh=1, kw=1, pad_top=0, pad_bottom=0, pad_left=0, pad_right=0)
    assert binding.amsim_conv2d_workspace_size(wide, 0, 7) == 0
    assert binding.amsim_conv2d_workspace_size(dict(wide, stride_w=2), 0, 7) > 0  # the convolution path
    with pytest.raises(binding.AmsimError):
        binding.amsim_conv2d_workspace_size(dict(wide, w=4096), 0, 7)
    # single-channel x: its 12-byte step-pair records (one per pixel) must stay below 2^31 bytes,
    # though the tensor itself is under 2^29 elements
    one = dict(wide, n=16, h=2048, w=2047, stride_h=4, stride_w=4)
    assert binding.amsim_conv2d_workspace_size(one, 0, 7) > 16 * 2048 * 2047 * 12
    with pytest.raises(binding.AmsimError):
        binding.amsim_conv2d_workspace_size(dict(one, n=90), 0, 7)   # 4.5 GB of records
    with pytest.raises(binding.AmsimError):
        binding.amsim_gemm_workspace_size(0, 0, 4, 4, 4, 12)


def test_workspace_covers_the_unfolded_conv_paths(L):
    """Few input channels: the forward pass's workspace holds x unfolded along w as step-pair
    records (12 bytes per output column and channel pair of kw * c), the backward-data pass's the
    unfolded input's gradient (4 bytes per output column and kw * c channel)."""
    stem = dict(n=32, h=224, w=224, c_in=3, c_out=64, kh=7, kw=7, stride_h=2, stride_w=2,
                pad_top=3, pad_bottom=3, pad_left=3, pad_right=3)
    hp, ow = 224 + 6, (224 + 6 - 7) // 2 + 1
    assert binding.amsim_conv2d_workspace_size(stem, 0, 7) >= 32 * hp * ow * ((7 * 3 + 1) // 2) * 12
    assert binding.amsim_conv2d_workspace_size(stem, 1, 7) >= 32 * 224 * ow * 7 * 3 * 4


def test_device_entry_points_reject_bad_arguments_before_launching(L):
    """Argument checks return before any HIP call, so these run without a GPU."""
    vp = ctypes.c_void_p
    fake = vp(4096)
    assert L.approx_gemm(0, 0, 4, 4, 4, fake, 4, fake, 4, fake, 4, fake, 0, None, 0, None) == binding.AMSIM_ERR_UNSUPPORTED
    assert L.approx_gemm(0, 0, -1, 4, 4, fake, 4, fake, 4, fake, 4, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
    assert L.approx_gemm(0, 0, 4, 4, 4, fake, 4, fake, 4, fake, 3, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
    assert L.approx_gemm(0, 0, 4, 4, 4, fake, 3, fake, 4, fake, 4, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
    assert L.approx_gemm(0, 0, 4, 4, 4, None, 4, fake, 4, fake, 4, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
    assert L.approx_gemm(0, 0, 4, 4, 4, fake, 4, fake, 4, fake, 4, fake, 7, None, 0, None) == binding.AMSIM_ERR_WORKSPACE
    assert L.approx_gemm(0, 0, 0, 4, 4, None, 4, None, 4, None, 4, None, 7, None, 0, None) == binding.AMSIM_OK
    s = binding.conv_desc_struct(dict(n=1, h=4, w=4, c_in=1, c_out=1, kh=3, kw=3, stride_h=1, stride_w=1,
                                      pad_top=0, pad_bottom=0, pad_left=0, pad_right=0))
    for fn in (L.approx_conv2d_fwd, L.approx_conv2d_bwd_data, L.approx_conv2d_bwd_weight):
        assert fn(ctypes.byref(s), fake, fake, fake, fake, 7, None, 0, None) == binding.AMSIM_ERR_WORKSPACE
        assert fn(ctypes.byref(s), None, fake, fake, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
        assert fn(ctypes.byref(s), fake, fake, fake, fake, 0, None, 0, None) == binding.AMSIM_ERR_UNSUPPORTED
        assert fn(None, fake, fake, fake, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
    bad = binding.conv_desc_struct(dict(n=1, h=4, w=4, c_in=1, c_out=1, kh=3, kw=3, stride_h=0, stride_w=1,
                                        pad_top=0, pad_bottom=0, pad_left=0, pad_right=0))
    assert L.approx_conv2d_fwd(ctypes.byref(bad), fake, fake, fake, fake, 7, None, 0, None) == binding.AMSIM_ERR_INVALID_ARG
    assert L.approx_mul_ew(4, None, fake, fake, fake, 7, None) == binding.AMSIM_ERR_INVALID_ARG
    assert L.approx_mul_ew(4, fake, fake, fake, fake, 12, None) == binding.AMSIM_ERR_UNSUPPORTED
    assert L.approx_mul_ew(0, None, None, None, None, 7, None) == binding.AMSIM_OK
    # the kernel timer's kind mask: at least one kind, none beyond the last
    assert L.amsim_profile_start_kinds(0, 1) == binding.AMSIM_ERR_INVALID_ARG
    assert L.amsim_profile_start_kinds(8, 0) == binding.AMSIM_ERR_INVALID_ARG
    assert L.amsim_profile_start_kinds(8, 1 << 8) == binding.AMSIM_ERR_INVALID_ARG
    direct = L.approx_gemm_direct
    assert direct(2, 7, 4, 4, 4, fake, 4, fake, 4, fake, 4, None) == binding.AMSIM_ERR_INVALID_ARG
    assert direct(binding.AMSIM_DIRECT_MITCHELL, 12, 4, 4, 4, fake, 4, fake, 4, fake, 4, None) == binding.AMSIM_ERR_UNSUPPORTED
    assert direct(binding.AMSIM_DIRECT_NATIVE, 0, 4, 4, 4, None, 4, fake, 4, fake, 4, None) == binding.AMSIM_ERR_INVALID_ARG
    assert direct(binding.AMSIM_DIRECT_NATIVE, 0, 4, 4, 4, fake, 3, fake, 4, fake, 4, None) == binding.AMSIM_ERR_INVALID_ARG
    assert direct(binding.AMSIM_DIRECT_NATIVE, 0, 4, 4, 4, fake, 4, fake, 4, fake, 3, None) == binding.AMSIM_ERR_INVALID_ARG
    assert direct(binding.AMSIM_DIRECT_NATIVE, 0, 0, 4, 4, None, 4, None, 4, None, 4, None) == binding.AMSIM_OK


def test_product_path_does_not_touch_the_oracle():
    """The library and binding neither link nor import the oracle."""
    pkg = os.path.join(ROOT, "paper_2209_04161_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")):
                with open(os.path.join(dirpath, fn)) as f:
                    text = f.read()
                assert "import oracle" not in text and "from oracle" not in text, fn
                assert "amsim_oracle" not in text and "orc_" not in text, fn
