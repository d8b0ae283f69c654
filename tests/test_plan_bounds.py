"""Host-side bounds harness of the launch planning and the table kernels' tap arithmetic, built
with the address and undefined-behaviour sanitizers (no GPU): over 10^4 seeded GEMM shapes and
10^4 seeded convolution descriptors (every pass) within the library's limits, every workspace
region, grid dimension, first-operand byte offset a tap can form, second-operand row and result
offset stays inside its buffer, with no overflow of the 32-bit forms the kernels use.  See
tests/bounds/plan_bounds_harness.hip."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SRC = os.path.join(ROOT, "tests", "bounds", "plan_bounds_harness.hip")


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    if not (os.path.exists(HIPCC) or shutil.which("hipcc")):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("bounds") / "plan_bounds_harness")
    # host-only build: the sanitizers apply to host code (each -fsanitize= behind -Xarch_host)
    cmd = [HIPCC, "-x", "hip", "--cuda-host-only", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2209_04161_amd", "csrc"),
           SRC, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


@pytest.mark.parametrize("seed", [1, 2])
def test_plans_and_taps_stay_in_bounds(harness, seed):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([harness, "10000", "10000", str(seed)], capture_output=True, text=True, timeout=600, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    line = [ln for ln in r.stdout.splitlines() if ln.startswith("OK ")]
    assert line, out[-4000:]
    fields = dict(kv.split("=") for kv in line[0].split()[1:])
    assert int(fields["gemm_cases"]) == 10000 and int(fields["conv_cases"]) == 10000
    # the sampled shapes reach the 32-bit offset range the kernels rely on
    assert int(fields["max_a_bytes"]) > 2 ** 31, line[0]
    # stride-1 backward-data passes that take the forward route are among them
    assert int(fields["bwd_data_as_fwd"]) > 100, line[0]
