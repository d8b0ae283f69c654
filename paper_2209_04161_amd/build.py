"""Compile libamsim.so (HIP kernels for gfx950 + host code) in-tree with hipcc.

Flags that matter for the numerics:
  -fgpu-flush-denormals-to-zero   f32 denormal results flush to signed zero; the product
                                  evaluation relies on it for AMSim's zero rule
  -ffp-contract=off               no implicit FMA contraction: every multiply rounds where the
                                  source says so (the only FMA is the explicit accumulate)
  -target-feature -packed-fp32-ops  no packed FP32 instructions
"""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
# (source, extra flags): the table kernels are compiled once per operation (0 GEMM, 1 forward,
# 2 backward data, 3 backward weight), in parallel with the rest.
UNITS = [("amsim_kernels.hip", []), ("amsim_host.cpp", [])] + [
    ("amsim_tab.hip", ["-DAMSIM_TAB_OP=%d" % op]) for op in range(4)]
LIB = os.path.join(HERE, "libamsim.so")
ARCH = os.environ.get("AMSIM_OFFLOAD_ARCH", "gfx950")
FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
         "-fgpu-flush-denormals-to-zero", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def hipcc():
    for cand in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), "hipcc"):
        if os.path.sep not in cand or os.path.exists(cand):
            return cand
    return "hipcc"


def _clean(text):
    # hipcc's host pass does not know the packed-fp32 target feature and says so: harmless.
    return "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)


def build(verbose: bool = False) -> str:
    with tempfile.TemporaryDirectory(prefix="amsim_build_") as tmpdir:
        jobs = []
        for i, (src, extra) in enumerate(UNITS):
            obj = os.path.join(tmpdir, "%d_%s.o" % (i, os.path.splitext(src)[0]))
            cmd = [hipcc()] + FLAGS + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            jobs.append((cmd, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                                    text=True)))
        failed = []
        for cmd, obj, proc in jobs:
            out = _clean(proc.communicate()[0])
            if proc.returncode != 0:
                failed.append(" ".join(cmd) + "\n" + out)
            elif verbose and out.strip():
                print(out)
        if failed:
            raise RuntimeError("hipcc failed:\n" + "\n\n".join(failed))
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = [hipcc(), "--offload-arch=" + ARCH, "--hip-link", "-shared", "-fPIC", "-o", tmp] + [o for _, o, _ in jobs]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        if res.returncode != 0:
            raise RuntimeError("hipcc link failed:\n" + _clean(res.stdout))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
