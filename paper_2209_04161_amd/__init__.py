"""MI355X-native approximate-multiplier GEMM and convolution (ApproxTrain's AMSim hot path).

The compute lives in ``libamsim.so`` (HIP kernels for gfx950 behind a C ABI declared in
``include/amsim.h``).  ``paper_2209_04161_amd.binding`` marshals torch tensors into that ABI.
Submodules are imported on first use so that ``paper_2209_04161_amd.workloads`` can be used
without loading the library.
"""
import importlib

__all__ = ["binding", "workloads"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(__name__ + "." + name)
    raise AttributeError(name)
