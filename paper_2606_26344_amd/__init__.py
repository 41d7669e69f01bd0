"""SiLU Gated MLP, Y = (silu(X Wg) * (X Wu)) Wd, on AMD MI355X (gfx950).

The compute path is the HIP library ``libgmlp.so`` behind the C ABI declared
in ``include/gmlp.h``; :mod:`paper_2606_26344_amd.gmlp` is a thin ctypes
binding (argument marshalling only; PyTorch supplies device memory and
streams).  :mod:`paper_2606_26344_amd.inputs` draws seeded synthetic inputs.
Submodules are imported lazily so that the input generator can be used
without loading the GPU library.
"""
import importlib

__all__ = ["gmlp", "inputs", "build"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module("." + name, __name__)
    raise AttributeError(name)
