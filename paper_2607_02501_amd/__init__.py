"""MI355X-native block-quantized linear layers (Q8_0 / Q4_0) for batch-1
embodied-model inference.

Submodules:
  eb        -- Python binding of the C-ABI library libeb.so (HIP kernels for gfx950)
  workloads -- seeded synthetic inputs and workload shapes
  build     -- compiles libeb.so with hipcc

Importing the package loads nothing native; ``paper_2607_02501_amd.eb`` loads
libeb.so and raises if it has not been built.
"""
import importlib

__all__ = ["eb", "workloads", "build"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module("." + name, __name__)
    raise AttributeError(name)
