"""PACE (Pixel-Adaptive Condense and Extract) hot path for AMD MI355X (gfx950).

The compute lives in ``libpace.so`` (hand-written HIP behind a C ABI, declared in
``include/pace.h``).  ``paper_2608_27206_amd.pace`` is the thin ctypes binding that
passes torch device pointers and the current HIP stream to it.  ``workloads``
draws the seeded synthetic inputs.  Submodules are imported on first use.
"""
import importlib

__all__ = ["pace", "workloads", "build"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
