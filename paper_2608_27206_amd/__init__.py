"""PACE (Pixel-Adaptive Condense and Extract) hot path for AMD MI355X (gfx950).

The compute lives in ``libpace.so`` (hand-written HIP behind a C ABI, declared in
``include/pace.h``).  ``paper_2608_27206_amd.pace`` is the thin ctypes binding that
passes torch device pointers and the current HIP stream to it.  ``workloads``
draws the seeded synthetic inputs.
"""
__all__ = ["pace", "workloads"]


def __getattr__(name):
    if name == "pace":
        from . import pace as _p
        return _p
    if name == "workloads":
        from . import workloads as _w
        return _w
    raise AttributeError(name)
