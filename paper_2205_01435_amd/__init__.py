"""MI355X-native World-Model dream library (RLFlow's model-based hot path).

``workloads`` draws the seeded synthetic inputs; ``_lib`` is the thin ctypes
binding of ``libwm.so`` (HIP kernels for gfx950 behind a C ABI, declared in
``include/wm.h``).  The library is loaded on first use and every entry point
raises if it is missing: there is no CPU fallback.
"""

from . import _lib, workloads  # noqa: F401

__all__ = ["_lib", "workloads"]
