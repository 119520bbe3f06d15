"""libscan: device-wide prefix sums and scan-based operators for one MI355X.

The compute path is the C-ABI library ``libscan.so`` (hand-written HIP for
gfx950, built from ``csrc/``); ``ops`` is a thin ctypes binding over it that
takes torch tensors for device memory and streams.  Importing the package does
not load the library; the first op call does, and fails loudly if it is absent.
"""
import importlib

__all__ = ["ops", "workloads"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
