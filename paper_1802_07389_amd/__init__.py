"""3LC compression hot path for MI355X (gfx950).

``paper_1802_07389_amd.tlc`` is the ctypes binding of the HIP library
``libtlc.so``; it is imported on first use so that ``workloads`` (seeded
input generators) can be used without a GPU.
"""
import importlib

__all__ = ["tlc", "workloads"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
