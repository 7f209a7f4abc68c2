"""MI355X-native InKAN KAN-layer forward.

The compute lives in ``libkan.so`` (hand-written HIP kernels for gfx950 behind
a C ABI declared in ``include/kan.h``).  ``paper_2609_01956_amd.binding``
exposes the same entry points to Python and marshals torch tensors into them;
importing this package does not load the library, the first call does, and
it raises if the library is missing.
"""
__all__ = ["binding", "workloads"]


def __getattr__(name):
    if name in ("binding", "workloads"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
