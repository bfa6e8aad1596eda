"""MI355X-native hot path of iFVS filtered vector search.

The product is libifvs.so (HIP kernels for gfx950 behind the C ABI in
include/ifvs.h); ``paper_2607_22922_amd.ifvs`` is its Python binding.  The
binding is imported lazily so that ``python -m paper_2607_22922_amd.build``
works before the library exists.
"""
import importlib

__all__ = ["ifvs", "build"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
