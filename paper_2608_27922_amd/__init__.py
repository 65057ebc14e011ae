"""DensityKV hot path for MI355X (gfx950): density-guided KV bank update and bank attention.

The compute runs in the HIP library ``libdensitykv.so`` behind a C ABI
(``include/densitykv.h``); ``paper_2608_27922_amd.api`` is the thin ctypes
binding with the same entry-point names.  ``synth`` holds the seeded
synthetic inputs.  Importing the package loads nothing; the binding loads the
library on first use and raises if it has not been built.
"""

__all__ = ["api", "synth"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
