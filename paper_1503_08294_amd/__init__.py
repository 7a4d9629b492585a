"""Multi-signal growing self-organizing network iteration on AMD MI355X (gfx950).

The iteration runs in hand-written HIP kernels behind the C ABI of ``include/gsn.h``
(``libgsn.so``); ``paper_1503_08294_amd.gsn`` is its thin Python binding.  Submodules are
imported on first use, so the input generators in ``clouds`` work without the library.
"""
import importlib


def __getattr__(name):
    if name in ("gsn", "clouds"):
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
