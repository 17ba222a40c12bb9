"""MI355X-native MeanField joint-configuration search.

`synth` draws seeded instances; `mf` is the binding to the HIP library
(libmf.so), imported on first use so that instance generation works on hosts
without the built library.
"""
import importlib

__all__ = ["synth", "mf"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
