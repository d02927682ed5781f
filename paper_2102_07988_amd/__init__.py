"""TeraPipe stage engine for MI355X (gfx950).

One pipeline stage's forward and backward over token slices of a causal-LM
training sequence, a slice-cost profiler and the optimal-slicing DP, behind the
C ABI declared in include/terapipe.h.  ``terapipe`` is the ctypes binding; it
is imported lazily so that the seeded-input module ``synth`` can be used
without loading the GPU library.
"""

__all__ = ["terapipe", "synth"]


def __getattr__(name):
    if name in ("terapipe", "synth"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
