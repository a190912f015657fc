"""MarginGate gated-decode hot path for MI355X (gfx950).

The compute lives in the HIP library libmg.so (C ABI declared in include/mg.h);
`paper_2605_30218_amd.mg` is its ctypes binding.  Importing the package loads
nothing; `paper_2605_30218_amd.mg.load()` opens the library and raises if it is
missing.
"""
__all__ = ["synth", "mg"]
