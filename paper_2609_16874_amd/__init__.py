"""MI355X (gfx950) decoder for sinusoidal centroid positional encodings.

``native`` binds the C ABI of ``libcpe_decode.so`` (declared in
``include/cpe_decode.h``); ``synth`` draws seeded synthetic frames;
``build`` compiles the HIP library.
"""
from . import synth  # noqa: F401

__all__ = ["synth", "native", "build"]
