"""MI355X-native quantized self-speculative decoding (EfficientRollout hot path).

The engine is the gfx950 HIP library behind ``include/sd_api.h``; ``sdrl``
is its Python binding and ``synth`` the seeded synthetic input generator.
"""
from . import synth  # noqa: F401

__all__ = ["synth", "sdrl"]
