"""MI355X-native hot path of Polestar's cached denoising step.

The compute lives in `libpolestar.so` (hand-written HIP for gfx950 behind a
C ABI, declared in include/polestar.h).  `polestar` is the thin ctypes
binding; importing this package does not load the library, so the input
generators in `inputs` work on machines without a GPU.
"""

__all__ = ["inputs", "polestar"]
