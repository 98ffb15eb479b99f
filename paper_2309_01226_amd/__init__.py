"""MI355X (gfx950) fine-tuning-step library: hand-written HIP kernels behind a
C ABI (include/saturn.h), driven from Python through a thin ctypes binding.

The library is loaded on first use, not at import time, so that the seeded
input generators and configuration presets can be imported without a GPU.
"""

from .configs import PRESETS, grid_members, preset  # noqa: F401
