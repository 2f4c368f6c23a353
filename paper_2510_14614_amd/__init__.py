"""MI355X-native FAL / FAL+ training hot path (arXiv 2510.14614).

The compute lives in ``libfal.so`` (HIP kernels for gfx950 behind a C ABI,
declared in ``include/fal.h``); ``paper_2510_14614_amd.fal`` is the thin
ctypes binding.  Importing this package does not load the library.
"""
from .config import Config, CONFIGS, get_config  # noqa: F401
