"""MI355X (gfx950) reverse-step library for discrete-diffusion language models.

The compute lives in libdd.so (HIP kernels behind the C ABI of include/dd.h);
this package holds the build script and a thin ctypes binding (`_lib`).
"""
from . import _lib as dd  # noqa: F401
