"""MI355X-native batched forecast scoring (prefill-only LLM surrogate) for gfx950.

The compute lives in libsurrogate.so (hand-written HIP kernels behind the C ABI of
include/surrogate.h); ``binding`` is its ctypes binding and ``synth`` draws the seeded
synthetic inputs.
"""
from . import synth  # noqa: F401
