"""MI355X (gfx950) library for decode attention over per-layer compressed KV caches.

The compute lives in libkvk.so (HIP kernels behind the C ABI of include/kvk.h);
`kvk` is its Python binding and `synth` the seeded synthetic-input generators.
"""
from . import kvk  # noqa: F401
