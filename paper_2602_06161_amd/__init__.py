"""COVER on MI355X (gfx950): cache-override attention with the diagonal correction and
stability-aware seed selection, as hand-written HIP kernels behind a C ABI
(``include/cover.h``).

Submodules:
  cover   ctypes binding of the C ABI (device memory and streams from torch)
  synth   seeded synthetic inputs shared by the tests and the benchmark
  build   hipcc build of the shared library

Importing the package loads nothing; ``cover`` loads the library on first use and
raises if it has not been built.
"""
__all__ = ["cover", "synth", "build"]
