"""MI355X-native asynchronous stochastic coordinate descent/ascent for generalized linear
models (arXiv 1702.07005): HIP kernels for gfx950 behind the C ABI declared in
``include/scd.h``; ``paper_1702_07005_amd.scd`` is the thin Python binding.

Importing the package loads nothing; the HIP library is loaded on first use of
``paper_1702_07005_amd.scd``.
"""
__all__ = ["scd", "synth"]
