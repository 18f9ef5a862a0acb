"""MI355X-native seeded perturbation engine for shared-randomness SPSA
("Just One Byte (per gradient)", arXiv 2306.10015).

Submodules:
  mezo  — Python binding of the C-ABI library libmezo.so (HIP kernels, gfx950)
  synth — seeded synthetic parameter sets, seeds and one-byte gradients
  build — compiles libmezo.so with hipcc

Importing the package loads nothing; ``paper_2306_10015_amd.mezo`` loads the
library and raises if it is not built.
"""
__all__ = ["mezo", "synth", "build"]
