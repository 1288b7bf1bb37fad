"""MI355X-native physics-informed GAN training step (arXiv 1910.13444).

The package holds the hot path of the method: a C-ABI library (``libpigan.so``,
built from the HIP sources under ``csrc/``) and a thin ctypes binding
(:mod:`paper_1910_13444_amd.pigan`).  Importing the package loads nothing; the
library is opened on first use by :func:`paper_1910_13444_amd.pigan.lib`.
"""

__all__ = ["configs", "inputs", "flops", "pigan"]
