"""MI355X-native ES parameter path: seeded perturb / restore / fused update /
reward z-score over lists of bf16 tensors (arXiv 2608.17310, Section 3).

The compute runs in the HIP library ``libesopt.so`` (csrc/); ``esopt`` is its
thin ctypes binding.  Importing this package does not load the library; the
first call into ``esopt`` does, and fails loudly if it has not been built.
"""

__all__ = ["esopt", "workloads"]
