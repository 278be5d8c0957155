"""MI355X-native hot path of adaptive expert prefetching for MoE decode.

The package holds the HIP kernels and the C-ABI library (``csrc/``), a thin ctypes
binding with the library's entry-point names (``native``), the decode runner that
strings the entry points together per layer (``runtime``), workload shapes
(``configs``) and the seeded input generators (``inputs``).

Importing the package loads nothing native; the library is loaded on first use of
``native`` and raises if it has not been built.
"""
__all__ = ["configs", "inputs"]
