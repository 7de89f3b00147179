"""MI355X-native tree verification for OoO-Spec-style speculative decoding.

The native library (``libooo.so``, HIP kernels for gfx950 behind a C ABI) is
loaded lazily by :mod:`paper_2608_00814_amd.ooo`; importing this package does
not touch the GPU.
"""

__all__ = ["workload"]
