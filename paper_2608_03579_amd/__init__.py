"""MI355X-native centroid + residual LoRA apply (SALT serving hot path).

``salt``  -- ctypes binding of the ``libsalt`` C ABI (``include/salt.h``).
``synth`` -- seeded synthetic workloads (inputs only; no method arithmetic).
``build`` -- compiles ``libsalt.so`` for gfx950 in-tree.

Submodules are imported on demand so that importing the package never loads
the shared library.
"""
__all__ = ["salt", "synth", "build"]
