"""Binarized CNN inference on MI355X (gfx950): bit-packed +-1 conv and FC
layers computed with XOR + popcount, behind the C ABI declared in
``include/bnn.h`` (library ``libbnn.so``).

Submodules:
  ``bnn``   -- ctypes binding of the C ABI (loads libbnn.so; fails loudly if
               it is missing)
  ``synth`` -- seeded synthetic inputs and workload shapes (host numpy)
  ``build`` -- compiles libbnn.so with hipcc for gfx950
"""
