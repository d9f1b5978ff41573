"""MI355X-native (gfx950 HIP) hot path of Archer cached-prompt diffusion-LM decoding.

* ``paper_2608_08086_amd.build``  -- compiles ``csrc/*.hip`` into ``_lib/libarcher.so``.
* ``paper_2608_08086_amd.archer`` -- ctypes binding of the C ABI (``include/archer.h``,
  ``include/archer_ops.h``); importing it requires the built library.
"""
