"""MI355X-native batched VLA rollout inference (VLA-RL, arXiv 2505.18719).

Submodules:
  * ``inputs`` -- seeded synthetic workloads (no decoder arithmetic);
  * ``vla``    -- ctypes binding of the HIP library ``libvla.so``;
  * ``build``  -- compiles the HIP library for gfx950.

Nothing is imported eagerly so that ``inputs`` can be used without the
compiled library.
"""
