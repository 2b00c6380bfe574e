"""NVFP4 W4A4 MoE expert layer with Residual Activation Compensation on MI355X.

QUADS (arXiv 2607.15810), rollout side: NVFP4 activation quantisation,
online top-K_s residual channel selection, grouped W4A4 expert GEMMs with a
fused residual term, SwiGLU and the weighted combine, as hand-written HIP
kernels for gfx950 behind a C ABI (``libquads.so``, declared in
``include/quads.h``).

Submodules:
  ``quads``  ctypes binding of the C ABI (loads the library on first use and
             raises if it is missing).
  ``ops``    the same calls on torch tensors (device memory, streams).
  ``synth``  seeded synthetic workloads.
"""

__all__ = ["quads", "ops", "synth"]
