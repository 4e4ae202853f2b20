"""MI355X (gfx950) implementation of the fused low-bit linear of a
world-action DiT (SteerQuant / Rudder, arXiv 2609.39056).

- ``binding``: ctypes binding of the C ABI in include/sq.h (libsq.so).
- ``synth``:   seeded synthetic layer inputs.
- ``_build``:  compiles the HIP sources in csrc/ for gfx950.
"""
__all__ = ["binding", "synth"]
