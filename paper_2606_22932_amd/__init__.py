"""MI355X (gfx950) fused weight-gradient + AdamW step (FORGE, arxiv 2606.22932).

``forge``  -- ctypes binding of the C ABI (include/forge.h); the HIP library is loaded on
              first use and calls fail loudly if it is not built.
``synth``  -- seeded synthetic inputs (no method arithmetic).
``build``  -- compiles ``libforge.so`` with hipcc for gfx950.
``accounting`` -- algorithmic bytes and flops of a step.
"""
from . import build, forge, synth  # noqa: F401
