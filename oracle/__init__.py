"""Plain CPU oracle for the EchoCache cached DiT block step.

TEST INFRASTRUCTURE ONLY.  This package is the slow, obviously correct
definition that the HIP path is checked against.  It shares no code with the
HIP path and never imports it; only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it.  The product path must never route
through it.

Modules follow the paper's method in order:
  energy  audio STFT energy per latent frame   (Sec. 3.3, saliency anchors)
  select  per-token saliency and top-K         (Sec. 3.1 Eq. 1; Sec. 3.3)
  block   DiT block on the selected tokens     (Sec. 3.3, latent-level caching)
  cache   int8 residual cache and reuse        (Sec. 3.3 fusion; Sec. 3.4)
  step    the composed cached step

Floating point is fp64 except where an integer is decided (ranking keys are
fp32 saliencies; int8 codes are decided in fp32, the precision of the kernel).
"""
from . import energy, select, block, cache, step  # noqa: F401
