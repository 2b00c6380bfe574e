"""CPU oracle for the NVFP4 W4A4 MoE expert layer with Residual Activation
Compensation (QUADS, arXiv 2607.15810).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, deliberately
unoptimised statement of what the GPU path computes.  Only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it; the GPU
library never calls into it and it shares no code with the GPU library.

Precision: element-wise steps are IEEE float32 (one rounding per operation,
round-to-nearest-even); contractions are float64 on exactly dequantised
values.  Every function cites the passage of the paper it follows.

Functions whose result the paper does not fix (and which no closed form or
library routine pins) say "parity unpinned" in their docstring.
"""

from . import formats, quant, route, rac, layer, fp8  # noqa: F401
