"""CPU oracle for the phase-specific quantized linear layer.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow reference that
the HIP path is checked against.  Only the tests, the smoke entry point and
the benchmark's CPU-baseline leg may import it; the product library never
does, and the two share no code (the seeded input generators in ``synth``
are the only common module, and they hold none of the method's arithmetic).

What it computes (paper, App. A "Quantization formats"):

* ``formats``  - the E2M1 element grid and the FP8-E4M3 scale format, with
  round-to-nearest-even and saturation; fp64 -> fp16 rounding.
* ``nvfp4``    - NVFP4 two-level scaling: an fp32 tensor scale
  ``max|W| / (6 * 448)``, one E4M3 scale per 16 elements along the
  contraction dimension, E2M1 codes (weights, activations, and the
  requantization of a GEMM output).
* ``mxfp4``    - MXFP4 (OCP MX: E8M0 power-of-two scale per 32 elements,
  E2M1 codes), the format of the paper's MXFP4 arms.
* ``lut``      - LUT weight-only formats: the per-row equal-count LUT fit
  (the benchmark's decode format) and the paper's fixed LUT3A16/LUT2A16
  grids with a signed E4M3 block scale.
* ``linalg``   - fp64 GEMM / GEMV over dequantized operands, SwiGLU.

Parity status per function is listed in each module header.  Every
floating-point step uses IEEE fp32 (NumPy float32, correctly rounded) or
exact fp64, in the order documented per function.
"""
from . import formats, nvfp4, mxfp4, lut, linalg  # noqa: F401
