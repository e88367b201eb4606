"""RMSNorm fused with the NVFP4 activation quantizer (oracle; test
infrastructure).

The paper quantizes activations inside the normalization kernels that feed
the quantized projections (App. C, "Prefill measurements": activation
processing is grouped with the norms).  It does not restate RMSNorm; the
reading taken here, in fp32 with this operation order:

* ``ss = sum_k x_k^2``, exactly (every square of a bf16 value is exact in
  fp64; the sum is the exactly rounded ``math.fsum``);
* ``ms = fp32(ss / K)`` (the fp64 quotient, then fp32), ``r = fp32(ms + eps)``;
* ``inv = fp32(1 / fp32(sqrt(r)))`` (correctly rounded square root and
  division);
* ``y_k = fp32(fp32(x_k * inv) * gamma_k)``;
* the NVFP4 activation rule of App. A on ``y`` (static global scale, or
  ``G = amax(y) / 2688``).

Pins (tests/test_oracle_norm.py): constant rows and power-of-two scalings
(exact closed forms), and agreement with the fp64 formula within the fp32
rounding of the steps.
"""
from __future__ import annotations

import math

import numpy as np

from . import formats, nvfp4


def rmsnorm_bf16(x_bits, gamma_bits, eps) -> np.ndarray:
    """fp32 RMSNorm of bf16 rows ``x[M, K]`` with bf16 weights ``gamma[K]``."""
    x = formats.f32_from_bf16_bits(x_bits)
    g = formats.f32_from_bf16_bits(np.asarray(gamma_bits).reshape(1, -1))[0]
    M, K = x.shape
    eps = np.float32(eps)
    out = np.empty((M, K), np.float32)
    for m in range(M):
        ss = math.fsum(float(v) * float(v) for v in x[m])
        ms = np.float32(ss / K)
        r = np.float32(ms + eps)
        inv = np.float32(np.float32(1.0) / np.sqrt(r, dtype=np.float32))
        out[m] = ((x[m] * inv).astype(np.float32) * g).astype(np.float32)
    return out


def quantize_rmsnorm_bf16(x_bits, gamma_bits, eps, G_static=None):
    """RMSNorm then NVFP4 activation quantization.  Returns ``(codes,
    scale_codes, G, y)`` with ``y`` the fp32 normalized activations."""
    y = rmsnorm_bf16(x_bits, gamma_bits, eps)
    G = nvfp4.global_scale(nvfp4.amax(y)) if G_static is None else np.float32(G_static)
    q, c = nvfp4.quantize(y, G)
    return q, c, G, y
