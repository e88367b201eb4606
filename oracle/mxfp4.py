"""MXFP4 quantization (oracle; test infrastructure).

The paper runs MXFP4 instead of NVFP4 for a model that is released natively
in that format (Sec. 3.2, the accuracy table's footnote, and the description of
the evaluation arms) and does not restate the format.  This follows the OCP
Microscaling Formats (MX) specification v1.0:

* blocks of 32 consecutive elements along the contraction dimension (the
  last axis here);
* one E8M0 scale per block: the power of two ``2**(code - 127)``, code
  0..254 (0xFF is NaN and is never produced);
* E2M1 elements ``sign << 3 | index``, index into {0, 0.5, 1, 1.5, 2, 3, 4, 6};
* no tensor-level scale.

Conversion (the specification's reference algorithm, which the paper does
not override):

1. ``a = max|x_i|`` over the block (fp32 values).
2. ``e = floor(log2(a)) - 2`` (2 is the exponent of E2M1's largest power of
   two: 6 = 1.5 * 2**2), clamped to [-127, 127]; an all-zero block takes
   ``e = -127``.  The scale code is ``e + 127``.
3. ``y_i = x_i * 2**-e``, exact, and ``q_i = sign(y_i) << 3 | E2M1(|y_i|)``
   (nearest, ties to even, saturating at 6: the block maximum, which lies in
   [4, 8) after scaling, saturates when it is 7 or more); a zero magnitude
   always carries sign 0.
4. dequantization: ``e2m1(q) * 2**(code - 127)``, exact in fp64.

Pins (tests/test_oracle_mxfp4.py): the E8M0 decode of all codes against
torch's float8_e8m0fnu, a hand-worked block per scale branch, exact
power-of-two invariance, a pure-Python brute-force quantizer on tiny tensors,
zero blocks, and the element error bound.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from . import formats

BLOCK = 32
E2M1_EMAX = 2          # 6 = 1.5 * 2**2
E8M0_BIAS = 127


def e8m0_decode(code) -> np.ndarray:
    """Value of E8M0 bytes as float64: 2**(code - 127); NaN for 0xFF."""
    c = np.asarray(code, dtype=np.uint8).astype(np.int64)
    return np.where(c == 0xFF, np.nan, np.exp2((c - E8M0_BIAS).astype(np.float64)))


def block_exponent(a) -> np.ndarray:
    """Shared exponent of blocks with maximum magnitude ``a`` (fp32, >= 0)."""
    a = np.asarray(a, dtype=np.float32).astype(np.float64)
    m, e = np.frexp(a)                       # a = m * 2**e with 0.5 <= m < 1: floor(log2 a) = e - 1
    x = (e - 1) - E2M1_EMAX
    x = np.where(a == 0, -E8M0_BIAS, x)
    return np.clip(x, -E8M0_BIAS, E8M0_BIAS).astype(np.int64)


def quantize(x) -> Tuple[np.ndarray, np.ndarray]:
    """MXFP4-quantize ``x[rows, cols]`` (fp32 values).

    Returns ``(codes[rows, cols] uint8 in 0..15, scale_codes[rows, cols/32] uint8)``.
    """
    x = np.asarray(x, dtype=np.float32)
    rows, cols = x.shape
    if cols % BLOCK:
        raise ValueError("cols must be a multiple of 32")
    blk = x.reshape(rows, cols // BLOCK, BLOCK).astype(np.float64)
    e = block_exponent(np.max(np.abs(blk), axis=-1))
    y = blk * np.exp2(-e.astype(np.float64))[..., None]     # exact: fp32 values times a power of two
    mag = formats.e2m1_rne_sat(y)
    neg = (y < 0) & (mag > 0)
    q = (neg.astype(np.uint8) << np.uint8(3)) | mag
    return q.reshape(rows, cols).astype(np.uint8), (e + E8M0_BIAS).astype(np.uint8)


def dequantize(codes, scale_codes) -> np.ndarray:
    """Exact fp64 value of an MXFP4 tensor."""
    q = np.asarray(codes, dtype=np.uint8)
    rows, cols = q.shape
    v = formats.e2m1_decode(q).reshape(rows, cols // BLOCK, BLOCK)
    return (v * e8m0_decode(scale_codes)[..., None]).reshape(rows, cols)


def quantize_bf16_activations(x_bits) -> Tuple[np.ndarray, np.ndarray]:
    """Quantize bf16 activations given as bit patterns."""
    return quantize(formats.f32_from_bf16_bits(x_bits))
