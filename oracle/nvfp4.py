"""NVFP4 quantization (oracle; test infrastructure).

Follows the paper's App. A, "NVFP4-esque two-level scaling" and "NVFP4":

* the tensor carries one fp32 global scale ``G = max|W| / (6 * 448)``;
* elements are grouped in blocks of 16 along the contraction dimension
  (the last axis here: rows are output features or tokens, columns are K);
* each block carries an E4M3 scale chosen so that the block's largest
  magnitude maps to about 6 on the E2M1 grid;
* elements are E2M1 codes ``sign << 3 | index`` with index into
  {0, 0.5, 1, 1.5, 2, 3, 4, 6}.

Activations use a static per-tensor scale from a running-maximum observer
(same section); the dynamic variant takes ``G`` from the tensor itself.

The fp32 operation order (the paper is silent on it) is:

1. ``amax = max|x|`` over the tensor; ``G = fp32(amax / 2688)``; ``G = 1`` if ``amax == 0``.
2. per block: ``a = max|x_i|``; ``den = fp32(6 * G)``; ``t = fp32(a / den)``.
3. ``c = E4M3(t)`` (nearest, ties to even, saturating at 448).
4. ``S = fp32(e4m3(c) * G)``.
5. ``S == 0``: all codes 0.  Else ``y_i = fp32(x_i / S)``,
   ``q_i = sign(y_i) << 3 | E2M1(|y_i|)``; a zero magnitude always carries sign 0.
6. dequantization: ``e2m1(q) * e4m3(c) * G``, exact in fp64.

Pins (tests/test_oracle_nvfp4.py): hand-worked tie block, the closed form
``G = 2**-k, a = 6 v G -> c = v``, a pure-Python brute-force quantizer on
tiny tensors, idempotence, sign symmetry, zero blocks, error bound.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from . import formats

BLOCK = 16
GLOBAL_DIVISOR = np.float32(6.0 * 448.0)   # 2688


def global_scale(amax) -> np.float32:
    """``G = fp32(amax / 2688)``, or 1 for an all-zero tensor."""
    a = np.float32(amax)
    if a == 0:
        return np.float32(1.0)
    return np.float32(a / GLOBAL_DIVISOR)


def amax(x) -> np.float32:
    return np.float32(np.max(np.abs(np.asarray(x, dtype=np.float32)))) if np.size(x) else np.float32(0)


def quantize(x, G) -> Tuple[np.ndarray, np.ndarray]:
    """NVFP4-quantize ``x[rows, cols]`` (fp32 values) under global scale ``G``.

    Returns ``(codes[rows, cols] uint8 in 0..15, scale_codes[rows, cols/16] uint8)``.
    """
    x = np.asarray(x, dtype=np.float32)
    rows, cols = x.shape
    if cols % BLOCK:
        raise ValueError("cols must be a multiple of 16")
    G = np.float32(G)
    blk = x.reshape(rows, cols // BLOCK, BLOCK)
    a = np.max(np.abs(blk), axis=-1)                            # fp32
    den = np.float32(np.float32(6.0) * G)
    t = (a / den).astype(np.float32)
    c = formats.e4m3_rne_satfinite(t)
    S = (formats.e4m3_decode(c).astype(np.float32) * G).astype(np.float32)
    safe = np.where(S == 0, np.float32(1.0), S)
    y = (blk / safe[..., None]).astype(np.float32)
    mag = formats.e2m1_rne_sat(y)
    neg = (y < 0) & (mag > 0)
    q = (neg.astype(np.uint8) << np.uint8(3)) | mag
    q = np.where((S == 0)[..., None], np.uint8(0), q).astype(np.uint8)
    return q.reshape(rows, cols), c


def quantize_dynamic(x) -> Tuple[np.ndarray, np.ndarray, np.float32]:
    G = global_scale(amax(x))
    q, c = quantize(x, G)
    return q, c, G


def dequantize(codes, scale_codes, G) -> np.ndarray:
    """Exact fp64 value of an NVFP4 tensor."""
    q = np.asarray(codes, dtype=np.uint8)
    rows, cols = q.shape
    e = formats.e2m1_decode(q).reshape(rows, cols // BLOCK, BLOCK)
    s = formats.e4m3_decode(scale_codes)[..., None]
    return (e * s * np.float64(np.float32(G))).reshape(rows, cols)


def pack_nibbles(codes) -> np.ndarray:
    """Two 4-bit codes per byte: element ``2j`` in the low nibble of byte ``j``."""
    q = np.asarray(codes, dtype=np.uint8)
    return (q[..., 0::2] | (q[..., 1::2] << np.uint8(4))).astype(np.uint8)


def unpack_nibbles(packed) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = p & np.uint8(0xF)
    out[..., 1::2] = p >> np.uint8(4)
    return out


def quantize_bf16_activations(x_bits, G_static=None):
    """Quantize bf16 activations (given as bit patterns); dynamic ``G`` when ``G_static`` is None."""
    x = formats.f32_from_bf16_bits(x_bits)
    if G_static is None:
        return quantize_dynamic(x)
    q, c = quantize(x, np.float32(G_static))
    return q, c, np.float32(G_static)
