"""Number formats used by NVFP4 and the LUT formats (oracle; test infrastructure).

The paper fixes the element grid of NVFP4 (E2M1 magnitudes
{0, 0.5, 1, 1.5, 2, 3, 4, 6} with a sign) and names FP8-E4M3 as the block
scale format (App. A, "NVFP4-esque two-level scaling" and "NVFP4").  It does
not spell out the encodings; these follow the OCP 8-bit floating point
specification (E4M3 "FN" variant: bias 7, no infinities, NaN = S.1111.111,
largest finite 448) and the OCP MX specification's E2M1 element.

Rounding reading (the paper says only that a block's extreme element maps to
"approximately" +-6): every rounding here is round-to-nearest, ties to the
even code, with saturation to the largest finite value.  Both grids are
monotone in the code for non-negative values, so "ties to even" is decided by
the code's parity.

Pins: hand-worked values, all 256 E4M3 codes, brute force against exact
rational arithmetic, and torch's float8_e4m3fn cast for in-range values
(tests/test_oracle_formats.py).
"""
from __future__ import annotations

import numpy as np

E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
E2M1_MAX = 6.0
E4M3_MAX = 448.0
E4M3_MAX_CODE = 0x7E


def e4m3_decode(code) -> np.ndarray:
    """Value of E4M3 bytes as float64 (sign in bit 7; NaN for S.1111.111)."""
    c = np.asarray(code, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 0xF) & (m == 0x7), np.nan, mag)
    return sign * mag


# Non-negative finite E4M3 values, indexed by code 0x00..0x7E (ascending).
E4M3_VALUES = e4m3_decode(np.arange(0, E4M3_MAX_CODE + 1, dtype=np.uint8))


def _nearest_even_code(t: np.ndarray, values: np.ndarray) -> np.ndarray:
    """Index of the nearest entry of ascending ``values`` (ties to even index).

    ``t`` must be non-negative and not above ``values[-1]`` (callers clamp).
    Distances are formed in float64, where they are exact: ``t`` is fp32 and
    the two candidates lie within a factor of two of it.
    """
    t = np.asarray(t, dtype=np.float64)
    lo = np.searchsorted(values, t, side="right") - 1
    lo = np.clip(lo, 0, len(values) - 1)
    hi = np.minimum(lo + 1, len(values) - 1)
    d_lo = t - values[lo]
    d_hi = values[hi] - t
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0) & (hi != lo))
    return np.where(take_hi, hi, lo).astype(np.int64)


def e4m3_rne_satfinite(t) -> np.ndarray:
    """Encode non-negative values as E4M3 codes: nearest, ties to even, saturating.

    Values at or above 448 give 0x7E; values at or below 2**-10 (half the
    smallest subnormal) give 0x00.
    """
    t = np.asarray(t, dtype=np.float64)
    if np.any(t < 0) or np.any(np.isnan(t)):
        raise ValueError("e4m3_rne_satfinite expects non-negative finite input")
    return _nearest_even_code(np.minimum(t, E4M3_MAX), E4M3_VALUES).astype(np.uint8)


def e2m1_rne_sat(y) -> np.ndarray:
    """Magnitude index (0..7) of the E2M1 value nearest to ``|y|``; ties to even; >= 6 -> 7."""
    a = np.abs(np.asarray(y, dtype=np.float64))
    return _nearest_even_code(np.minimum(a, E2M1_MAX), E2M1_MAGNITUDES).astype(np.uint8)


def e2m1_decode(code) -> np.ndarray:
    """Value of 4-bit E2M1 codes ``sign << 3 | magnitude index`` as float64."""
    c = np.asarray(code, dtype=np.uint8).astype(np.int64)
    return np.where(c & 8, -1.0, 1.0) * E2M1_MAGNITUDES[c & 7]


def fp16_from_f64(x) -> np.ndarray:
    """Round float64 values to fp16 (nearest, ties to even), in one rounding.

    NumPy converts float64 to float16 directly from the double's bits (not
    through float32); the tests pin this against exact rational rounding.
    """
    return np.asarray(x, dtype=np.float64).astype(np.float16)


def f64_from_bf16_bits(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f32_from_bf16_bits(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def bf16_rne_from_f64(x) -> np.ndarray:
    """Round float64 values to bf16, nearest-even, in one rounding (returns float64 values).

    Used to form the rounded reference for bf16 GEMM / GEMV outputs.  Works on
    exact rationals through the fp64 significand: bf16 keeps 8 significant bits.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                  # x = m * 2**e, 0.5 <= |m| < 1
    scaled = m * 256.0                  # 8 significant bits -> integer part
    r = np.round(scaled)                # numpy rounds half to even
    out = np.ldexp(r / 256.0, e)
    return np.where(x == 0, x, out)
