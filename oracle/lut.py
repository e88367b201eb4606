"""LUT weight-only formats (oracle; test infrastructure).

Two ways to build a b-bit LUT weight (b = 3: LUT3, b = 2: LUT2):

``PER_ROW`` - one 2**b-entry fp16 table per output row.  The row is sorted
ascending and cut into 2**b bins of K / 2**b consecutive elements; each entry
is the mean of its bin; each weight gets the code of the nearest entry.  This
is the decode format of every benchmark workload here.  The paper itself does
not define it; the readings taken are:

* bin mean = exactly rounded sum (``math.fsum``) / count in fp64, then fp16
  round-to-nearest-even;
* code = ``#{j : w > m_j}`` with the exact fp64 midpoints
  ``m_j = (L_j + L_{j+1}) / 2``, i.e. the nearest entry with ties going to
  the lower index (not the bin rank).

``PAPER_GRID`` - the paper's LUT3A16 / LUT2A16 formats (App. A, "LUT
formats" and "Storage cost"): a fixed grid that contains 0 and +6, the same
two-level scaling as NVFP4 (fp32 global scale ``max|W| / 2688``, one E4M3
scale per 16 elements along K), except that the block scale is *signed*: it
takes the sign of the block's largest-magnitude element so that this element
normalizes to +6.  Readings:

* the largest-magnitude element is the first one (lowest k) on ties;
* the block scale magnitude is ``E4M3(fp32(|w*| / fp32(6 G)))`` (nearest,
  ties to even, saturating), ``S = fp32(d * G)`` with the sign applied;
* code = nearest grid level of ``fp32(w / S)`` (exact fp64 midpoints, ties to
  the lower index, clamped at the ends);
* a block whose scale is zero gets scale byte 0x00 and the code of level 0;
* the grid is data: an fp16 table passed to both sides; the default is the
  paper's printed grid rounded to fp16.

Pins (tests/test_oracle_lut.py): rows with at most 2**b distinct values are
reproduced exactly, entries are non-decreasing, brute-force nearest search,
sign absorption (the block maximum always codes to +6), zero blocks, and the
printed grid's own optimality claim for LUT3 (a constrained Lloyd-Max fit
under N(0,1) with two-level scaling lands on it).
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np

from . import formats, nvfp4

PER_ROW = 0
PAPER_GRID = 1

# Paper, App. A "LUT formats": printed to four decimals.
PAPER_GRID_LUT3 = (-4.7038, -2.8698, -1.3696, 0.0, 1.2204, 2.5285, 4.0473, 6.0)
PAPER_GRID_LUT2 = (-3.6517, 0.0, 2.5227, 6.0)


def default_grid(bits: int) -> np.ndarray:
    """The paper's grid for ``bits`` rounded to fp16 (returned as float16)."""
    g = PAPER_GRID_LUT3 if bits == 3 else PAPER_GRID_LUT2 if bits == 2 else None
    if g is None:
        raise ValueError("bits must be 2 or 3")
    return formats.fp16_from_f64(np.array(g, dtype=np.float64))


def nearest_code(values, table) -> np.ndarray:
    """``#{j : v > m_j}`` with exact fp64 midpoints of the ascending ``table``."""
    t = np.asarray(table, dtype=np.float64)
    mids = (t[:-1] + t[1:]) / 2.0           # exact: fp16/fp32 entries
    v = np.asarray(values, dtype=np.float64)
    return np.sum(v[..., None] > mids, axis=-1).astype(np.uint8)


# ---------------------------------------------------------------- PER_ROW
def fit_row(row, bits: int) -> np.ndarray:
    """Equal-count bin means of one row, rounded to fp16 (float16 array)."""
    w = np.sort(np.asarray(row, dtype=np.float32).astype(np.float64))
    nb = 1 << bits
    if len(w) % nb:
        raise ValueError("row length must be a multiple of 2**bits")
    cnt = len(w) // nb
    means = [math.fsum(w[j * cnt:(j + 1) * cnt]) / cnt for j in range(nb)]
    return formats.fp16_from_f64(np.array(means, dtype=np.float64))


def quantize_per_row(W, bits: int) -> Tuple[np.ndarray, np.ndarray]:
    """Returns ``(codes[N, K] uint8, lut[N, 2**bits] float16)``."""
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    lut = np.empty((N, 1 << bits), dtype=np.float16)
    codes = np.empty((N, K), dtype=np.uint8)
    for n in range(N):
        lut[n] = fit_row(W[n], bits)
        codes[n] = nearest_code(W[n], lut[n])
    return codes, lut


def dequantize_per_row(codes, lut) -> np.ndarray:
    lut = np.asarray(lut, dtype=np.float16).astype(np.float64)
    c = np.asarray(codes, dtype=np.int64)
    return np.take_along_axis(lut, c, axis=1)


# ---------------------------------------------------------------- PAPER_GRID
def zero_level(grid) -> int:
    g = np.asarray(grid, dtype=np.float64)
    idx = np.nonzero(g == 0.0)[0]
    if len(idx) != 1:
        raise ValueError("grid must contain exactly one zero level")
    return int(idx[0])


def quantize_paper_grid(W, grid, G=None):
    """Returns ``(codes[N, K], scale_bytes[N, K/16] signed E4M3, G)``."""
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    if K % 16:
        raise ValueError("K must be a multiple of 16")
    grid = np.asarray(grid, dtype=np.float16)
    if G is None:
        a = np.float32(np.max(np.abs(W))) if W.size else np.float32(0)
        G = np.float32(1.0) if a == 0 else np.float32(a / np.float32(2688.0))
    G = np.float32(G)
    blk = W.reshape(N, K // 16, 16)
    i_star = np.argmax(np.abs(blk), axis=-1)                     # first max on ties
    w_star = np.take_along_axis(blk, i_star[..., None], axis=-1)[..., 0]
    den = np.float32(np.float32(6.0) * G)
    t = (np.abs(w_star) / den).astype(np.float32)
    mag = formats.e4m3_rne_satfinite(t)
    neg = (w_star < 0) & (mag != 0)
    sbyte = (mag | (neg.astype(np.uint8) << np.uint8(7))).astype(np.uint8)
    S = (formats.e4m3_decode(sbyte).astype(np.float32) * G).astype(np.float32)
    safe = np.where(S == 0, np.float32(1.0), S)
    y = (blk / safe[..., None]).astype(np.float32)
    codes = nearest_code(y, grid.astype(np.float64))
    codes = np.where((S == 0)[..., None], np.uint8(zero_level(grid)), codes)
    return codes.reshape(N, K).astype(np.uint8), sbyte, G


def dequantize_paper_grid(codes, scale_bytes, G, grid) -> np.ndarray:
    c = np.asarray(codes, dtype=np.int64)
    N, K = c.shape
    g = np.asarray(grid, dtype=np.float16).astype(np.float64)
    v = g[c].reshape(N, K // 16, 16)
    d = formats.e4m3_decode(scale_bytes)[..., None]
    return (v * d * np.float64(np.float32(G))).reshape(N, K)


# ---------------------------------------------------------------- autocast
def autocast_to_nvfp4(w_hat, G=None):
    """LUT -> NVFP4 autocast (Sec. 2.3: the LUT weights are re-quantized to
    NVFP4 for native low-precision prefill).  ``w_hat`` is the dequantized LUT
    weight (fp64, exact); it is rounded once to fp32 (exact for PER_ROW
    tables, one rounding of an exact product for PAPER_GRID) and quantized by
    the NVFP4 weight rule of App. A: ``G = amax / 2688`` unless given.

    Returns ``(codes, scale_codes, G)``."""
    w32 = np.asarray(w_hat, dtype=np.float64).astype(np.float32)
    if G is None:
        return nvfp4.quantize_dynamic(w32)
    q, c = nvfp4.quantize(w32, np.float32(G))
    return q, c, np.float32(G)
