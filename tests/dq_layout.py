"""CPU converters between the logical formats and the tiled device layouts of
include/dq.h (test infrastructure; written from the header's layout text).

NVFP4 ("32x64 tiles"): codes tile (tr, tc) at byte (tr*(C64/64)+tc)*1024, row r
at r*32, byte j = columns 2j (low nibble), 2j+1 (high nibble); scales tile at
(tr*(C64/64)+tc)*128, row r block b at r*4+b.

LUT ("16x128 tiles"): group g = q*16+i of tile (tr, c) at ((tr*C128/128+c)*64+g)*GB
holds columns 128c+32q+t; code t in dword/bit positions per dq.h.
"""
import numpy as np


def _ru(x, m):
    return (x + m - 1) // m * m


# ---------------------------------------------------------------- NVFP4
def nvfp4_unpack(codes: np.ndarray, scales: np.ndarray, rows: int, cols: int):
    R, C = _ru(rows, 32), _ru(cols, 64)
    tr, tc = R // 32, C // 64
    cb = np.asarray(codes, np.uint8)[: R * C // 2].reshape(tr, tc, 32, 32)
    q = np.empty((tr, tc, 32, 64), np.uint8)
    q[..., 0::2] = cb & 0xF
    q[..., 1::2] = cb >> 4
    q = q.transpose(0, 2, 1, 3).reshape(R, C)
    sb = np.asarray(scales, np.uint8)[: R * C // 16].reshape(tr, tc, 32, 4).transpose(0, 2, 1, 3).reshape(R, C // 16)
    return q[:rows, :cols], sb[:rows, : cols // 16], q, sb


def nvfp4_pack(codes: np.ndarray, scale_codes: np.ndarray):
    """Logical codes [rows, cols] (0..15) and scales [rows, cols/16] -> tiled buffers."""
    rows, cols = codes.shape
    R, C = _ru(rows, 32), _ru(cols, 64)
    q = np.zeros((R, C), np.uint8)
    q[:rows, :cols] = codes
    s = np.zeros((R, C // 16), np.uint8)
    s[:rows, : cols // 16] = scale_codes
    tr, tc = R // 32, C // 64
    qt = q.reshape(tr, 32, tc, 64).transpose(0, 2, 1, 3)
    cb = (qt[..., 0::2] | (qt[..., 1::2] << 4)).astype(np.uint8).reshape(-1)
    sb = s.reshape(tr, 32, tc, 4).transpose(0, 2, 1, 3).reshape(-1).astype(np.uint8)
    return cb, sb


# ---------------------------------------------------------------- MXFP4
def mxfp4_unpack(codes: np.ndarray, scales: np.ndarray, rows: int, cols: int):
    """Tiled MXFP4 buffers -> logical codes [rows, cols] and scale codes [rows, cols/32]
    (plus the padded arrays)."""
    R, C = _ru(rows, 32), _ru(cols, 64)
    tr, tc = R // 32, C // 64
    cb = np.asarray(codes, np.uint8)[: R * C // 2].reshape(tr, tc, 32, 32)
    q = np.empty((tr, tc, 32, 64), np.uint8)
    q[..., 0::2] = cb & 0xF
    q[..., 1::2] = cb >> 4
    q = q.transpose(0, 2, 1, 3).reshape(R, C)
    # 4-tile scale groups: byte 4*(r + 32h) + q of group (g, tc) = row 128g + 32q + r, block 2tc + h
    R4 = _ru(rows, 128)
    sb = (np.asarray(scales, np.uint8)[: R4 * C // 32].reshape(R4 // 128, tc, 2, 32, 4)
          .transpose(0, 4, 3, 1, 2).reshape(R4, C // 32))
    return q[:rows, :cols], sb[:rows, : cols // 32], q, sb


def mxfp4_pack(codes: np.ndarray, scale_codes: np.ndarray):
    """Logical codes [rows, cols] and scale codes [rows, cols/32] -> tiled buffers."""
    rows, cols = codes.shape
    R, C = _ru(rows, 32), _ru(cols, 64)
    q = np.zeros((R, C), np.uint8)
    q[:rows, :cols] = codes
    R4 = _ru(rows, 128)
    s = np.zeros((R4, C // 32), np.uint8)
    s[:rows, : cols // 32] = scale_codes
    tr, tc = R // 32, C // 64
    qt = q.reshape(tr, 32, tc, 64).transpose(0, 2, 1, 3)
    cb = (qt[..., 0::2] | (qt[..., 1::2] << 4)).astype(np.uint8).reshape(-1)
    # [g, q, r, tc, h] -> [g, tc, h, r, q]
    sb = s.reshape(R4 // 128, 4, 32, tc, 2).transpose(0, 3, 4, 2, 1).reshape(-1).astype(np.uint8)
    return cb, sb


# ---------------------------------------------------------------- LUT
def _code_positions(bits):
    """For t in 0..31: list of (dword, shift, width, value_shift) pieces."""
    out = []
    for t in range(32):
        s, b = t // 4, t % 4
        if bits == 3:
            if s < 6:
                out.append([(s // 2, 8 * b + 3 * (s % 2), 3, 0)])
            else:
                out.append([(s - 6, 8 * b + 6, 2, 0), (2, 8 * b + 6 + (s - 6), 1, 2)])
        else:
            out.append([(s // 4, 8 * b + 2 * (s % 4), 2, 0)])
    return out


def lut_codes_unpack(codes: np.ndarray, rows: int, cols: int, bits: int) -> np.ndarray:
    R, C = _ru(rows, 16), _ru(cols, 128)
    tr, tcn = R // 16, C // 128
    nd = 3 if bits == 3 else 2
    w = np.asarray(codes, np.uint8)[: tr * tcn * 64 * nd * 4].view(np.uint32).reshape(tr, tcn, 4, 16, nd)
    out = np.zeros((tr, tcn, 4, 16, 32), np.uint8)
    for t, pieces in enumerate(_code_positions(bits)):
        v = np.zeros(w.shape[:-1], np.uint32)
        for d, sh, wd, vs in pieces:
            v |= ((w[..., d] >> np.uint32(sh)) & np.uint32((1 << wd) - 1)) << np.uint32(vs)
        out[..., t] = v
    # [tr, c, q, i, t] -> rows tr*16+i, cols c*128 + q*32 + t
    full = out.transpose(0, 3, 1, 2, 4).reshape(R, C)
    return full[:rows, :cols]


def lut_scales_unpack(scales: np.ndarray, rows: int, cols: int) -> np.ndarray:
    R, C = _ru(rows, 16), _ru(cols, 128)
    tr, tcn = R // 16, C // 128
    s = np.asarray(scales, np.uint8)[: tr * tcn * 128].reshape(tr, tcn, 4, 16, 2)
    full = s.transpose(0, 3, 1, 2, 4).reshape(R, C // 16)
    return full[:rows, : cols // 16]


def lut_codes_pack(codes: np.ndarray, bits: int) -> np.ndarray:
    rows, cols = codes.shape
    R, C = _ru(rows, 16), _ru(cols, 128)
    full = np.zeros((R, C), np.uint32)
    full[:rows, :cols] = codes
    tr, tcn = R // 16, C // 128
    g = full.reshape(tr, 16, tcn, 4, 32).transpose(0, 2, 3, 1, 4)     # [tr, c, q, i, t]
    nd = 3 if bits == 3 else 2
    w = np.zeros(g.shape[:-1] + (nd,), np.uint32)
    for t, pieces in enumerate(_code_positions(bits)):
        for d, sh, wd, vs in pieces:
            w[..., d] |= ((g[..., t] >> np.uint32(vs)) & np.uint32((1 << wd) - 1)) << np.uint32(sh)
    return w.reshape(-1).view(np.uint8)
