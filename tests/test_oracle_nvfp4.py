"""Pins for the oracle's NVFP4 quantizer (CPU only).

Checks: a hand-worked tie block (tests/golden/e2m1_tie_block.txt), the
closed-form scale rule (block amax / 6 rounded to E4M3), a scalar
brute-force quantizer written with exact rationals, and invariants:
idempotent requantization, codes in range, zero blocks, sign symmetry,
the per-element error bound.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import formats, nvfp4

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load_tie_block():
    d = {}
    for line in open(os.path.join(GOLDEN, "e2m1_tie_block.txt")):
        if line.strip() and not line.startswith("#"):
            k, *v = line.split()
            d[k] = v
    return d


def test_hand_worked_tie_block():
    d = _load_tie_block()
    x = np.array([float(v) for v in d["x"]], dtype=np.float32)[None, :]
    q, c = nvfp4.quantize(x, np.float32(float(d["G"][0])))
    assert c[0, 0] == int(d["scale_code"][0], 16)
    assert list(q[0]) == [int(v) for v in d["codes"]]


def test_closed_form_scale_rule():
    """G = 2**-k and a block max of 6 v G (v an E4M3 value) give scale code v and max code 6."""
    rng = np.random.default_rng(10)
    codes_v = rng.integers(0x08, 0x7E, 256).astype(np.uint8)      # normal range
    v = formats.e4m3_decode(codes_v)
    for k in (0, 3, 7):
        G = np.float32(2.0 ** -k)
        x = rng.uniform(-1, 1, (256, 16)) * (6 * v * float(G))[:, None]
        j = rng.integers(0, 16, 256)
        sign = np.where(rng.random(256) < 0.5, -1.0, 1.0)
        x[np.arange(256), j] = sign * 6 * v * float(G)
        x = x.astype(np.float32)
        assert np.array_equal(x[np.arange(256), j].astype(np.float64), sign * 6 * v * float(G))
        q, c = nvfp4.quantize(x, G)
        assert np.array_equal(c[:, 0], codes_v)
        want = np.where(sign < 0, 15, 7)
        assert np.array_equal(q[np.arange(256), j], want)


def _brute_block(xs, G):
    """Scalar NVFP4 for one 16-block with exact rational nearest searches."""
    G = np.float32(G)
    a = max(abs(np.float32(v)) for v in xs)
    den = np.float32(np.float32(6.0) * G)
    t = np.float32(a / den)
    vals = [Fraction(0)] + []
    e4 = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        e4.append(Fraction(m, 512) if e == 0 else (1 + Fraction(m, 8)) * Fraction(2) ** (e - 7))
    tt = min(Fraction(float(t)), Fraction(448))
    best = None
    for i, v in enumerate(e4):
        dd = abs(tt - v)
        if best is None or dd < best[0] or (dd == best[0] and i % 2 == 0):
            best = (dd, i)
    c = best[1]
    S = np.float32(np.float32(float(e4[c])) * G)
    grid = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2), Fraction(2),
            Fraction(3), Fraction(4), Fraction(6)]
    out = []
    for v in xs:
        if S == 0:
            out.append(0)
            continue
        y = np.float32(np.float32(v) / S)
        ay = min(abs(Fraction(float(y))), Fraction(6))
        bb = None
        for i, g in enumerate(grid):
            dd = abs(ay - g)
            if bb is None or dd < bb[0] or (dd == bb[0] and i % 2 == 0):
                bb = (dd, i)
        mag = bb[1]
        out.append((8 if (y < 0 and mag > 0) else 0) | mag)
    return out, c


@pytest.mark.parametrize("shape,scale", [((4, 32), 1.0), ((16, 64), 0.02), ((3, 48), 1e-3)])
def test_brute_force_tiny(shape, scale):
    rng = np.random.default_rng(11)
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    x[0, 3] *= 40                      # an outlier
    x[1, 16:32] = 0                    # a zero block
    G = nvfp4.global_scale(nvfp4.amax(x))
    q, c = nvfp4.quantize(x, G)
    for r in range(shape[0]):
        for b in range(shape[1] // 16):
            codes, sc = _brute_block(x[r, 16 * b:16 * b + 16], G)
            assert c[r, b] == sc
            assert list(q[r, 16 * b:16 * b + 16]) == codes


def test_static_scale_saturates():
    """A static G smaller than the tensor's own gives saturated scales and codes."""
    x = np.full((1, 16), 10.0, dtype=np.float32)
    q, c = nvfp4.quantize(x, np.float32(1e-3))        # t = 10/0.006 >> 448
    assert c[0, 0] == 0x7E and np.all(q == 7)


def test_zero_tensor_and_zero_blocks():
    x = np.zeros((2, 32), dtype=np.float32)
    q, c, G = nvfp4.quantize_dynamic(x)
    assert G == 1.0 and not q.any() and not c.any()
    x[1, :16] = np.linspace(-1, 1, 16)
    q, c, G = nvfp4.quantize_dynamic(x)
    assert not q[0].any() and not c[0].any() and not q[1, 16:].any() and c[1, 1] == 0


def test_underflowing_block_scale_gives_zero_codes():
    G = np.float32(1.0)
    x = np.full((1, 16), 1e-3 * 6 * 2.0 ** -10, dtype=np.float32)    # t far below 2**-10
    q, c = nvfp4.quantize(x, G)
    assert c[0, 0] == 0 and not q.any()


def test_dynamic_global_scale_formula():
    rng = np.random.default_rng(12)
    x = rng.standard_normal((8, 64)).astype(np.float32)
    q, c, G = nvfp4.quantize_dynamic(x)
    assert G == np.float32(np.float32(np.abs(x).max()) / np.float32(2688.0))
    # the tensor maximum maps to a scale at or just below the top of E4M3
    assert formats.e4m3_decode(c).max() <= 448.0


def test_invariants_random():
    rng = np.random.default_rng(13)
    x = rng.standard_normal((256, 4096)).astype(np.float32)
    x[:, rng.choice(4096, 20, replace=False)] *= 30
    q, c, G = nvfp4.quantize_dynamic(x)
    assert q.max() <= 15 and c.max() <= 0x7E
    assert not np.any(q == 8)                          # zero magnitude never carries a sign
    xh = nvfp4.dequantize(q, c, G)
    S = formats.e4m3_decode(c) * np.float64(G)
    normal = (c >= 0x08) & (c < 0x7E)
    err = np.abs(xh - x.astype(np.float64)).reshape(256, 256, 16).max(-1)
    assert np.all(err[normal] <= S[normal])            # half of the widest E2M1 gap is 1
    # sign symmetry
    qn, cn = nvfp4.quantize(-x, G)
    assert np.array_equal(cn, c)
    assert np.array_equal(qn, np.where(q & 7, q ^ 8, q))
    # idempotence under the same G (normal, unsaturated scales)
    q2, c2 = nvfp4.quantize(xh.astype(np.float32), G)
    rows = normal.all(axis=1)
    assert np.array_equal(q2[rows], q[rows]) and np.array_equal(c2[rows], c[rows])


def test_idempotence_recomputed_G():
    rng = np.random.default_rng(14)
    x = rng.standard_normal((64, 512)).astype(np.float32)
    q, c, G = nvfp4.quantize_dynamic(x)
    xh = nvfp4.dequantize(q, c, G).astype(np.float32)
    q2, c2, G2 = nvfp4.quantize_dynamic(xh)
    assert np.array_equal(q2, q) and np.array_equal(c2, c)


def test_nibble_packing_layout():
    codes = np.array([[1, 2, 3, 4, 15, 0]], dtype=np.uint8)
    p = nvfp4.pack_nibbles(codes)
    assert list(p[0]) == [0x21, 0x43, 0x0F]
    assert np.array_equal(nvfp4.unpack_nibbles(p), codes)


def test_dequantize_values():
    q = np.array([[7, 15] + [0] * 14], dtype=np.uint8)
    c = np.array([[0x38]], dtype=np.uint8)       # 1.0
    xh = nvfp4.dequantize(q, c, np.float32(0.5))
    assert xh[0, 0] == 3.0 and xh[0, 1] == -3.0


def test_bf16_activation_path():
    from synth import bf16_bits_from_f32
    x = np.array([[1.5, -2.25] + [0.0] * 14], dtype=np.float32)
    bits = bf16_bits_from_f32(x)
    q, c, G = nvfp4.quantize_bf16_activations(bits)
    q2, c2, G2 = nvfp4.quantize_dynamic(x)
    assert np.array_equal(q, q2) and np.array_equal(c, c2) and G == G2
