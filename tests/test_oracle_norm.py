"""Pins for the RMSNorm + NVFP4 oracle (CPU only)."""
import numpy as np

from oracle import formats, norm, nvfp4
from synth import bf16_bits_from_f32


def _bits(a):
    return bf16_bits_from_f32(np.asarray(a, np.float32))


def test_constant_rows_normalize_to_gamma():
    """A row of +-c with eps = 0: ms = c^2, inv = 1/c, y = sign * gamma."""
    K = 64
    gamma = np.linspace(-2.0, 2.0, K).astype(np.float32)
    x = np.array([[0.25] * K, [-8.0] * K, [3.0] * K], np.float32)
    y = norm.rmsnorm_bf16(_bits(x), _bits(gamma), 0.0)
    g = formats.f32_from_bf16_bits(_bits(gamma).reshape(1, -1))[0]
    assert np.array_equal(y[0], g) and np.array_equal(y[1], -g)
    # 1/sqrt(9) = 1/3 rounds: y = fp32(fp32(3 * fp32(1/3)) * g)
    inv = np.float32(np.float32(1.0) / np.float32(3.0))
    assert np.array_equal(y[2], (np.float32(3.0) * inv).astype(np.float32) * g)


def test_power_of_two_scaling_is_invariant():
    """Scaling a row by 2^k (eps = 0) leaves y unchanged bit for bit."""
    rng = np.random.default_rng(60)
    K = 256
    x = rng.standard_normal((4, K)).astype(np.float32)
    gamma = (1.0 + 0.1 * rng.standard_normal(K)).astype(np.float32)
    y0 = norm.rmsnorm_bf16(_bits(x), _bits(gamma), 0.0)
    for k in (-5, 3, 11):
        yk = norm.rmsnorm_bf16(_bits(x * np.float32(2.0 ** k)), _bits(gamma), 0.0)
        assert np.array_equal(yk, y0)


def test_matches_fp64_formula():
    rng = np.random.default_rng(61)
    M, K = 8, 1024
    xb = _bits(rng.standard_normal((M, K)).astype(np.float32) * 3)
    gb = _bits((1.0 + 0.2 * rng.standard_normal(K)).astype(np.float32))
    eps = 1e-6
    y = norm.rmsnorm_bf16(xb, gb, eps).astype(np.float64)
    x = formats.f64_from_bf16_bits(xb)
    g = formats.f64_from_bf16_bits(gb.reshape(1, -1))[0]
    ref = x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps) * g
    assert np.max(np.abs(y - ref) / np.maximum(np.abs(ref), 1e-30)) < 6 * 2.0 ** -24


def test_quantize_dynamic_uses_the_normalized_amax():
    rng = np.random.default_rng(62)
    xb = _bits(rng.standard_normal((5, 96)).astype(np.float32))
    gb = _bits(np.full(96, 1.5, np.float32))
    q, c, G, y = norm.quantize_rmsnorm_bf16(xb, gb, 1e-5)
    assert G == nvfp4.global_scale(np.max(np.abs(y)))
    q2, c2 = nvfp4.quantize(y, G)
    assert np.array_equal(q, q2) and np.array_equal(c, c2)
