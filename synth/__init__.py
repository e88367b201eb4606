"""Seeded synthetic inputs for the phase-specific quantized linear layer.

This module is shared by the CPU oracle (``oracle/``), the tests, the
benchmark and the smoke entry point.  It holds only input generation:
random draws, the outlier-channel pattern, and the bf16 encoding of
activations.  None of the quantization method's arithmetic lives here.

Shapes follow the layer shapes the paper lists for Qwen3-8B
(d_model 4096, d_ffn 12288) and Qwen3.8-27B (d_model 5120, d_ffn 17408)
in its model table (App. A, "Models").  Distributions:

* weights: ``0.02 * N(0,1)`` per element, optionally times a per-row factor
  ``exp(0.3 * N(0,1))`` (a log-normal row scale), fp32;
* activations: ``N(0,1)`` per element with a fixed set of outlier channels
  (a fraction of the K columns, chosen without replacement) multiplied by a
  constant factor, built in fp32 and rounded to bf16 (round to nearest even).

Every draw is keyed by ``numpy.random.default_rng([seed, stream, tag, index])``
(PCG64) so that any tensor can be regenerated independently of the others.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

# Tags keep the RNG streams of different tensors apart.
TAG_WEIGHT = 1
TAG_ROWSCALE = 2
TAG_ACT = 3
TAG_CHANNELS = 4
TAG_DECODE_X = 5
TAG_CALIB = 6
TAG_ATTN_OUT = 7

CALIB_SEED_OFFSET = 1000


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return the raw bits.

    Inputs are finite by construction.  This is an input encoding, not part
    of the method.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, stream: int, tag: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng([seed, stream, tag, index])


def outlier_count(frac: float, k: int) -> int:
    """Number of outlier channels: ``round(frac * k)`` with ties to even."""
    return int(np.round(frac * k))


def outlier_channels(seed: int, stream: int, k: int, frac: float) -> np.ndarray:
    n = outlier_count(frac, k)
    ch = _rng(seed, stream, TAG_CHANNELS, k).choice(k, size=n, replace=False)
    return np.sort(ch).astype(np.int64)


def weight_f32(seed: int, stream: int, n: int, k: int, *, std: float = 0.02,
               lognormal_rows: bool = True, index: int = 0) -> np.ndarray:
    """Weights ``[n, k]`` fp32 (``nn.Linear`` layout: K contiguous)."""
    z = _rng(seed, stream, TAG_WEIGHT, index).standard_normal((n, k), dtype=np.float32)
    w = z * np.float32(std)
    if lognormal_rows:
        r = np.exp(np.float32(0.3) *
                   _rng(seed, stream, TAG_ROWSCALE, index).standard_normal((n, 1), dtype=np.float32))
        w *= r.astype(np.float32)
    return w


def act_f32(seed: int, stream: int, m: int, k: int, channels: np.ndarray,
            factor: float, *, tag: int = TAG_ACT, index: int = 0) -> np.ndarray:
    """Activations ``[m, k]`` in fp32 before the bf16 rounding."""
    x = _rng(seed, stream, tag, index).standard_normal((m, k), dtype=np.float32)
    if len(channels):
        x[:, channels] *= np.float32(factor)
    return x


def act_bf16(seed: int, stream: int, m: int, k: int, channels: np.ndarray,
             factor: float, *, tag: int = TAG_ACT, index: int = 0) -> np.ndarray:
    """Activations as bf16 bit patterns (``uint16``), shape ``[m, k]``."""
    return bf16_bits_from_f32(act_f32(seed, stream, m, k, channels, factor, tag=tag, index=index))


@dataclasses.dataclass(frozen=True)
class Linear:
    """One linear layer of a workload: weight ``[n, k]`` and prefill rows ``m``."""
    name: str
    n: int
    k: int


@dataclasses.dataclass(frozen=True)
class Config:
    stream: int
    name: str
    layers: Tuple[Linear, ...]
    m: int                      # prefill tokens
    decode_batches: Tuple[int, ...]
    outlier_frac: float
    outlier_factor: float
    lognormal_rows: bool
    fused_act_quant: bool = False
    chained: bool = False
    stacked_blocks: int = 1

    @property
    def k(self) -> int:
        return self.layers[0].k


_BLOCK_27B = (
    Linear("qkv", 7168, 5120),       # q 40x128 + k 8x128 + v 8x128 heads, fused
    Linear("o", 5120, 5120),
    Linear("gate_up", 34816, 5120),  # gate 17408 + up 17408, fused
    Linear("down", 5120, 17408),
)

# The workloads, each with its own RNG stream number.
TINY_512 = Config(0, "tiny single linear 512x512", (Linear("w", 512, 512),), 128, (1,),
                  0.01, 20.0, False)
UP_8B_M2048 = Config(1, "8B-scale MLP up-projection K=4096 N=12288 M=2048",
                     (Linear("up", 12288, 4096),), 2048, (1, 4), 0.005, 30.0, True)
DOWN_27B_M8192 = Config(2, "27B-scale MLP down-projection K=17408 N=5120 M=8192",
                        (Linear("down", 5120, 17408),), 8192, (1,), 0.005, 30.0, True,
                        fused_act_quant=True)
BLOCK_27B_M4096 = Config(3, "27B-scale dense block linear set, M=4096", _BLOCK_27B, 4096, (1,),
                         0.005, 30.0, True, chained=True)
STACK_27B_M32768 = Config(4, "decode sweep over 64 stacked 27B-scale blocks + prefill M=32768",
                          _BLOCK_27B, 32768, (1, 8, 16), 0.005, 30.0, True, stacked_blocks=64)
WORKLOADS: Tuple[Config, ...] = (TINY_512, UP_8B_M2048, DOWN_27B_M8192, BLOCK_27B_M4096, STACK_27B_M32768)


def channels_for(cfg: Config, k: int, seed: int = 0) -> np.ndarray:
    return outlier_channels(seed, cfg.stream, k, cfg.outlier_frac)


def layer_weight(cfg: Config, layer: Linear, seed: int = 0, block: int = 0) -> np.ndarray:
    index = block * 16 + [l.name for l in cfg.layers].index(layer.name)
    std = 0.02
    return weight_f32(seed, cfg.stream, layer.n, layer.k, std=std,
                      lognormal_rows=cfg.lognormal_rows, index=index)


def prefill_x(cfg: Config, k: int, m: Optional[int] = None, seed: int = 0,
              calib: bool = False) -> np.ndarray:
    """bf16 prefill activations ``[m, k]``; ``calib=True`` draws the calibration batch."""
    m = cfg.m if m is None else m
    ch = channels_for(cfg, k, seed)
    s = seed + (CALIB_SEED_OFFSET if calib else 0)
    tag = TAG_CALIB if calib else TAG_ACT
    return act_bf16(s, cfg.stream, m, k, ch, cfg.outlier_factor, tag=tag, index=k)


def decode_x(cfg: Config, k: int, batch: int, seed: int = 0) -> np.ndarray:
    ch = channels_for(cfg, k, seed)
    return act_bf16(seed, cfg.stream, batch, k, ch, cfg.outlier_factor,
                    tag=TAG_DECODE_X, index=k * 64 + batch)


def attn_out_standin(cfg: Config, m: int, k: int, seed: int = 0) -> np.ndarray:
    """Synthetic N(0,1) stand-in for an attention output (input of ``o``)."""
    return act_bf16(seed, cfg.stream, m, k, np.zeros(0, np.int64), 1.0, tag=TAG_ATTN_OUT, index=k)


def random_f32(seed: int, shape: Tuple[int, ...], scale: float = 1.0, tag: int = 99) -> np.ndarray:
    """Generic seeded fp32 normal tensor for parity tests at arbitrary shapes."""
    return (_rng(seed, 0, tag).standard_normal(shape, dtype=np.float32) * np.float32(scale))


def random_bf16(seed: int, shape: Tuple[int, ...], scale: float = 1.0,
                outlier_frac: float = 0.0, outlier_factor: float = 1.0, tag: int = 98) -> np.ndarray:
    x = random_f32(seed, shape, scale, tag)
    if outlier_frac > 0:
        ch = outlier_channels(seed, 0, shape[-1], outlier_frac)
        x[..., ch] *= np.float32(outlier_factor)
    return bf16_bits_from_f32(x)


__all__: List[str] = [n for n in dir() if not n.startswith("_")]
