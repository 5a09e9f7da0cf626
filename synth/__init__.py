"""Seeded synthetic inputs for the Sherry 3:4 ternary product.

This module holds input generation only: none of the method's arithmetic
(no code table, no packing, no quantization, no product).  Both the oracle
side (tests, CPU baseline) and the GPU side (tests, benchmark) draw their
inputs here, so that the two sides see the same numbers.

Workload recipes follow the LLaMA-3.2 projection shapes the paper evaluates
(Sec. 4.1, LLaMA-3.2-1B and 3B) plus an 8B-scale stress shape:

* ternary weights: per block of 4 along the reduction dimension, the zero
  position is uniform in {0..3} and the three other weights are uniform +-1
  (the 3:4 constraint of Eq. 3 with no preference between patterns);
* per-tensor weight scale: U(0.01, 0.05), or fixed;
* activations: fp32 N(0, 1) per token, optionally with 1% of the channels
  scaled by 20 for every token (outlier channels).

Every draw is keyed by (seed, name...) through numpy's SeedSequence, so a
tensor can be regenerated alone, in any order.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

DEFAULT_SEED = 20260107


def _rng(seed: int, *key) -> np.random.Generator:
    h = hashlib.sha256(repr((int(seed),) + tuple(key)).encode()).digest()
    words = [int.from_bytes(h[i:i + 4], "little") for i in range(0, 32, 4)]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(words)))


def ternary_34(n: int, k: int, seed: int = DEFAULT_SEED, *key) -> np.ndarray:
    """int8 [n][k] in {-1,0,+1}; each 4-block along k has exactly one zero."""
    if k % 4:
        raise ValueError("k must be a multiple of 4")
    rng = _rng(seed, "ternary", n, k, *key)
    bits = rng.integers(0, 256, size=(n, k // 4), dtype=np.uint8)
    # bits 0-1: zero position; bits 2-5: one sign bit per position
    t = np.empty((n, k // 4, 4), dtype=np.int8)
    for p in range(4):
        t[:, :, p] = 1 - 2 * ((bits >> (2 + p)) & 1).astype(np.int8)
    zpos = (bits & 3).astype(np.intp)
    np.put_along_axis(t, zpos[:, :, None], 0, axis=2)
    return t.reshape(n, k)


def ternary_any(n: int, k: int, seed: int = DEFAULT_SEED, *key) -> np.ndarray:
    """int8 [n][k] in {-1,0,+1} with no block constraint (error-path tests)."""
    rng = _rng(seed, "ternary_any", n, k, *key)
    return rng.integers(-1, 2, size=(n, k), dtype=np.int8)


def weight_scale(seed: int = DEFAULT_SEED, *key, lo=0.01, hi=0.05) -> float:
    rng = _rng(seed, "wscale", *key)
    return float(np.float32(rng.uniform(lo, hi)))


def activations(m: int, k: int, seed: int = DEFAULT_SEED, *key,
                outlier_frac: float = 0.0, outlier_gain: float = 20.0) -> np.ndarray:
    """fp32 [m][k] ~ N(0,1); optionally round(outlier_frac*k) channels x gain."""
    rng = _rng(seed, "act", m, k, *key)
    x = rng.standard_normal(size=(m, k), dtype=np.float32)
    n_out = int(round(outlier_frac * k))
    if n_out:
        ch = _rng(seed, "outlier_ch", k, *key).choice(k, size=n_out, replace=False)
        x[:, ch] *= np.float32(outlier_gain)
    return x


def int8_any(m: int, k: int, seed: int = DEFAULT_SEED, *key, lo=-128, hi=127) -> np.ndarray:
    """Uniform int8 [m][k] in [lo, hi] (already-quantized activations)."""
    rng = _rng(seed, "int8", m, k, *key)
    return rng.integers(lo, hi + 1, size=(m, k), dtype=np.int8)


def dense_weights(n: int, k: int, seed: int = DEFAULT_SEED, *key) -> np.ndarray:
    """fp32 [n][k] ~ N(0, 0.02^2): latent full-precision weights."""
    rng = _rng(seed, "dense", n, k, *key)
    return (rng.standard_normal(size=(n, k), dtype=np.float32) * np.float32(0.02))


# --------------------------------------------------------------------------
# Workloads: the linear layers of a decoder block at LLaMA-3.2 shapes
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Linear:
    name: str
    n: int  # output features (rows of T)
    k: int  # input features (reduction dimension)


def llama_block(hidden: int, kv: int, inter: int) -> list[Linear]:
    return [
        Linear("q", hidden, hidden),
        Linear("k", kv, hidden),
        Linear("v", kv, hidden),
        Linear("o", hidden, hidden),
        Linear("gate", inter, hidden),
        Linear("up", inter, hidden),
        Linear("down", hidden, inter),
    ]


# LLaMA-3.2-1B: hidden 2048, 8 KV heads x 64 = 512, intermediate 8192, 16 layers
LLAMA_1B = dict(hidden=2048, kv=512, inter=8192, layers=16)
# LLaMA-3.2-3B: hidden 3072, 8 KV heads x 128 = 1024, intermediate 8192, 28 layers
LLAMA_3B = dict(hidden=3072, kv=1024, inter=8192, layers=28)
# 8B-scale stress: hidden 4096, kv 1024, intermediate 14336, 32 layers
STRESS_8B = dict(hidden=4096, kv=1024, inter=14336, layers=32)


def model_linears(spec: dict) -> list[tuple[int, Linear]]:
    """(layer, Linear) for every linear layer of every decoder block."""
    blk = llama_block(spec["hidden"], spec["kv"], spec["inter"])
    return [(layer, lin) for layer in range(spec["layers"]) for lin in blk]
