"""Seeded synthetic inputs for the cached Picard sampler.

This module is the only code shared by the HIP path and the CPU oracle. It draws
random numbers and packs them into the storage formats the sampler consumes; it
holds none of the sampler's arithmetic (no schedule, no network, no update rule).

Generator: ``numpy.random.default_rng(seed)`` (PCG64). Seeds follow one fixed
convention so every consumer sees the same arrays:

* seed 0 -> initial latent ``x_init`` ~ N(0, 1), fp32;
* seed 1 -> linear-network coefficients ``c_j`` ~ U(0.5, 1.5) per sampling step, fp32;
* seed 2 -> patch-MLP weights, drawn in the order W1, Wt, W2, W3, each N(0, 1/fan_in)
  in fp32, then stored as bf16 bit patterns (round to nearest even);
* seed 3 -> per-step noise z ~ N(0, 1) of the stochastic sampler, [N][T][D] fp32;
* sample n of a batch draws its initial latent from seed 1000 + n (sample 0 of a batch
  is therefore not the seed-0 latent of single-sample runs).

The stand-in for the paper's Stable Diffusion v1.5 latents (4x64x64 for 512^2 images,
Sec. 3.2) is plain N(0, 1) noise of the same shape; there is no text conditioning.
"""
from __future__ import annotations

import numpy as np

SEED_X_INIT = 0
SEED_LINEAR_C = 1
SEED_WEIGHTS = 2
SEED_STEP_NOISE = 3
SEED_BATCH_BASE = 1000


def x_init(shape, seed: int = SEED_X_INIT) -> np.ndarray:
    """Initial latent of ``shape`` (C, H, W), fp32 N(0, 1)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(tuple(shape)).astype(np.float32)


def x_init_batch(shape, batch: int, base: int = SEED_BATCH_BASE) -> np.ndarray:
    """Initial latents of a batch, [batch, C, H, W] fp32; sample n uses seed base + n."""
    return np.stack([x_init(shape, base + n) for n in range(batch)])


def step_noise(batch: int, T: int, D: int, seed: int = SEED_STEP_NOISE) -> np.ndarray:
    """Per-step noise z[n][i] ~ N(0, 1) of the stochastic sampler, [batch, T, D] fp32."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((batch, T, D)).astype(np.float32)


def linear_coefficients(T: int, seed: int = SEED_LINEAR_C) -> np.ndarray:
    """c_j ~ U(0.5, 1.5) for sampling steps j = 0..T-1, drawn in ascending j, fp32."""
    rng = np.random.default_rng(seed)
    return rng.uniform(0.5, 1.5, size=T).astype(np.float32)


def _f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Pack fp32 values as bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    return ((u + bias) >> 16).astype(np.uint16)


def mlp_weights(hidden: int, in_dim: int = 16, temb_dim: int = 128,
                seed: int = SEED_WEIGHTS) -> dict:
    """Patch-MLP weights as bf16 bit patterns, row-major [in][out].

    Returns ``{"w1": [in_dim, H], "wt": [temb_dim, H], "w2": [H, H], "w3": [H, in_dim]}``
    (uint16). Each matrix is N(0, 1/fan_in) with fan_in its row count; no biases.
    """
    rng = np.random.default_rng(seed)
    shapes = (("w1", in_dim, hidden), ("wt", temb_dim, hidden),
              ("w2", hidden, hidden), ("w3", hidden, in_dim))
    out = {}
    for name, fan_in, fan_out in shapes:
        w = rng.standard_normal((fan_in, fan_out)) / np.sqrt(fan_in)
        out[name] = _f32_to_bf16_bits(w.astype(np.float32))
    return out

