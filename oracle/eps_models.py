"""Synthetic noise-prediction networks eps(x, j) (oracle; test infrastructure only).

The paper evaluates the Stable Diffusion v1.5 UNet (Sec. 3.2); its weights are not
available, so two synthetic networks stand in for it (readings where the paper is silent):

* linear:    eps_j(x) = c_j * x, one fp32 multiply per element (exact in fp64, then
             rounded once to the storage type);
* patch-MLP: 2x2 patchify -> 16 features per token; h1 = GELU(bf16(x) W1 + e_j);
             h2 = GELU(bf16(h1) W2); eps_tok = bf16(h2) W3; unpatchify. e_j is the
             128-d sinusoidal embedding of the sampling timestep t_j projected by Wt.
             GELU is the erf form. Weights are bf16 values; every dot product is
             accumulated in float64 and rounded once to fp32; each activation is
             rounded to fp32 first and then to bf16 (nearest even) before it feeds the
             next product, as the device computes it.

All functions are written for clarity, not speed.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf

F64 = np.float64
F32 = np.float32


# --------------------------------------------------------------------------- bf16
def bf16_round(x) -> np.ndarray:
    """Round fp32 values to the nearest bf16 value (ties to even); returns fp32.

    Adding 0x7FFF plus the lowest kept bit to the fp32 bit pattern and clearing the low 16
    bits rounds to nearest even. In 32-bit arithmetic only NaN patterns can wrap around;
    they are passed through unchanged."""
    a = np.ascontiguousarray(x, dtype=F32)
    u = a.view(np.uint32)
    r = ((u + (((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF))) & np.uint32(0xFFFF0000)).view(F32)
    return np.where(np.isnan(a), a, r).reshape(a.shape)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns -> float64 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(F32).astype(F64)


# --------------------------------------------------------------------------- linear
def linear_eps(c):
    """eps_j(x) = c_j * x for a batch; ``c`` holds one coefficient per sampling step."""
    c64 = np.asarray(c, dtype=F64)

    def eps(X, steps):
        X = np.asarray(X)
        out = c64[np.asarray(steps)][:, None] * X.astype(F64)
        return out.astype(X.dtype)

    return eps


# --------------------------------------------------------------------------- patch-MLP
def patchify(x: np.ndarray, p: int = 2) -> np.ndarray:
    """[C, H, W] -> [(H/p)(W/p), C p p]; token = hp (W/p) + wp, feature = c p^2 + dh p + dw."""
    C, H, W = x.shape
    t = x.reshape(C, H // p, p, W // p, p).transpose(1, 3, 0, 2, 4)
    return t.reshape((H // p) * (W // p), C * p * p)


def unpatchify(tok: np.ndarray, shape, p: int = 2) -> np.ndarray:
    """Inverse of :func:`patchify`."""
    C, H, W = shape
    t = tok.reshape(H // p, W // p, C, p, p).transpose(2, 0, 3, 1, 4)
    return t.reshape(C, H, W)


def timestep_embedding(t, dim: int = 128) -> np.ndarray:
    """Sinusoidal embedding: sin(t w_k) for k < dim/2, cos(t w_{k-dim/2}) above,
    w_k = exp(-ln(10000) k / (dim/2)). float64, shape [len(t), dim]."""
    half = dim // 2
    t = np.atleast_1d(np.asarray(t, dtype=F64))
    w = np.exp(-math.log(10000.0) * np.arange(half, dtype=F64) / half)
    arg = t[:, None] * w[None, :]
    return np.concatenate([np.sin(arg), np.cos(arg)], axis=1)


def gelu(x) -> np.ndarray:
    """Erf GELU in float64: 0.5 x (1 + erf(x / sqrt 2))."""
    x = np.asarray(x, dtype=F64)
    return 0.5 * x * (1.0 + _erf(x / math.sqrt(2.0)))


class PatchMLP:
    """The synthetic patch-MLP eps-network (weights as bf16 bit patterns, [in][out])."""

    def __init__(self, weights: dict, t_values, latent_shape, patch: int = 2):
        self.W1 = bf16_bits_to_f64(weights["w1"])
        self.Wt = bf16_bits_to_f64(weights["wt"])
        self.W2 = bf16_bits_to_f64(weights["w2"])
        self.W3 = bf16_bits_to_f64(weights["w3"])
        self.shape = tuple(latent_shape)
        self.p = patch
        self.t_values = np.asarray(t_values)
        # e_j = fp32(temb(t_j) Wt): one row per sampling step.
        emb = timestep_embedding(self.t_values, self.Wt.shape[0])
        self.temb = (emb @ self.Wt).astype(F32)

    def eval_one(self, x_flat: np.ndarray, j: int) -> np.ndarray:
        """eps for one latent (flat fp32 [D]) at sampling step j -> flat fp32 [D]."""
        tok = patchify(np.asarray(x_flat, dtype=F32).reshape(self.shape), self.p)
        xb = bf16_round(tok).astype(F64)
        pre1 = (xb @ self.W1 + self.temb[j].astype(F64)).astype(F32)
        h1 = bf16_round(gelu(pre1).astype(F32)).astype(F64)
        pre2 = (h1 @ self.W2).astype(F32)
        h2 = bf16_round(gelu(pre2).astype(F32)).astype(F64)
        out = (h2 @ self.W3).astype(F32)
        return unpatchify(out, self.shape, self.p).reshape(-1)

    def __call__(self, X, steps):
        X = np.asarray(X)
        out = np.empty(X.shape, dtype=X.dtype)
        for r, j in enumerate(steps):
            out[r] = self.eval_one(X[r], int(j)).astype(X.dtype)
        return out
