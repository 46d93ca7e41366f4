"""Derivation of the erf-GELU constants used by k_epsnet.hip (run by hand; not a build step).

    python paper_2609_36522_amd/csrc/gelu_fit.py

GELU(x) = x Phi(x) = max(x, 0) - a Q(a),  a = |x|,  Q(a) = 1 - Phi(a) the normal upper tail.
The kernel evaluates Q(a) = 2^(-P(min(a, A_MAX))) with P a polynomial in a, i.e. one v_exp_f32
and a Horner chain of fused multiply-adds. P is fitted to -log2(Q(a)) on [0, A_MAX] by
iteratively reweighted least squares toward the minimax (equal-ripple) solution of the
absolute error of P, which is the relative error of Q (times ln 2). Above A_MAX,
a Q(a) < 2.2e-7 a, so clamping the argument costs at most that much.

Prints the coefficients (low to high degree, as float32 literals) and the accuracy of the
float32 evaluation against scipy's erf in float64.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf, erfc

A_MAX = 5.0
DEG = 7


def fit(deg=DEG, amax=A_MAX, iters=60):
    a = 0.5 * amax * (1 - np.cos(np.linspace(0, np.pi, 20001)))     # Chebyshev-spaced
    target = -np.log2(0.5 * erfc(a / np.sqrt(2.0)))
    V = np.polynomial.chebyshev.chebvander(2 * a / amax - 1, deg)
    w = np.ones_like(a)
    for _ in range(iters):
        c, *_ = np.linalg.lstsq(V * w[:, None], target * w, rcond=None)
        r = np.abs(V @ c - target)
        w = w * (r / r.max() + 1e-3) ** 0.5
        w /= w.max()
    poly = np.polynomial.chebyshev.Chebyshev(c, domain=[0, amax]).convert(
        kind=np.polynomial.Polynomial).coef
    return poly.astype(np.float32)


def gelu_f32(x, coef, amax=A_MAX):
    f32 = np.float32
    x = x.astype(f32)
    a = np.minimum(np.abs(x), f32(amax))
    p = np.full_like(a, coef[-1])
    for k in range(len(coef) - 2, -1, -1):
        p = (p * a + coef[k]).astype(f32)
    q = np.exp2(-p.astype(np.float64)).astype(f32)          # v_exp_f32 ~ correctly rounded
    return (np.maximum(x, f32(0)) - np.abs(x) * q).astype(f32)


def report(coef):
    x = np.linspace(-12, 12, 2_400_001)
    ref = 0.5 * x * (1 + erf(x / np.sqrt(2)))
    g = gelu_f32(x, coef).astype(np.float64)
    e = np.abs(g - ref)
    rel = e / np.maximum(np.abs(ref), 1e-300)
    print(f"max |err| / max(1,|x|)      = {np.max(e / np.maximum(np.abs(x), 1)):.3e}")
    print(f"max rel err, x > 0.01       = {rel[x > 0.01].max():.3e}")
    print(f"max rel err, -4 < x < -0.01 = {rel[(x < -0.01) & (x > -4)].max():.3e}")


if __name__ == "__main__":
    c = fit()
    print("coefficients (low -> high):")
    for k, v in enumerate(c):
        print(f"  c{k} = {float(v)!r}f")
    report(c)
