"""Derivation of the erf-GELU constants used by k_epsnet.hip (run by hand; not a build step).

    python paper_2609_36522_amd/csrc/gelu_fit.py

GELU(x) = x Phi(x) = max(x, 0) - a Q(a),  a = |x|,  Q(a) = 1 - Phi(a) the normal upper tail.
The kernels evaluate twice the GELU,

    2 GELU(x) = (x + a) - a 2Q(a),   2Q(a) = 2^(-(P(a) - 1)),

with P a polynomial in a: one v_add_f32 (x + a = 2 max(x, 0) exactly), a Horner chain of
fused multiply-adds whose constant term is lowered by 1, one v_exp_f32 and one last FMA. The
factor 2 is exact and is undone in the next product (the following weight matrix is stored
halved).

What the fit minimizes. Every GELU output is rounded to bf16 next, and what an error costs
downstream is the chance that it moves a value across a bf16 rounding boundary times the size
of that step: both scale with the value, so the expected effect of an error is its absolute
size. An error dP of P changes the result by a 2Q(a) ln2 dP (absolute), so P is fitted to
-log2 Q(a) on [0, A_MAX] toward the minimax (equal-ripple) solution of the absolute error
weighted by a 2Q(a) ln 2 (floored at FLOOR so that P keeps tracking -log2 Q at large a), by
iteratively reweighted least squares. Against an unweighted fit of the same degree (uniform
relative error of Q) this lowers the absolute error of the result about threefold at the same
cost. The argument is not clamped: the script checks that P increases monotonically well
beyond A_MAX and keeps tracking -log2 Q there, so that a Q(a) stays tiny (and P overflows to
+inf, Q to 0, for huge a).

Prints the coefficients (low to high degree, as float32 literals), the constant term used by
the kernels, and the accuracy of the float32 evaluation against scipy's erf in float64.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf, erfc

A_MAX = 7.0
DEG = 7
FLOOR = 1e-4


def fit(deg=DEG, amax=A_MAX, floor=FLOOR, iters=80):
    a = 0.5 * amax * (1 - np.cos(np.linspace(0, np.pi, 40001)))     # Chebyshev-spaced
    q = 0.5 * erfc(a / np.sqrt(2.0))
    target = -np.log2(q)
    wt = np.maximum(a * 2.0 * q * np.log(2.0), floor)             # |d result / d P|
    V = np.polynomial.chebyshev.chebvander(2 * a / amax - 1, deg)
    w = wt.copy()
    for _ in range(iters):
        c, *_ = np.linalg.lstsq(V * w[:, None], target * w, rcond=None)
        r = np.abs(V @ c - target) * wt
        w = w * (r / r.max() + 1e-3) ** 0.5
        w /= w.max()
    poly = np.polynomial.chebyshev.Chebyshev(c, domain=[0, amax]).convert(
        kind=np.polynomial.Polynomial).coef
    return poly.astype(np.float32)


def gelu2_f32(x, coef):
    """Float32 emulation of the kernels' 2 GELU(x) (v_exp_f32 taken as correctly rounded)."""
    f32 = np.float32
    x = x.astype(f32)
    a = np.abs(x)
    c = coef.copy()
    c[0] = f32(c[0] - f32(1))                                  # P(a) - 1
    p = np.full_like(a, c[-1])
    for k in range(len(c) - 2, -1, -1):
        p = (p * a + c[k]).astype(f32)
    with np.errstate(over="ignore"):
        q2 = np.exp2(-p.astype(np.float64)).astype(f32)
    return ((x + a) - a * q2).astype(f32)


def report(coef):
    x = np.linspace(-12, 12, 2_400_001)
    ref = x * (1 + erf(x / np.sqrt(2)))                        # twice the GELU
    g = gelu2_f32(x, coef).astype(np.float64)
    e = np.abs(g - ref)
    rel = e / np.maximum(np.abs(ref), 1e-300)
    print(f"max |err| / max(1,|x|)      = {np.max(e / np.maximum(np.abs(x), 1)):.3e}")
    print(f"max rel err, x > 0.01       = {rel[x > 0.01].max():.3e}")
    print(f"max rel err, -1 < x < -0.01 = {rel[(x < -0.01) & (x > -1)].max():.3e}")
    a = np.linspace(0, 200, 2_000_001)
    P = np.polynomial.Polynomial(coef.astype(np.float64))(a)
    print(f"P increasing on [0, 200]    = {bool(np.all(np.diff(P) > 0))}")
    t = np.array([7.0, 8.0, 10.0, 12.0])
    qa = np.exp2(-np.polynomial.Polynomial(coef.astype(np.float64))(t))
    qt = 0.5 * erfc(t / np.sqrt(2.0))
    print("Q(a) fitted / exact above A_MAX: " + ", ".join(f"a={u:g}: {v:.4f}" for u, v in zip(t, qa / qt)))


if __name__ == "__main__":
    c = fit()
    print("coefficients (low -> high):")
    for k, v in enumerate(c):
        print(f"  c{k} = {float(v)!r}f")
    print(f"constant term used by the kernels (c0 - 1): {float(np.float32(c[0] - np.float32(1)))!r}f")
    report(c)
