"""Scalar simulator of the cached Picard sampler for the linear network (oracle pin).

With eps_j(x) = c_j x every state, cached input and cached output stays a scalar
multiple of the initial latent x0: x_t = g_t x0, x^_t = gh_t x0, eps^_t = c_t gh_t x0.
The quantities that decide the control flow then reduce to scalars:

* Eq. (4):  delta_t = |g_t - gh_t| * mean|x0|
* Eq. (2):  r_t     = (g_t^new - g_t^old)^2 * mean(x0^2)
* Eq. (1):  g_{t+1} = g_s + sum_{i=s}^{t} (alpha_i g_i + b_i c_i gh_i)

This is a separate, scalar formulation of the same sampler, written without the
D-dimensional code; the tests run both on tiny grids and require the same decisions
(hit masks, miss lists, window positions, counters). Float64 throughout.
"""
from __future__ import annotations

import numpy as np


def simulate(x0, T: int, P: int, delta: float, tau: float, alpha, b, c):
    x0 = np.asarray(x0, dtype=np.float64).reshape(-1)
    m1 = float(np.mean(np.abs(x0)))
    m2 = float(np.mean(x0 * x0))
    g = [0.0] * (T + 1)
    gh = [0.0] * T
    seen = [False] * T
    g[0] = 1.0
    known = 0                       # highest state with an estimate
    s = 0
    nfe = hits = sweeps = 0
    records = []
    while s < T:
        e = min(s + P, T)
        while known < e:            # new states start as copies of the newest one
            known += 1
            g[known] = g[known - 1]
        hit_mask, dev, miss = [], [], []
        for t in range(s, e):
            if seen[t]:
                d = abs(g[t] - gh[t]) * m1
                dev.append(d)
                h = d < delta
            else:
                dev.append(float("nan"))
                h = False
            hit_mask.append(h)
            if not h:
                miss.append(t)
        for t in miss:              # evaluate the misses, refresh their cache entries
            gh[t] = g[t]
            seen[t] = True
        new = [0.0] * (e - s)
        run = g[s]
        for k, t in enumerate(range(s, e)):
            run += alpha[t] * g[t] + b[t] * c[t] * gh[t]
            new[k] = run
        r = [(new[k] - g[s + 1 + k]) ** 2 * m2 for k in range(e - s)]
        for k in range(e - s):
            g[s + 1 + k] = new[k]
        cnt = 0
        for k in range(e - s - 1):
            if r[k] <= tau:
                cnt += 1
            else:
                break
        nfe += len(miss)
        hits += (e - s) - len(miss)
        sweeps += 1
        records.append({"s": s, "e": e, "hit": hit_mask, "dev": dev, "miss": miss,
                        "r": r, "c": cnt, "s_next": s + 1 + cnt})
        s = s + 1 + cnt
    return {"gamma_T": g[T], "records": records, "nfe": nfe, "hits": hits, "sweeps": sweeps}


def serial_gain(alpha, b, c) -> float:
    """Closed form of serial DDIM with the linear network: x_T = prod_j (1 + alpha_j + b_j c_j) x0."""
    return float(np.prod(1.0 + np.asarray(alpha) + np.asarray(b) * np.asarray(c)))
