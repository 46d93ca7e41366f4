"""Cached Picard sliding-window sampler, step by step (oracle; test infrastructure only).

Follows Sec. 2.1 (Eq. (1) Picard iteration, the sliding window of P timesteps and the
Eq. (2) convergence test) and Sec. 2.2 (Eq. (3) output cache, Eq. (4) mean absolute
deviation, first-entry miss rule, Eq. (5) hit/miss partition, Eq. (6) assembly, one
batched evaluation of the misses, Eq. (7) miss-only cache update, and the drift taken
at the current latent with the assembled network output).

Readings where the paper is silent:

* the drift of Eq. (1) is the DDIM one-step increment d_i = alpha_i x_i + b_i eps_i;
* the Picard sum is anchored at the window start s (whose state is final);
* window: drift points s..e-1 with e = min(s + P, T); states s+1..e are updated;
* residual r_t = mean((x_t^k - x_t^{k-1})^2) for t = s+1..e (Eq. (2), literal, '<= tau');
* slide: s' = s + 1 + c, c = number of leading t in s+1..e-1 with r_t <= tau;
* states that enter the window start as copies of the newest computed state;
* misses are listed in ascending t; hit test is strict '<' (Eq. (5)).

Stochastic steps (a reading; the paper names DDPM but prints no step): with pre-drawn step noise z_i and scale sigma_i the drift
gains the term sigma_i z_i, which is the same in every sweep; ``noise`` below is the array
of those terms, [T, D] (None for the deterministic sampler).

Storage is ``store_dtype`` (fp32 like the device, or fp64 for closed-form checks); all
arithmetic is float64 with one rounding on store.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

F64 = np.float64


@dataclass
class State:
    X: np.ndarray        # [T+1, D] trajectory estimate x_t^k, state 0 = initial noise
    Xh: np.ndarray       # [T, D]   cached inputs  x^_t   (Eq. (3))
    Eh: np.ndarray       # [T, D]   cached outputs eps^_t (Eq. (3))
    valid: np.ndarray    # [T] bool: t has a cache entry (evaluated at least once)
    s: int = 0           # window start (state s is final)
    newest: int = 0      # highest state index computed so far
    nfe: int = 0
    hits: int = 0
    sweeps: int = 0

    @property
    def T(self) -> int:
        return self.X.shape[0] - 1

    @property
    def done(self) -> bool:
        return self.s >= self.T


def init_state(x_init, T: int, store_dtype=np.float32) -> State:
    """State before the first sweep: only state 0 is known."""
    x = np.asarray(x_init, dtype=store_dtype).reshape(-1)
    D = x.size
    X = np.zeros((T + 1, D), dtype=store_dtype)
    X[0] = x
    return State(X=X, Xh=np.zeros((T, D), store_dtype), Eh=np.zeros((T, D), store_dtype),
                 valid=np.zeros(T, dtype=bool))


def window_end(s: int, T: int, P: int) -> int:
    return min(s + P, T)


def fill_new_states(X: np.ndarray, newest: int, e: int) -> None:
    """Initial estimate for states entering the window: copies of the newest state."""
    for t in range(newest + 1, e + 1):
        X[t] = X[newest]


def mean_abs_deviation(x, xh) -> float:
    """Eq. (4): (1/D) ||x - x^||_1."""
    x = np.asarray(x, dtype=F64)
    return float(np.abs(x - np.asarray(xh, dtype=F64)).sum() / x.size)


def cache_test(X, Xh, valid, s: int, e: int, delta: float):
    """Eq. (4)-(5) with the first-entry rule. Returns (dev, hit) over window slots
    t = s..e-1; dev is NaN for a timestep that has no cache entry yet."""
    W = e - s
    dev = np.full(W, np.nan)
    hit = np.zeros(W, dtype=bool)
    for j in range(W):
        t = s + j
        if valid[t]:
            dev[j] = mean_abs_deviation(X[t], Xh[t])
            hit[j] = dev[j] < delta
    return dev, hit


def miss_list(hit, s: int) -> list:
    """M = W \\ H in ascending t (Eq. (5))."""
    return [s + j for j in range(len(hit)) if not hit[j]]


def cache_update(st: State, M, E) -> None:
    """Eq. (7): C[t] <- (x_t^k, eps_t^k) for t in M only."""
    for r, t in enumerate(M):
        st.Xh[t] = st.X[t]
        st.Eh[t] = E[r]
        st.valid[t] = True


def step_noise_terms(sigma, Z) -> np.ndarray:
    """sigma_i z_i for every step i (float64), from the scales and the pre-drawn noise."""
    return np.asarray(sigma, dtype=F64)[:, None] * np.asarray(Z, dtype=F64)


def picard_update(X, Eh, s: int, e: int, alpha, b, noise=None) -> np.ndarray:
    """Eq. (1) over the window, anchored at state s:
    x_{t+1}^{k+1} = x_s + sum_{i=s}^{t} (alpha_i x_i^k + b_i eps_i^k [+ sigma_i z_i]), t = s..e-1.
    Overwrites X[s+1..e]; returns the Eq. (2) residuals r for states s+1..e."""
    acc = X[s].astype(F64)
    Y = np.empty((e - s, X.shape[1]), dtype=X.dtype)
    for j in range(e - s):
        t = s + j
        d = float(alpha[t]) * X[t].astype(F64) + float(b[t]) * Eh[t].astype(F64)
        if noise is not None:
            d = d + noise[t]
        acc = acc + d
        Y[j] = acc
    r = np.empty(e - s)
    for j in range(e - s):
        diff = Y[j].astype(F64) - X[s + 1 + j].astype(F64)
        r[j] = float(np.mean(diff * diff))
    X[s + 1:e + 1] = Y
    return r


def leading_converged(r, tau: float) -> int:
    """Number of leading residuals r_{s+1}, r_{s+2}, ... (states s+1..e-1) with r <= tau.
    ``r`` is indexed by state s+1..e; the last entry (state e) does not decide the slide."""
    c = 0
    for j in range(len(r) - 1):
        if r[j] <= tau:
            c += 1
        else:
            break
    return c


def sweep(st: State, P: int, delta: float, tau: float, alpha, b, eps_fn, *,
          force_hit=None, noise=None) -> dict:
    """One Picard sweep with the output cache. ``force_hit`` (test hook) replaces the
    hit mask computed by the cache test. Returns the sweep's trace record."""
    T = st.T
    s = st.s
    e = window_end(s, T, P)
    fill_new_states(st.X, st.newest, e)
    st.newest = max(st.newest, e)
    dev, hit = cache_test(st.X, st.Xh, st.valid, s, e, delta)
    if force_hit is not None:
        hit = np.asarray(force_hit, dtype=bool).copy()
    M = miss_list(hit, s)
    if M:
        E = eps_fn(st.X[M], M)          # one batched evaluation of the misses
        cache_update(st, M, E)
    # Eq. (6): after the update, Eh[t] is eps^_t for hits and the fresh output for misses.
    r = picard_update(st.X, st.Eh, s, e, alpha, b, noise)
    c = leading_converged(r, tau)
    s_next = s + 1 + c
    st.nfe += len(M)
    st.hits += (e - s) - len(M)
    st.sweeps += 1
    st.s = s_next
    return {"s": s, "e": e, "dev": dev, "hit": hit, "miss": list(M), "m": len(M),
            "r": r, "c": c, "s_next": s_next}


def sample(x_init, T: int, P: int, delta: float, tau: float, alpha, b, eps_fn,
           store_dtype=np.float32, max_sweeps=None, noise=None):
    """Run sweeps until the window start reaches T. Returns (x_T, trace, state)."""
    st = init_state(x_init, T, store_dtype)
    trace = []
    limit = T if max_sweeps is None else max_sweeps
    while not st.done and st.sweeps < limit:
        trace.append(sweep(st, P, delta, tau, alpha, b, eps_fn, noise=noise))
    return st.X[T].copy(), trace, st


def revisit_counts(trace, threshold: float):
    """The revisit statistic of Sec. 1 over a run's trace: (requested evaluations, revisits,
    revisits whose Eq. (4) deviation from the cached input is below ``threshold``). A window
    slot is a requested drift evaluation; it is a revisit if its timestep holds a cache
    entry (its deviation is a number, not NaN)."""
    requests = revisits = below = 0
    for rec in trace:
        dev = np.asarray(rec["dev"], dtype=F64)
        requests += dev.size
        seen = ~np.isnan(dev)
        revisits += int(np.count_nonzero(seen))
        below += int(np.count_nonzero(dev[seen] < threshold))
    return requests, revisits, below


# --------------------------------------------------------------------------- references
def picard_uncached(x_init, T: int, P: int, tau: float, alpha, b, eps_fn,
                    store_dtype=np.float32, noise=None):
    """Sliding-window Picard with no cache: every window timestep is evaluated each sweep.
    Same readings as :func:`sweep`; shares none of the cache code."""
    X = np.zeros((T + 1, np.asarray(x_init).size), dtype=store_dtype)
    X[0] = np.asarray(x_init, dtype=store_dtype).reshape(-1)
    s, newest, nfe, trace = 0, 0, 0, []
    while s < T:
        e = min(s + P, T)
        for t in range(newest + 1, e + 1):
            X[t] = X[newest]
        newest = max(newest, e)
        steps = list(range(s, e))
        E = eps_fn(X[steps], steps)
        nfe += len(steps)
        acc = X[s].astype(F64)
        Y = np.empty((e - s, X.shape[1]), dtype=store_dtype)
        for j, t in enumerate(steps):
            acc = acc + (float(alpha[t]) * X[t].astype(F64) + float(b[t]) * E[j].astype(F64))
            if noise is not None:
                acc = acc + noise[t]
            Y[j] = acc
        r = np.array([float(np.mean((Y[j].astype(F64) - X[s + 1 + j].astype(F64)) ** 2))
                      for j in range(e - s)])
        X[s + 1:e + 1] = Y
        c = 0
        while c < e - s - 1 and r[c] <= tau:
            c += 1
        trace.append({"s": s, "e": e, "r": r, "c": c, "s_next": s + 1 + c})
        s = s + 1 + c
    return X[T].copy(), trace, nfe


def ddim_serial_drift(x_init, alpha, b, eps_fn, store_dtype=np.float32, noise=None):
    """Serial DDIM in drift form: x_{i+1} = x_i + (alpha_i x_i + b_i eps_i [+ sigma_i z_i])."""
    x = np.asarray(x_init, dtype=store_dtype).reshape(-1)
    for i in range(len(alpha)):
        e = eps_fn(x[None, :], [i])[0]
        d = float(alpha[i]) * x.astype(F64) + float(b[i]) * e.astype(F64)
        if noise is not None:
            d = d + noise[i]
        x = (x.astype(F64) + d).astype(store_dtype)
    return x


def ddpm_serial_textbook(x_init, ab, eps_fn, Z, store_dtype=np.float32):
    """Serial ancestral DDPM in its textbook form over the sampler's states: with
    beta'_i = 1 - ab_i / ab_{i+1} (the step's beta on the possibly respaced grid),
    x_{i+1} = (x_i - beta'_i / sqrt(1 - ab_i) eps) / sqrt(1 - beta'_i) + s_i z_i,
    s_i^2 = beta'_i (1 - ab_{i+1}) / (1 - ab_i) (the posterior variance)."""
    x = np.asarray(x_init, dtype=store_dtype).reshape(-1)
    ab = np.asarray(ab, dtype=F64)
    for i in range(len(ab) - 1):
        e = eps_fn(x[None, :], [i])[0].astype(F64)
        beta = 1.0 - ab[i] / ab[i + 1]
        mean = (x.astype(F64) - beta / np.sqrt(1.0 - ab[i]) * e) / np.sqrt(1.0 - beta)
        var = beta * (1.0 - ab[i + 1]) / (1.0 - ab[i])
        x = (mean + np.sqrt(var) * np.asarray(Z[i], dtype=F64)).astype(store_dtype)
    return x


def ddim_serial_textbook(x_init, ab, eps_fn, store_dtype=np.float32):
    """Serial deterministic DDIM in its textbook form:
    x0^ = (x_i - sqrt(1 - ab_i) eps) / sqrt(ab_i); x_{i+1} = sqrt(ab_{i+1}) x0^ + sqrt(1 - ab_{i+1}) eps."""
    x = np.asarray(x_init, dtype=store_dtype).reshape(-1)
    ab = np.asarray(ab, dtype=F64)
    for i in range(len(ab) - 1):
        e = eps_fn(x[None, :], [i])[0].astype(F64)
        x0 = (x.astype(F64) - np.sqrt(1.0 - ab[i]) * e) / np.sqrt(ab[i])
        x = (np.sqrt(ab[i + 1]) * x0 + np.sqrt(1.0 - ab[i + 1]) * e).astype(store_dtype)
    return x
