"""Parareal-based sampler with the output cache (oracle; test infrastructure only).

Sec. 2.1 describes Parareal-based samplers (SRDS) as a coarse solver that initializes the
trajectory and fine solvers that refine it; Sec. 2.2 applies the same cache to their
network evaluations, leaving the Parareal update rule unchanged. The paper does not print
the update rule; the textbook Parareal iteration is used (a reading):

* T sampling steps split into B blocks of L = T / B fine steps; boundary n is state nL.
* Fine propagator F_n(u): L serial DDIM steps from state nL, x_{t+1} = x_t + d_t with the
  drift d_t = alpha_t x_t + b_t eps(x_t, t) of the fine grid (the DDIM one-step increment).
* Coarse propagator G_n(u): one DDIM step from state nL to state (n+1)L,
  u + (ac_n u + bc_n eps(u, nL)), with ac_n = sqrt(ab_{(n+1)L} / ab_{nL}) - 1 and
  bc_n = sqrt(1 - ab_{(n+1)L}) - (1 + ac_n) sqrt(1 - ab_{nL}).
* Initialization: U_0 = x_init, U_{n+1} = G_n(U_n) serially.
* Iteration k = 0, 1, ...: fine solves F_n(U_n) for the blocks n >= k that are not final
  yet, all blocks advancing one fine step at a time (one batch of requests per step);
  then U_{k+1} = F_k (exact from here on), and serially for n = k+1 .. B-1:
  U_{n+1} <- G_n(U_n^new) + (F_n - G_n(U_n^old)), the predictor-corrector update.
  Blocks n <= k are final and are not recomputed (Parareal is exact after k iterations
  on them).
* Convergence: the Eq. (2) residual r_n = (1/D) ||U_n^new - U_n^old||^2 over n = k+1..B;
  stop when every r_n <= tau, or after B iterations (then the result is serial fine DDIM).
* Cache: one entry per fine-grid timestep t (Eq. (3)), consulted by every evaluation
  request, coarse or fine (a coarse step from boundary n asks for eps at t = nL, the same
  key as the first fine step of block n). Request (t, x): hit iff t has an entry and
  (1/D) ||x - x^_t||_1 < delta (Eq. (4), (5)); a miss is evaluated and replaces the entry
  (Eq. (7)). Requests of one batch have distinct timesteps and are listed ascending.

Storage fp32 (states, coarse values, cache); arithmetic float64, one rounding on store.
The coarse value G_n is stored (fp32) and the correction uses the stored value.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def coarse_coefficients(ab, B: int):
    """(ac, bc) of the coarse DDIM step of each block, from the sampler's alpha_bar."""
    ab = np.asarray(ab, dtype=F64)
    T = ab.size - 1
    L = T // B
    a0 = ab[0:T:L]
    a1 = ab[L:T + 1:L]
    ac = np.sqrt(a1 / a0) - 1.0
    bc = np.sqrt(1.0 - a1) - (1.0 + ac) * np.sqrt(1.0 - a0)
    return ac, bc


class Cache:
    """Eq. (3) cache over the fine grid with the Eq. (4)-(5) test and the Eq. (7) update."""

    def __init__(self, T, D, delta, dtype=np.float32):
        self.Xh = np.zeros((T, D), dtype)
        self.Eh = np.zeros((T, D), dtype)
        self.valid = np.zeros(T, dtype=bool)
        self.delta = delta
        self.nfe = 0
        self.hits = 0

    def request(self, ts, xs, eps_fn):
        """Serve a batch of requests (distinct timesteps ``ts``, inputs ``xs``): cached
        outputs for hits, one batched evaluation of the misses. Returns (outputs, record)."""
        dev = np.full(len(ts), np.nan)
        hit = np.zeros(len(ts), dtype=bool)
        for i, (t, x) in enumerate(zip(ts, xs)):
            if self.valid[t]:
                dev[i] = float(np.abs(np.asarray(x, F64) - self.Xh[t].astype(F64)).sum() / x.size)
                hit[i] = dev[i] < self.delta
        miss = [i for i in range(len(ts)) if not hit[i]]
        if miss:
            E = eps_fn(np.stack([xs[i] for i in miss]), [ts[i] for i in miss])
            for r, i in enumerate(miss):
                t = ts[i]
                self.Xh[t] = xs[i]
                self.Eh[t] = E[r]
                self.valid[t] = True
        self.nfe += len(miss)
        self.hits += len(ts) - len(miss)
        out = [self.Eh[t].copy() for t in ts]
        return out, {"t": list(ts), "dev": dev, "hit": hit, "miss": [ts[i] for i in miss]}


def _step(x, e, a, b, dtype):
    x64 = np.asarray(x, F64)
    return (x64 + (a * x64 + b * np.asarray(e, F64))).astype(dtype)


def sample(x_init, T: int, B: int, delta: float, tau: float, ab, alpha, b, eps_fn,
           store_dtype=np.float32, max_iters=None):
    """Cached Parareal. Returns (x_T, trace, stats); trace[0] is the initialization."""
    if T % B:
        raise ValueError("T must be a multiple of the number of blocks")
    L = T // B
    ac, bc = coarse_coefficients(ab, B)
    x0 = np.asarray(x_init, store_dtype).reshape(-1)
    D = x0.size
    cache = Cache(T, D, delta, store_dtype)
    U = np.zeros((B + 1, D), store_dtype)
    G = np.zeros((B, D), store_dtype)
    U[0] = x0
    trace = []
    # initialization: serial coarse sweep
    init = []
    for n in range(B):
        (e,), rec = cache.request([n * L], [U[n]], eps_fn)
        init.append(rec)
        G[n] = _step(U[n], e, ac[n], bc[n], store_dtype)
        U[n + 1] = G[n]
    trace.append({"kind": "init", "coarse": init})
    iters = 0
    limit = B if max_iters is None else min(B, max_iters)
    for k in range(limit):
        # fine solves of the blocks that are not final, one batched step at a time
        active = list(range(k, B))
        Xf = {n: U[n].copy() for n in active}
        fine = []
        for j in range(L):
            ts = [n * L + j for n in active]
            outs, rec = cache.request(ts, [Xf[n] for n in active], eps_fn)
            fine.append(rec)
            for n, e in zip(active, outs):
                t = n * L + j
                Xf[n] = _step(Xf[n], e, alpha[t], b[t], store_dtype)
        Uold = U.copy()
        U[k + 1] = Xf[k]                       # exact: the fine solve of a final state
        coarse = []
        for n in range(k + 1, B):
            (e,), rec = cache.request([n * L], [U[n]], eps_fn)
            coarse.append(rec)
            g = _step(U[n], e, ac[n], bc[n], store_dtype)
            U[n + 1] = (g.astype(F64) + (Xf[n].astype(F64) - G[n].astype(F64))).astype(store_dtype)
            G[n] = g
        r = np.array([float(np.mean((U[n].astype(F64) - Uold[n].astype(F64)) ** 2))
                      for n in range(k + 1, B + 1)])
        iters += 1
        done = bool(np.all(r <= tau)) or k + 1 == B
        trace.append({"kind": "iter", "k": k, "fine": fine, "coarse": coarse, "r": r,
                      "done": done})
        if done:
            break
    stats = {"nfe": cache.nfe, "hits": cache.hits, "iters": iters, "U": U.copy()}
    return U[B].copy(), trace, stats


def uncached(x_init, T: int, B: int, tau: float, ab, alpha, b, eps_fn,
             store_dtype=np.float32):
    """The same Parareal iteration with every request evaluated (no cache code)."""
    L = T // B
    ac, bc = coarse_coefficients(ab, B)
    x0 = np.asarray(x_init, store_dtype).reshape(-1)
    U = np.zeros((B + 1, x0.size), store_dtype)
    G = np.zeros((B, x0.size), store_dtype)
    U[0] = x0
    nfe = 0

    def ev(xs, ts):
        nonlocal nfe
        nfe += len(ts)
        return eps_fn(np.stack(xs), list(ts))

    for n in range(B):
        e = ev([U[n]], [n * L])[0]
        G[n] = _step(U[n], e, ac[n], bc[n], store_dtype)
        U[n + 1] = G[n]
    iters = 0
    for k in range(B):
        Xf = [U[n].copy() for n in range(B)]
        for j in range(L):
            act = list(range(k, B))
            E = ev([Xf[n] for n in act], [n * L + j for n in act])
            for n, e in zip(act, E):
                Xf[n] = _step(Xf[n], e, alpha[n * L + j], b[n * L + j], store_dtype)
        Uold = U.copy()
        U[k + 1] = Xf[k]
        for n in range(k + 1, B):
            e = ev([U[n]], [n * L])[0]
            g = _step(U[n], e, ac[n], bc[n], store_dtype)
            U[n + 1] = (g.astype(F64) + (Xf[n].astype(F64) - G[n].astype(F64))).astype(store_dtype)
            G[n] = g
        iters += 1
        r = [float(np.mean((U[n].astype(F64) - Uold[n].astype(F64)) ** 2)) for n in range(k + 1, B + 1)]
        if all(v <= tau for v in r) or k + 1 == B:
            break
    return U[B].copy(), nfe, iters
