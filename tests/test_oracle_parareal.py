"""Pins for the oracle's cached Parareal sampler (Sec. 2.1 Parareal-based samplers, Sec. 2.2
cache; the textbook Parareal predictor-corrector, the paper printing no rule). CPU only.

* delta = 0 reproduces the uncached Parareal iteration exactly.
* Parareal exactness: after k iterations the boundaries 0..k equal serial fine DDIM bit for
  bit, and run to B iterations the output is serial fine DDIM bit for bit.
* The initialization is serial DDIM on the coarse grid, checked against the textbook form.
* delta = +inf: every fine-grid timestep is evaluated exactly once (NFE = T).
* Linear network: a scalar formulation of the same cached iteration (written separately)
  makes the same hit/miss decisions and lands on the same output.
"""
import numpy as np
import pytest

from oracle import eps_models as em
from oracle import parareal as pr
from oracle import sampler as sp
from oracle import schedule as sch
from paper_2609_36522_amd import inputs


def _setup(T, model="linear", shape=(4, 8, 8)):
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    if model == "linear":
        eps = em.linear_eps(inputs.linear_coefficients(T))
    else:
        eps = em.PatchMLP(inputs.mlp_weights(32), t, shape)
    x = inputs.x_init(shape).reshape(-1)
    return ab, alpha, b, eps, x


@pytest.mark.parametrize("model", ["linear", "mlp"])
@pytest.mark.parametrize("T,B", [(20, 4), (30, 5)])
def test_delta0_equals_uncached(model, T, B):
    ab, alpha, b, eps, x = _setup(T, model)
    xc, tr, st = pr.sample(x, T, B, 0.0, 1e-3, ab, alpha, b, eps)
    xu, nfe, iters = pr.uncached(x, T, B, 1e-3, ab, alpha, b, eps)
    assert np.array_equal(xc, xu) and st["nfe"] == nfe and st["iters"] == iters and st["hits"] == 0


def _serial_boundaries(x, T, B, alpha, b, eps):
    L = T // B
    ref = [x.astype(np.float32)]
    cur = x.astype(np.float32)
    for n in range(B):
        for j in range(L):
            t = n * L + j
            e = eps(cur[None, :], [t])[0]
            cur = (cur.astype(np.float64) + (alpha[t] * cur.astype(np.float64) + b[t] * e.astype(np.float64))
                   ).astype(np.float32)
        ref.append(cur.copy())
    return ref


@pytest.mark.parametrize("model", ["linear", "mlp"])
def test_full_iterations_give_serial_fine_ddim(model):
    T, B = 20, 4
    ab, alpha, b, eps, x = _setup(T, model)
    serial = sp.ddim_serial_drift(x, alpha, b, eps)
    out, tr, st = pr.sample(x, T, B, 0.0, -1.0, ab, alpha, b, eps)   # never converged early
    assert st["iters"] == B
    assert np.array_equal(out, serial)
    # the iteration ends itself after B iterations (exactness), flagged as done
    assert tr[-1]["done"] and not any(r["done"] for r in tr[1:-1])


@pytest.mark.parametrize("model", ["linear", "mlp"])
def test_exact_prefix_after_k_iterations(model):
    """After k iterations the boundaries 0..k hold the serial fine values bit for bit, and
    boundary k+1 differs (the prefix is exact, not the whole trajectory)."""
    T, B = 20, 5
    ab, alpha, b, eps, x = _setup(T, model)
    ref = _serial_boundaries(x, T, B, alpha, b, eps)
    for k in range(1, B + 1):
        _, _, st = pr.sample(x, T, B, 0.0, -1.0, ab, alpha, b, eps, max_iters=k)
        U = st["U"]
        for n in range(k + 1):
            assert np.array_equal(U[n], ref[n]), (k, n)
        if k + 1 <= B:
            assert not np.array_equal(U[k + 1], ref[k + 1])


@pytest.mark.parametrize("T,B", [(20, 4), (12, 3), (10, 10)])
def test_zero_steps_stop_after_one_iteration(T, B):
    """The Eq. (2) stop taken literally (every r <= tau): with alpha_bar = 1 at every state
    both propagators are the identity, the first iteration changes no boundary (r = 0), and
    at tau = 0 the sampler stops there."""
    ab = np.ones(T + 1)
    alpha = np.zeros(T)
    b = np.zeros(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    xp, trace, st = pr.sample(x, T, B, 0.0, 0.0, ab, alpha, b, eps)
    assert st["iters"] == 1 and trace[-1]["done"] and np.all(trace[-1]["r"] == 0.0)
    assert np.array_equal(xp, x.astype(np.float32))
    # delta = 0, no hits: B coarse requests of the initialization, T fine steps and the B - 1
    # coarse corrections of blocks 1..B-1
    assert st["nfe"] == T + 2 * B - 1 and st["hits"] == 0
    xu, nfe_u, iters_u = pr.uncached(x, T, B, 0.0, ab, alpha, b, eps)
    assert iters_u == 1 and np.array_equal(xu, xp)


def test_initialization_is_coarse_textbook_ddim():
    T, B = 30, 6
    L = T // B
    ab, alpha, b, eps, x = _setup(T)
    out, tr, st = pr.sample(x, T, B, 0.05, 1e-3, ab, alpha, b, eps, store_dtype=np.float64, max_iters=0)
    assert st["iters"] == 0 and st["nfe"] == B
    coarse_eps = lambda X, idx: eps(X, [i * L for i in idx])
    ref = sp.ddim_serial_textbook(x, ab[0::L], coarse_eps, store_dtype=np.float64)
    assert np.max(np.abs(out - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("T,B", [(20, 4), (30, 10), (12, 3)])
def test_delta_inf_evaluates_each_timestep_once(T, B):
    ab, alpha, b, eps, x = _setup(T)
    _, tr, st = pr.sample(x, T, B, np.inf, 1e-3, ab, alpha, b, eps)
    assert st["nfe"] == T


# ------------------------------------------------------------------ scalar formulation
def _scalar_parareal(x0, T, B, delta, tau, ab, alpha, b, c):
    """Linear network eps_t(x) = c_t x: every vector is a multiple of x0, so the cached
    Parareal iteration runs on scalars (float64)."""
    L = T // B
    m1 = float(np.mean(np.abs(x0)))
    m2 = float(np.mean(np.asarray(x0, np.float64) ** 2))
    a0 = np.asarray(ab[0:T:L]); a1 = np.asarray(ab[L:T + 1:L])
    ac = np.sqrt(a1 / a0) - 1.0
    bc = np.sqrt(1.0 - a1) - (1.0 + ac) * np.sqrt(1.0 - a0)
    gh = [None] * T                    # cached input multiple per timestep
    decisions = []
    nfe = 0

    def req(t, g):
        nonlocal nfe
        if gh[t] is not None and abs(g - gh[t]) * m1 < delta:
            decisions.append((t, True))
            return c[t] * gh[t]
        gh[t] = g
        nfe += 1
        decisions.append((t, False))
        return c[t] * g

    U = [1.0] + [0.0] * B
    G = [0.0] * B
    for n in range(B):
        e = req(n * L, U[n])
        G[n] = U[n] + ac[n] * U[n] + bc[n] * e
        U[n + 1] = G[n]
    iters = 0
    for k in range(B):
        F = {n: U[n] for n in range(k, B)}
        for j in range(L):
            es = {n: req(n * L + j, F[n]) for n in range(k, B)}
            for n in range(k, B):
                t = n * L + j
                F[n] = F[n] + alpha[t] * F[n] + b[t] * es[n]
        old = list(U)
        U[k + 1] = F[k]
        for n in range(k + 1, B):
            e = req(n * L, U[n])
            g = U[n] + ac[n] * U[n] + bc[n] * e
            U[n + 1] = g + (F[n] - G[n])
            G[n] = g
        iters += 1
        r = [(U[n] - old[n]) ** 2 * m2 for n in range(k + 1, B + 1)]
        if all(v <= tau for v in r) or k + 1 == B:
            break
    return U[B], decisions, nfe, iters


@pytest.mark.parametrize("T,B,delta", [(20, 4, 0.05), (20, 4, 0.2), (30, 5, 0.02), (12, 3, 0.1),
                                       (20, 10, 0.05), (20, 4, 0.0)])
def test_scalar_formulation_agrees(T, B, delta):
    ab, alpha, b, _, x = _setup(T)
    c = inputs.linear_coefficients(T).astype(np.float64)
    out, tr, st = pr.sample(x, T, B, delta, 1e-3, ab, alpha, b, em.linear_eps(c), store_dtype=np.float64)
    g, dec, nfe, iters = _scalar_parareal(x, T, B, delta, 1e-3, ab, alpha, b, c)
    mine = []
    for rec in tr:
        groups = rec["coarse"] if rec["kind"] == "init" else rec["fine"] + rec["coarse"]
        for r in groups:
            mine += list(zip(r["t"], map(bool, r["hit"])))
    assert mine == dec
    assert st["nfe"] == nfe and st["iters"] == iters
    ref = g * x.astype(np.float64)
    assert np.max(np.abs(out - ref)) <= 1e-11 * np.max(np.abs(ref))


def test_cache_invariant_and_counts():
    T, B = 20, 4
    ab, alpha, b, eps, x = _setup(T, "mlp")
    out, tr, st = pr.sample(x, T, B, 0.05, 1e-3, ab, alpha, b, eps)
    req = sum(len(r["t"]) for rec in tr for r in (rec["coarse"] if rec["kind"] == "init"
                                                   else rec["fine"] + rec["coarse"]))
    assert st["nfe"] + st["hits"] == req and st["nfe"] >= T and st["hits"] > 0
