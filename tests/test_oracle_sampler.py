"""Pins for the oracle's cached Picard sampler. CPU only.

1. delta = 0 reproduces uncached Picard exactly (strict '<' in Eq. (5)).
2. window = 1 reproduces serial DDIM (textbook form).
3. The Picard fixed point matches serial DDIM: exactly at tau = 0 (fp64 storage), within
   tau in Eq. (2) units at tau = 1e-3.
4. The linear network reduces to a scalar recurrence and a closed-form serial product.
Plus: true-noise exactness under any cache tolerance, delta = +inf counts, per-sweep
invariants (first-entry misses, miss-only cache writes, the cache invariant of Sec. 2.2).
"""
import itertools

import numpy as np
import pytest

from oracle import eps_models as em
from oracle import sampler as sp
from oracle import scalar_sim
from oracle import schedule as sch
from paper_2609_36522_amd import inputs


def _coef(T):
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    return ab, t, alpha, b


def _tiny_mlp(T, shape=(4, 8, 8), hid=32):
    _, t, _, _ = _coef(T)
    return em.PatchMLP(inputs.mlp_weights(hid), t, shape)


# ------------------------------------------------------------------ 1. delta = 0
@pytest.mark.parametrize("model", ["linear", "mlp"])
def test_delta0_equals_uncached(model):
    T, P, tau = 12, 4, 1e-3
    ab, t, alpha, b = _coef(T)
    shape = (4, 8, 8)
    x = inputs.x_init(shape).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T)) if model == "linear" else _tiny_mlp(T)
    xc, trc, st = sp.sample(x, T, P, 0.0, tau, alpha, b, eps)
    xu, tru, nfe_u = sp.picard_uncached(x, T, P, tau, alpha, b, eps)
    assert np.array_equal(xc, xu)
    assert [(r["s"], r["e"], r["c"]) for r in trc] == [(r["s"], r["e"], r["c"]) for r in tru]
    for a, u in zip(trc, tru):
        assert np.array_equal(a["r"], u["r"])
    assert st.hits == 0 and st.nfe == nfe_u


# ------------------------------------------------------------------ 2. window = 1
@pytest.mark.parametrize("delta", [0.0, 0.05, np.inf])
def test_window1_is_serial_ddim(delta):
    T = 10
    ab, t, alpha, b = _coef(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    x64, tr, st = sp.sample(x, T, 1, delta, 1e-3, alpha, b, eps, store_dtype=np.float64)
    ref64 = sp.ddim_serial_textbook(x, ab, eps, store_dtype=np.float64)
    assert st.sweeps == T and st.nfe == T and st.hits == 0
    assert np.max(np.abs(x64 - ref64)) <= 1e-12 * np.max(np.abs(ref64))
    x32, _, _ = sp.sample(x, T, 1, delta, 1e-3, alpha, b, eps)
    ref32 = sp.ddim_serial_textbook(x, ab, eps)
    rms = np.sqrt(np.mean(ref64 ** 2))
    assert np.max(np.abs(x32.astype(np.float64) - ref32)) <= 1e-6 * rms


def test_window1_mlp_is_serial_ddim():
    T = 6
    ab, t, alpha, b = _coef(T)
    net = _tiny_mlp(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    xs, _, st = sp.sample(x, T, 1, 0.05, 1e-3, alpha, b, net)
    ref = sp.ddim_serial_drift(x, alpha, b, net)
    assert st.nfe == T and np.array_equal(xs, ref)


# ------------------------------------------------------------------ 3. fixed point
def test_fixed_point_tau0_is_serial_exactly():
    T, P = 10, 4
    ab, t, alpha, b = _coef(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    xp, tr, st = sp.sample(x, T, P, 0.0, 0.0, alpha, b, eps, store_dtype=np.float64)
    ref = sp.ddim_serial_drift(x, alpha, b, eps, store_dtype=np.float64)
    assert np.max(np.abs(xp - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("T,P", [(10, 4), (12, 3), (7, 7), (9, 1), (30, 8)])
@pytest.mark.parametrize("delta", [0.0, 0.05])
def test_zero_drift_converges_in_one_sweep_per_window(T, P, delta):
    """Eq. (2) taken literally (r <= tau): with zero drift the trajectory is constant, every
    residual is exactly 0, and at tau = 0 every state of a window counts as converged, so
    each sweep slides the window to its end: ceil(T / P) sweeps, every step evaluated once.
    The uncached reference and the scalar simulator agree."""
    alpha = np.zeros(T)
    b = np.zeros(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    c = inputs.linear_coefficients(T)
    eps = em.linear_eps(c)
    xp, tr, st = sp.sample(x, T, P, delta, 0.0, alpha, b, eps)
    assert np.array_equal(xp, x.astype(np.float32))
    assert st.sweeps == -(-T // P) and st.nfe == T and st.hits == 0
    for rec in tr:
        assert np.all(rec["r"] == 0.0) and rec["s_next"] == rec["e"]
    xu, tru, nfe_u = sp.picard_uncached(x, T, P, 0.0, alpha, b, eps)
    assert len(tru) == st.sweeps and nfe_u == T and np.array_equal(xu, xp)
    sim = scalar_sim.simulate(x, T, P, delta, 0.0, alpha, b, c)
    assert sim["sweeps"] == st.sweeps and sim["nfe"] == T


@pytest.mark.parametrize("model,delta", [("linear", 0.0), ("mlp", 0.0)])
def test_fixed_point_within_tau(model, delta):
    T, P, tau = 10, 4, 1e-3
    ab, t, alpha, b = _coef(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T)) if model == "linear" else _tiny_mlp(T)
    xp, tr, st = sp.sample(x, T, P, delta, tau, alpha, b, eps)
    ref = sp.ddim_serial_drift(x, alpha, b, eps)
    assert np.mean((xp.astype(np.float64) - ref) ** 2) <= tau
    assert st.nfe >= T


# ------------------------------------------------------------------ 4. linear closed form
def test_linear_closed_form_serial_product():
    T = 10
    ab, t, alpha, b = _coef(T)
    c = inputs.linear_coefficients(T).astype(np.float64)
    x = inputs.x_init((4, 8, 8)).reshape(-1).astype(np.float64)
    gain = scalar_sim.serial_gain(alpha, b, c)
    xs, _, _ = sp.sample(x, T, 1, 0.0, 0.0, alpha, b, em.linear_eps(c), store_dtype=np.float64)
    assert np.max(np.abs(xs - gain * x)) <= 1e-12 * np.max(np.abs(gain * x))


def _decisions(records):
    return [(r["s"], r["e"], list(map(bool, r["hit"])), list(r["miss"]), r["c"], r["s_next"])
            for r in records]


def _band_ok(a_rec, b_rec, delta, tau, rel=1e-9):
    """True if two decision traces differ only through a decision taken within rel of its
    threshold (Eq. (5) for hits, Eq. (2) for the converged count).

    Up to the first such flip every window, hit mask, miss list, converged count and slide
    must be equal. In the sweep of the flip, hit masks may differ only in slots whose
    deviation lies within the band of delta on both sides, each miss list must be the one
    its own mask gives, and converged counts may differ only if the residual that ends the
    shorter count lies within the band of tau on both sides. After the flip the two runs
    hold different states, so later sweeps are not comparable and are not compared. A
    difference with no such flip (a miss list, a count or a slide that differs while the
    masks agree) fails."""
    near = lambda v, thr: abs(v - thr) <= rel * max(abs(thr), 1e-300)
    for ra, rb in zip(a_rec, b_rec):
        if (ra["s"], ra["e"]) != (rb["s"], rb["e"]):
            return False
        W = ra["e"] - ra["s"]
        for r in (ra, rb):
            if list(r["miss"]) != [r["s"] + j for j in range(W) if not r["hit"][j]]:
                return False
            if r["s_next"] != r["s"] + 1 + r["c"]:
                return False
        flipped = False
        for j in range(W):
            if bool(ra["hit"][j]) != bool(rb["hit"][j]):
                if not (near(ra["dev"][j], delta) and near(rb["dev"][j], delta)):
                    return False
                flipped = True
        if flipped:
            return True
        if ra["c"] != rb["c"]:
            j = min(ra["c"], rb["c"])
            return j < W - 1 and near(ra["r"][j], tau) and near(rb["r"][j], tau)
    return False


def test_band_ok_rejects_differences_outside_the_band():
    """The pin's fallback accepts an in-band flip and nothing else."""
    base = {"s": 0, "e": 3, "hit": [False, True, False], "dev": [np.nan, 0.01, 0.2],
            "miss": [0, 2], "r": [1e-4, 2e-3, 5e-3], "c": 1, "s_next": 2}
    same = dict(base)
    assert not _band_ok([base], [same], 0.05, 1e-3)                  # no flip: not explained
    miss = dict(base, miss=[0, 1])                                   # same mask, other list
    assert not _band_ok([base], [miss], 0.05, 1e-3)
    count = dict(base, c=0, s_next=1)                                # count differs, r far
    assert not _band_ok([base], [count], 0.05, 1e-3)
    near_tau = dict(base, r=[1e-3, 2e-3, 5e-3])
    assert _band_ok([near_tau], [dict(near_tau, c=0, s_next=1)], 0.05, 1e-3)
    hit_far = dict(base, hit=[False, False, False], miss=[0, 1, 2])  # flip at dev 0.01
    assert not _band_ok([base], [hit_far], 0.05, 1e-3)
    near_d = dict(base, dev=[np.nan, 0.05, 0.2])
    assert _band_ok([near_d], [dict(near_d, hit=[False, False, False], miss=[0, 1, 2])], 0.05, 1e-3)
    first = dict(base, hit=[True, True, False], miss=[2])            # a first entry "hit"
    assert not _band_ok([base], [first], 0.05, 1e-3)
    slide = dict(base, s_next=3)                                     # slide not s + 1 + c
    assert not _band_ok([base], [slide], 0.05, 1e-3)


GRID = [(T, P, d, tau) for T in range(1, 13) for P in range(1, T + 1)
        for d in (0.0, 0.05, np.inf) for tau in (0.0, 1e-3)]


@pytest.mark.parametrize("T,P,delta,tau", GRID[::3] + GRID[1::7])
def test_scalar_simulator_brute_force(T, P, delta, tau):
    ab, t, alpha, b = _coef(T)
    c = inputs.linear_coefficients(T).astype(np.float64)
    x = inputs.x_init((4, 8, 8)).reshape(-1).astype(np.float64)   # D = 256
    xs, tr, st = sp.sample(x, T, P, delta, tau, alpha, b, em.linear_eps(c), store_dtype=np.float64)
    sim = scalar_sim.simulate(x, T, P, delta, tau, alpha, b, c)
    if _decisions(tr) != _decisions(sim["records"]):
        assert _band_ok(tr, sim["records"], delta, tau)
    else:
        assert (st.nfe, st.hits, st.sweeps) == (sim["nfe"], sim["hits"], sim["sweeps"])
        assert np.max(np.abs(xs - sim["gamma_T"] * x)) <= 1e-10 * np.max(np.abs(x))


def test_scalar_simulator_tiny_linear_workload_fp32():
    """The tiny linear workload in fp32 storage follows the scalar recurrence decision by
    decision (its decisions are far from both thresholds)."""
    T, P, delta, tau = 10, 4, 0.05, 1e-3
    ab, t, alpha, b = _coef(T)
    c = inputs.linear_coefficients(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    xs, tr, st = sp.sample(x, T, P, delta, tau, alpha, b, em.linear_eps(c))
    sim = scalar_sim.simulate(x, T, P, delta, tau, alpha, b, c.astype(np.float64))
    assert _decisions(tr) == _decisions(sim["records"])
    assert st.hits > 0                      # the cache is exercised
    rms = np.sqrt(np.mean(x.astype(np.float64) ** 2)) * abs(sim["gamma_T"])
    assert np.max(np.abs(xs - sim["gamma_T"] * x.astype(np.float64))) <= 1e-5 * rms


# ------------------------------------------------------------------ special cases
@pytest.mark.parametrize("delta", [0.0, 0.05, np.inf])
def test_true_noise_is_exact_under_any_cache_tolerance(delta):
    """eps(x) = n for every x: the cached output equals the fresh one, and the drift must be
    taken at the *current* latent (Sec. 2.2) for the sampler to land on x0 exactly."""
    T, P = 20, 6
    ab, t, alpha, b = _coef(T)
    rng = np.random.default_rng(3)
    x0, n = rng.standard_normal(256), rng.standard_normal(256)
    xi = np.sqrt(ab[0]) * x0 + np.sqrt(1 - ab[0]) * n
    const = lambda X, steps: np.repeat(n[None, :], len(steps), axis=0).astype(X.dtype)
    xT, tr, st = sp.sample(xi, T, P, delta, 0.0, alpha, b, const, store_dtype=np.float64)
    assert np.max(np.abs(xT - x0)) < 1e-10
    if delta == np.inf:
        assert st.nfe == T


@pytest.mark.parametrize("T,P", [(10, 4), (12, 5), (7, 7), (30, 8)])
def test_delta_inf_counts(T, P):
    ab, t, alpha, b = _coef(T)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    xs, tr, st = sp.sample(x, T, P, np.inf, 1e-3, alpha, b, eps)
    assert st.nfe == T
    assert st.hits == sum(r["e"] - r["s"] for r in tr) - T


def test_hit_test_is_strict():
    X = np.zeros((3, 8), np.float32)
    Xh = np.full((2, 8), 0.5, np.float32)
    dev, hit = sp.cache_test(X, Xh, np.array([True, True]), 0, 2, 0.5)
    assert np.all(dev == 0.5) and not hit.any()
    dev, hit = sp.cache_test(X, Xh, np.array([True, False]), 0, 2, 0.75)
    assert hit.tolist() == [True, False] and np.isnan(dev[1])


@pytest.mark.parametrize("model,delta", [("linear", 0.05), ("linear", 0.3), ("mlp", 0.05)])
def test_invariants_every_sweep(model, delta):
    T, P, tau = 16, 5, 1e-3
    ab, t, alpha, b = _coef(T)
    eps = em.linear_eps(inputs.linear_coefficients(T)) if model == "linear" else _tiny_mlp(T)
    st = sp.init_state(inputs.x_init((4, 8, 8)), T)
    prev_s = -1
    first = True
    while not st.done:
        seen_before = st.valid.copy()
        Xh0, Eh0 = st.Xh.copy(), st.Eh.copy()
        rec = sp.sweep(st, P, delta, tau, alpha, b, eps)
        s, e = rec["s"], rec["e"]
        new_entries = [t_ for t_ in range(s, e) if not seen_before[t_]]
        assert set(new_entries) <= set(rec["miss"])                      # first entry = miss
        if first:
            assert rec["m"] == min(P, T)
            first = False
        assert rec["miss"] == sorted(rec["miss"])
        hits = [t_ for t_ in range(s, e) if t_ not in rec["miss"]]
        for t_ in hits:                                                  # miss-only update
            assert np.array_equal(st.Xh[t_], Xh0[t_]) and np.array_equal(st.Eh[t_], Eh0[t_])
        for t_ in np.nonzero(st.valid)[0]:                               # cache invariant
            assert np.array_equal(st.Eh[t_], eps(st.Xh[t_][None, :], [int(t_)])[0])
        assert s > prev_s
        prev_s = s
        assert rec["s_next"] >= s + 1
    assert st.sweeps <= T and st.nfe >= T


def test_nfe_falls_as_delta_grows():
    T, P, tau = 30, 8, 1e-3
    ab, t, alpha, b = _coef(T)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    nfe = [sp.sample(x, T, P, d, tau, alpha, b, eps)[2].nfe for d in (0.0, 0.02, 0.05, 0.1, np.inf)]
    assert all(a >= b_ for a, b_ in zip(nfe, nfe[1:]))
    assert nfe[-1] == T and nfe[0] > nfe[-1]
