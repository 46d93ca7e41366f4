"""Pins for the oracle's extensions beyond the deterministic single-sample sampler. CPU only.

Stochastic step (ancestral DDPM with pre-drawn step noise, the window study's sampler,
Sec. 3.4; the generalized DDIM step with eta = 1, the paper printing no step):
  * eta = 0 gives the DDIM coefficients; the last step (alpha_bar = 1) carries no noise;
  * window = 1 reproduces serial DDPM in its textbook (posterior mean + variance) form,
    which is written without the generalized-DDIM coefficients;
  * delta = 0 reproduces uncached Picard with the same noise exactly;
  * the Picard fixed point (tau = 0) is the serial drift-form recurrence;
  * zero noise with eta = 0 is the deterministic sampler bit for bit.
Revisit statistic (Sec. 1):
  * every timestep is a first entry exactly once: revisits = requests - T;
  * threshold 0 counts nothing (deviations are >= 0, the test is strict), +inf counts
    every revisit;
  * the scalar simulator of the linear network (a separate formulation) gives the same
    counts on a grid of T, P, delta.
"""
import numpy as np
import pytest

from oracle import eps_models as em
from oracle import sampler as sp
from oracle import scalar_sim
from oracle import schedule as sch
from paper_2609_36522_amd import inputs


def _ddpm(T, eta=1.0):
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b, sigma = sch.step_coefficients(ab, eta)
    return ab, t, alpha, b, sigma


def _tiny_mlp(T, shape=(4, 8, 8), hid=32):
    _, t = sch.sampler_alpha_bar(T)
    return em.PatchMLP(inputs.mlp_weights(hid), t, shape)


# ------------------------------------------------------------------ stochastic step
def test_eta0_is_ddim_and_last_step_is_noise_free():
    for T in (1, 10, 100, 1000):
        ab, _ = sch.sampler_alpha_bar(T)
        a0, b0 = sch.ddim_coefficients(ab)
        a, b, s = sch.step_coefficients(ab, 0.0)
        assert np.array_equal(a, a0) and np.array_equal(b, b0) and not s.any()
        _, _, s1 = sch.step_coefficients(ab, 1.0)
        assert s1[-1] == 0.0 and np.all(s1[:-1] > 0.0)


@pytest.mark.parametrize("eta", [0.0, 0.5, 1.0])
def test_noiseless_steps_of_degenerate_schedules(eta):
    """sigma_i = eta x two factors is 0 at eta = 0 and wherever ab_{i+1} = ab_i (the second
    factor is 0; the first is at most 1, and 0/0 where both are 1): alpha_bar = 1 at every
    state gives the identity step, alpha = b = sigma = 0, with no NaN; a repeated value
    below 1 gives sigma = 0 at that step only."""
    a, b, sig = sch.step_coefficients(np.ones(7), eta)
    assert np.all(a == 0.0) and np.all(b == 0.0) and np.all(sig == 0.0)
    ab = np.array([0.2, 0.2, 0.5, 0.5, 1.0])
    a, b, sig = sch.step_coefficients(ab, eta)
    assert np.all(np.isfinite(a)) and np.all(np.isfinite(b)) and np.all(np.isfinite(sig))
    assert sig[0] == 0.0 and sig[2] == 0.0 and a[0] == 0.0 and a[2] == 0.0
    assert (sig[1] > 0.0) == (eta > 0.0)
    # eta = 0 is DDIM for any schedule, a decreasing one included (sigma is never formed)
    dec = np.array([0.9, 0.6, 0.7, 0.3])
    a0, b0, s0 = sch.step_coefficients(dec, 0.0)
    ad, bd = sch.ddim_coefficients(dec)
    assert np.array_equal(a0, ad) and np.array_equal(b0, bd) and np.all(s0 == 0.0)


@pytest.mark.parametrize("T", [10, 50])
@pytest.mark.parametrize("model", ["linear", "mlp"])
def test_ddpm_window1_is_textbook_ddpm(T, model):
    ab, t, alpha, b, sigma = _ddpm(T)
    shape = (4, 8, 8)
    x = inputs.x_init(shape).reshape(-1)
    Z = inputs.step_noise(1, T, x.size)[0]
    noise = sp.step_noise_terms(sigma, Z)
    eps = em.linear_eps(inputs.linear_coefficients(T)) if model == "linear" else _tiny_mlp(T)
    x64, _, st = sp.sample(x, T, 1, 0.05, 1e-3, alpha, b, eps, store_dtype=np.float64, noise=noise)
    ref = sp.ddpm_serial_textbook(x, ab, eps, Z, store_dtype=np.float64)
    assert st.sweeps == T and st.nfe == T
    assert np.max(np.abs(x64 - ref)) <= 1e-11 * np.max(np.abs(ref))


def test_ddpm_textbook_differs_from_ddim():
    """The noise term is live: the same run with eta = 0 lands elsewhere."""
    T = 10
    ab, t, alpha, b, sigma = _ddpm(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    Z = inputs.step_noise(1, T, x.size)[0]
    eps = em.linear_eps(inputs.linear_coefficients(T))
    ref = sp.ddpm_serial_textbook(x, ab, eps, Z, store_dtype=np.float64)
    ddim = sp.ddim_serial_textbook(x, ab, eps, store_dtype=np.float64)
    assert np.sqrt(np.mean((ref - ddim) ** 2)) > 1e-2


@pytest.mark.parametrize("model", ["linear", "mlp"])
def test_ddpm_delta0_equals_uncached(model):
    T, P, tau = 12, 4, 1e-3
    ab, t, alpha, b, sigma = _ddpm(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    noise = sp.step_noise_terms(sigma, inputs.step_noise(1, T, x.size)[0])
    eps = em.linear_eps(inputs.linear_coefficients(T)) if model == "linear" else _tiny_mlp(T)
    xc, trc, st = sp.sample(x, T, P, 0.0, tau, alpha, b, eps, noise=noise)
    xu, tru, nfe_u = sp.picard_uncached(x, T, P, tau, alpha, b, eps, noise=noise)
    assert np.array_equal(xc, xu)
    assert [(r["s"], r["c"]) for r in trc] == [(r["s"], r["c"]) for r in tru]
    assert st.nfe == nfe_u


def test_ddpm_fixed_point_tau0_is_serial():
    T, P = 10, 4
    ab, t, alpha, b, sigma = _ddpm(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    noise = sp.step_noise_terms(sigma, inputs.step_noise(1, T, x.size)[0])
    eps = em.linear_eps(inputs.linear_coefficients(T))
    xp, _, _ = sp.sample(x, T, P, 0.0, 0.0, alpha, b, eps, store_dtype=np.float64, noise=noise)
    ref = sp.ddim_serial_drift(x, alpha, b, eps, store_dtype=np.float64, noise=noise)
    assert np.max(np.abs(xp - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_zero_noise_eta0_is_the_deterministic_sampler():
    T, P = 10, 4
    ab, t, alpha, b, sigma = _ddpm(T, eta=0.0)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    noise = sp.step_noise_terms(sigma, inputs.step_noise(1, T, x.size)[0])
    a, tra, _ = sp.sample(x, T, P, 0.05, 1e-3, alpha, b, eps, noise=noise)
    d, trd, _ = sp.sample(x, T, P, 0.05, 1e-3, alpha, b, eps)
    assert np.array_equal(a, d)


# ------------------------------------------------------------------ revisit statistic
@pytest.mark.parametrize("T,P", [(10, 4), (12, 12), (30, 8), (7, 1)])
def test_revisit_identities(T, P):
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    eps = em.linear_eps(inputs.linear_coefficients(T))
    _, tr, st = sp.sample(x, T, P, 0.0, 1e-3, alpha, b, eps)
    req, rev, below = sp.revisit_counts(tr, 0.05)
    assert req == st.nfe + st.hits
    assert rev == req - T                       # one first entry per timestep
    assert sp.revisit_counts(tr, 0.0)[2] == 0
    assert sp.revisit_counts(tr, np.inf)[2] == rev
    assert 0 <= below <= rev


def _scalar_counts(records, thr):
    req = rev = below = 0
    for r in records:
        for d in r["dev"]:
            req += 1
            if not np.isnan(d):
                rev += 1
                below += d < thr
    return req, rev, below


@pytest.mark.parametrize("T,P,delta", [(T, P, d) for T in (5, 9, 12) for P in (1, 3, T)
                                       for d in (0.0, 0.05)])
def test_revisit_counts_match_scalar_simulator(T, P, delta):
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    c = inputs.linear_coefficients(T)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    _, tr, _ = sp.sample(x, T, P, delta, 1e-3, alpha, b, em.linear_eps(c), store_dtype=np.float64)
    sim = scalar_sim.simulate(x, T, P, delta, 1e-3, alpha, b, c.astype(np.float64))
    for thr in (0.0, 0.01, 0.05, 0.5, np.inf):
        a = sp.revisit_counts(tr, thr)
        s = _scalar_counts(sim["records"], thr)
        assert a == s, (thr, a, s)


def test_cached_hits_are_revisits_below_delta():
    """In a cached run the hit count is the revisit count below delta itself."""
    T, P, delta = 30, 8, 0.05
    ab, t = sch.sampler_alpha_bar(T)
    alpha, b = sch.ddim_coefficients(ab)
    x = inputs.x_init((4, 8, 8)).reshape(-1)
    _, tr, st = sp.sample(x, T, P, delta, 1e-3, alpha, b, _tiny_mlp(T))
    assert sp.revisit_counts(tr, delta)[2] == st.hits


# ------------------------------------------------------------------ batch inputs
def test_batch_latents_are_distinct_seeds():
    xb = inputs.x_init_batch((4, 8, 8), 3)
    assert xb.shape == (3, 4, 8, 8)
    for n in range(3):
        assert np.array_equal(xb[n], inputs.x_init((4, 8, 8), inputs.SEED_BATCH_BASE + n))
    assert not np.array_equal(xb[0], xb[1])


def test_revisit_threshold_is_strict():
    """'Below the threshold' is strict; first entries (NaN) are no revisits."""
    nan = float("nan")
    trace = [{"dev": [nan, nan]}, {"dev": [0.05, 0.04, nan]}, {"dev": [0.0, 0.0500001]}]
    assert sp.revisit_counts(trace, 0.05) == (7, 4, 2)
    assert sp.revisit_counts(trace, 0.0) == (7, 4, 0)
