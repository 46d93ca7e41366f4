"""Noise schedule and DDIM coefficients (oracle; test infrastructure only).

The paper samples Stable Diffusion v1.5 with DDIM (Sec. 3.3) and writes the drift
s_theta of Eq. (1) as a combination of the current latent and the noise prediction
with schedule-determined coefficients (Sec. 2.1). It does not print the schedule;
the reading used here:

* training betas "scaled linear": beta_j = (sqrt(b0) + j (sqrt(b1) - sqrt(b0)) / (N-1))^2,
  j = 0..N-1, with b0 = 0.00085, b1 = 0.012, N = 1000; alpha_bar_j = prod_{i<=j} (1 - beta_i);
* sampling timesteps, "trailing" spacing: t_j = round(N - j N / T) - 1, j = 0..T-1;
* sampler state i = 0..T, state 0 the noisiest; alpha_bar of state i is alpha_bar_{t_i}
  for i < T and 1 for the final state i = T;
* deterministic DDIM (eta = 0) from state i to i+1 is x_{i+1} = a_i x_i + b_i eps_i with
  a_i = sqrt(ab_{i+1} / ab_i), b_i = sqrt(1 - ab_{i+1}) - a_i sqrt(1 - ab_i); the
  per-step drift is d_i = x_{i+1} - x_i = alpha_i x_i + b_i eps_i with alpha_i = a_i - 1
  (the 1/T factor of Eq. (1) is absorbed into the one-step increment);
* the stochastic sampler of the window study (DDPM, Sec. 3.4) is the generalized DDIM step
  with eta = 1: x_{i+1} = sqrt(ab_{i+1}) x0^ + sqrt(1 - ab_{i+1} - sigma_i^2) eps + sigma_i z_i,
  sigma_i = eta sqrt((1 - ab_{i+1}) / (1 - ab_i)) sqrt(1 - ab_i / ab_{i+1}), with the noise
  z_i drawn before sampling so that the Picard iteration solves a fixed recurrence.

Everything is float64.
"""
from __future__ import annotations

import numpy as np


def scaled_linear_alpha_bar(beta_start: float = 0.00085, beta_end: float = 0.012,
                            train_steps: int = 1000) -> np.ndarray:
    """alpha_bar_j = prod_{i<=j} (1 - beta_i) for the scaled-linear betas, j = 0..N-1."""
    j = np.arange(train_steps, dtype=np.float64)
    root = np.sqrt(beta_start) + j * (np.sqrt(beta_end) - np.sqrt(beta_start)) / (train_steps - 1)
    betas = root * root
    return np.cumprod(1.0 - betas)


def trailing_timesteps(T: int, train_steps: int = 1000) -> np.ndarray:
    """Sampling timesteps t_j = round(N - j N / T) - 1 for j = 0..T-1 (descending)."""
    if not (1 <= T <= train_steps):
        raise ValueError("need 1 <= T <= train_steps")
    j = np.arange(T, dtype=np.float64)
    return (np.round(train_steps - j * train_steps / T) - 1).astype(np.int64)


def sampler_alpha_bar(T: int, beta_start: float = 0.00085, beta_end: float = 0.012,
                      train_steps: int = 1000):
    """(ab, t): ab[i] for sampler states i = 0..T (ab[T] = 1) and timesteps t[0..T-1]."""
    abar = scaled_linear_alpha_bar(beta_start, beta_end, train_steps)
    t = trailing_timesteps(T, train_steps)
    ab = np.empty(T + 1, dtype=np.float64)
    ab[:T] = abar[t]
    ab[T] = 1.0
    return ab, t


def ddim_coefficients(ab: np.ndarray):
    """(alpha, b) with d_i = alpha_i x_i + b_i eps_i the DDIM one-step increment."""
    ab = np.asarray(ab, dtype=np.float64)
    a = np.sqrt(ab[1:] / ab[:-1])
    alpha = a - 1.0
    b = np.sqrt(1.0 - ab[1:]) - a * np.sqrt(1.0 - ab[:-1])
    return alpha, b


def step_coefficients(ab: np.ndarray, eta: float):
    """(alpha, b, sigma) of the generalized DDIM step with parameter eta, as the one-step
    increment d_i = alpha_i x_i + b_i eps_i + sigma_i z_i (eta = 0 gives ddim_coefficients)."""
    ab = np.asarray(ab, dtype=np.float64)
    ab0, ab1 = ab[:-1], ab[1:]
    # sigma_i is eta times the two factors: 0 at eta = 0 by definition, and 0 where
    # ab_{i+1} = ab_i (the second factor is 0, the first at most 1), also where both are 1
    # and the first factor is 0/0.
    noiseless = (ab1 == ab0) | (eta == 0.0)
    with np.errstate(invalid="ignore", divide="ignore"):
        full = eta * np.sqrt((1.0 - ab1) / (1.0 - ab0)) * np.sqrt(1.0 - ab0 / ab1)
    sigma = np.where(noiseless, 0.0, full)
    a = np.sqrt(ab1 / ab0)
    alpha = a - 1.0
    x0_coef_eps = np.sqrt(1.0 - ab1 - sigma * sigma)
    b = x0_coef_eps - a * np.sqrt(1.0 - ab0)
    return alpha, b, sigma
