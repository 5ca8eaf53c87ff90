"""SDE dynamics of Flow-GRPO (Sec. 3.1, Eq. 1 and Table 1), float64.

Conventions (readings where the paper is silent):
  * Time runs from t = 1 (pure noise) to t = 0 (data) on the uniform grid
    t_k = 1 - k/K, so the step dt = t_{k+1} - t_k is negative.
  * Eq. 1 writes the noise term as sigma_t * sqrt(dt) * eps; with dt < 0 the
    noise is scaled by sqrt(|dt|).
  * sigma_t and the drift are evaluated at the left point t_k (Euler-Maruyama).
  * Flow-SDE's sigma_t = eta * sqrt(t / (1 - t)) is infinite at t = 1; at
    t_k = 1 the denominator 1 - t uses the next grid point t_1 instead.
  * The transition log-probability is the Gaussian density of the stored
    x_{t+dt} under N(mean, (sigma_t^2 |dt|) I), summed over all elements of a
    sample.  sigma_t = 0 (an ODE step) has no density.
"""
from __future__ import annotations

import math

import numpy as np


def time_grid(K: int) -> np.ndarray:
    """Uniform grid t_k = 1 - k/K, k = 0..K (Flow-GRPO samples on a uniform grid from 1 to 0)."""
    return np.array([1.0 - k / K for k in range(K + 1)], dtype=np.float64)


def sigma_flow_sde(t: float, eta: float, t_clip: float) -> float:
    """Flow-SDE noise level eta * sqrt(t / (1 - t)) (Table 1, row Flow-SDE).

    ``t_clip`` replaces t inside (1 - t) when t == 1, where the schedule is
    singular (the next grid point is used).
    """
    denom_t = t_clip if t >= 1.0 else t
    return eta * math.sqrt(t / (1.0 - denom_t))


def sigma_dance_sde(t: float, eta: float) -> float:
    """Dance-SDE noise level: the constant eta (Table 1, row Dance-SDE)."""
    return float(eta)


def schedule_sigmas(ts: np.ndarray, eta: float, kind: str = "flow", sde_steps=None) -> np.ndarray:
    """sigma_k for each step k = 0..K-1; steps outside ``sde_steps`` are ODE steps (sigma = 0).

    MixGRPO / Flow-GRPO-Fast (Sec. 3.1) applies the SDE only on selected steps
    and the deterministic ODE elsewhere.
    """
    K = len(ts) - 1
    out = np.zeros(K, dtype=np.float64)
    for k in range(K):
        if sde_steps is not None and k not in sde_steps:
            continue
        if kind == "flow":
            out[k] = sigma_flow_sde(float(ts[k]), eta, float(ts[1]))
        elif kind == "dance":
            out[k] = sigma_dance_sde(float(ts[k]), eta)
        elif kind == "ode":
            out[k] = 0.0
        else:
            raise ValueError(kind)
    return out


def sde_mean(x: np.ndarray, v: np.ndarray, t: float, dt: float, sigma: float) -> np.ndarray:
    """Deterministic part of Eq. 1: x_t + [v + sigma^2/(2t) (x_t + (1-t) v)] dt."""
    x = np.asarray(x, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if sigma == 0.0:
        # The ODE update x_t + v dt (Sec. 3.1; Table 1 row ODE).
        return x + v * dt
    drift = v + (sigma * sigma) / (2.0 * t) * (x + (1.0 - t) * v)
    return x + drift * dt


def sde_step(x, v, eps, t: float, t_next: float, sigma: float) -> np.ndarray:
    """One Euler-Maruyama step of Eq. 1 from t to t_next (< t), noise eps ~ N(0, I)."""
    dt = t_next - t
    mean = sde_mean(x, v, t, dt, sigma)
    if sigma == 0.0:
        return mean
    return mean + sigma * math.sqrt(abs(dt)) * np.asarray(eps, dtype=np.float64)


def log_prob(x_next, mean, sigma: float, dt: float) -> np.ndarray:
    """Sum over the elements of each sample (leading axis) of log N(x_next; mean, sigma^2 |dt|).

    Returns one float64 value per sample.  Undefined for sigma = 0.
    """
    if sigma == 0.0 or dt == 0.0:
        raise ValueError("transition density undefined for sigma * sqrt(|dt|) = 0")
    x_next = np.asarray(x_next, dtype=np.float64)
    mean = np.asarray(mean, dtype=np.float64)
    B = x_next.shape[0]
    var = sigma * sigma * abs(dt)
    r = (x_next - mean).reshape(B, -1)
    D = r.shape[1]
    quad = np.sum(r * r, axis=1) / (2.0 * var)
    return -quad - 0.5 * D * math.log(2.0 * math.pi * var)


def step_log_prob(x, v, x_next, t: float, t_next: float, sigma: float) -> np.ndarray:
    """Log-probability of the stored x_next given (x, v) at step t -> t_next."""
    dt = t_next - t
    return log_prob(x_next, sde_mean(x, v, t, dt, sigma), sigma, dt)
