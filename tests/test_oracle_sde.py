"""Pins of the oracle's SDE step, schedule and log-probability (CPU only).

Each pin rests on something other than the oracle itself: hand-derived worked
examples of Eq. 1, the ODE special case, the closed-form log-density at the
mean, scipy's normal log-pdf, the chi-square law of the sampled noise, and the
exact marginals of a Gaussian data distribution under the exact velocity.
"""
import json
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle import sde

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


@pytest.mark.parametrize("key", ["sde_eq1_sigma1", "sde_eq1_sigma05"])
def test_eq1_hand_examples(key):
    g = GOLD[key]
    x, v, eps = np.array([g["x"]]), np.array([g["v"]]), np.array([g["eps"]])
    dt = g["t_next"] - g["t"]
    mean = sde.sde_mean(x, v, g["t"], dt, g["sigma"])
    assert mean[0] == pytest.approx(g["mean"], abs=1e-15)
    xn = sde.sde_step(x, v, eps, g["t"], g["t_next"], g["sigma"])
    assert xn[0] == pytest.approx(g["x_next"], abs=1e-15)
    lp = sde.step_log_prob(x[None], v[None], xn[None], g["t"], g["t_next"], g["sigma"])
    assert lp[0] == pytest.approx(g["logp"], abs=1e-14)


def test_ode_special_case_hand_example():
    g = GOLD["ode_step"]
    xn = sde.sde_step(np.array(g["x"]), np.array(g["v"]), np.zeros(2), g["t"], g["t_next"], 0.0)
    np.testing.assert_array_equal(xn, g["x_next"])


def test_sigma_zero_reduces_to_euler():
    """P1: sigma = 0 turns Eq. 1 into the deterministic Euler ODE step."""
    rng = np.random.default_rng(0)
    x, v, eps = rng.standard_normal((3, 4, 50))
    for t, tn in [(1.0, 0.9), (0.55, 0.3), (0.1, 0.0)]:
        np.testing.assert_array_equal(sde.sde_step(x, v, eps, t, tn, 0.0), x + v * (tn - t))
    # the SDE drift tends to the ODE drift as sigma -> 0
    a = sde.sde_step(x, v, 0 * eps, 0.5, 0.4, 1e-6)
    np.testing.assert_allclose(a, x + v * (-0.1), atol=1e-12)


def test_flow_sde_schedule_hand_values():
    g = GOLD["flow_sde_sigmas_K4_eta07"]
    ts = sde.time_grid(g["K"])
    np.testing.assert_allclose(ts, [1.0, 0.75, 0.5, 0.25, 0.0], atol=0)
    np.testing.assert_allclose(sde.schedule_sigmas(ts, g["eta"]), g["sigmas"], rtol=1e-15)


def test_dance_and_mixed_schedule():
    ts = sde.time_grid(10)
    np.testing.assert_array_equal(sde.schedule_sigmas(ts, 0.3, "dance"), np.full(10, 0.3))
    s = sde.schedule_sigmas(ts, 0.7, "flow", sde_steps={1, 2, 3})
    assert [k for k in range(10) if s[k] > 0] == [1, 2, 3]
    assert np.all(sde.schedule_sigmas(ts, 0.7, "ode") == 0)


def test_logprob_at_mean_closed_form():
    """P2: at x_next = mean the summed log-density is -D/2 log(2 pi sigma^2 |dt|)."""
    rng = np.random.default_rng(1)
    B, D = 3, 777
    mean = rng.standard_normal((B, D))
    for sigma, dt in [(1.4, -0.25), (0.05, -0.1), (2.0, -1e-3)]:
        lp = sde.log_prob(mean, mean, sigma, dt)
        np.testing.assert_allclose(lp, -0.5 * D * math.log(2 * math.pi * sigma ** 2 * abs(dt)), rtol=1e-14)


def test_logprob_one_element_matches_scipy():
    """P3: with one element it is the textbook normal log-pdf."""
    rng = np.random.default_rng(2)
    for _ in range(20):
        x, v, eps = rng.standard_normal(3)
        t = rng.uniform(0.05, 1.0)
        tn = t - rng.uniform(0.01, t)
        sigma = rng.uniform(0.1, 2.0)
        xn = sde.sde_step(np.array([x]), np.array([v]), np.array([eps]), t, tn, sigma)
        mean = sde.sde_mean(np.array([x]), np.array([v]), t, tn - t, sigma)[0]
        ref = stats.norm.logpdf(xn[0], loc=mean, scale=sigma * math.sqrt(t - tn))
        got = sde.step_log_prob(np.array([[x]]), np.array([[v]]), xn[None], t, tn, sigma)[0]
        assert got == pytest.approx(ref, abs=1e-12)


def test_logprob_sums_independent_coordinates():
    """The noise of Eq. 1 is isotropic, so the density of a sample factorises over its elements:
    the log-density of [a | b] is that of a plus that of b, for every split (scipy per element
    for the one-element parts), and a sample with no elements has log-density 0."""
    rng = np.random.default_rng(4)
    B, D = 3, 50
    mean = rng.standard_normal((B, D))
    xn = mean + 0.3 * rng.standard_normal((B, D))
    sigma, dt = 0.8, -0.15
    whole = sde.log_prob(xn, mean, sigma, dt)
    for cut in (1, 17, 49):
        parts = sde.log_prob(xn[:, :cut], mean[:, :cut], sigma, dt) + sde.log_prob(xn[:, cut:], mean[:, cut:], sigma, dt)
        np.testing.assert_allclose(whole, parts, rtol=1e-13)
    per_elem = stats.norm.logpdf(xn, loc=mean, scale=sigma * math.sqrt(-dt)).sum(axis=1)
    np.testing.assert_allclose(whole, per_elem, rtol=1e-12)
    assert np.all(sde.log_prob(np.zeros((B, 0)), np.zeros((B, 0)), sigma, dt) == 0.0)


def test_logprob_undefined_for_ode_step():
    with pytest.raises(ValueError):
        sde.log_prob(np.zeros((1, 2)), np.zeros((1, 2)), 0.0, -0.1)


def test_noise_scale_matches_density_scale():
    """P5: samples of Eq. 1 give chi-square(D) quadratic forms under the density's own scale."""
    rng = np.random.default_rng(3)
    B, D = 400, 64
    x, v = rng.standard_normal((2, B, D))
    t, tn, sigma = 0.7, 0.6, 0.9
    xn = sde.sde_step(x, v, rng.standard_normal((B, D)), t, tn, sigma)
    lp = sde.step_log_prob(x, v, xn, t, tn, sigma)
    var = sigma ** 2 * (t - tn)
    quad = -(lp + 0.5 * D * math.log(2 * math.pi * var)) * 2.0   # = chi2_D samples
    # mean D, variance 2D: the sample mean of 400 lies within 5 standard errors
    assert abs(quad.mean() - D) < 5 * math.sqrt(2 * D / B)
    assert stats.kstest(quad, stats.chi2(D).cdf).pvalue > 1e-3


def _exact_velocity(m, s):
    """E[noise - data | x_t = x] for data ~ N(m, s^2), noise ~ N(0, 1), x_t = (1-t) data + t noise."""
    def v(x, t):
        var = (1 - t) ** 2 * s * s + t * t
        cov = t - (1 - t) * s * s
        return -m + cov / var * (x - (1 - t) * m)
    return v


def _integrate(m, s, eta, K, n, seed, step=sde.sde_step):
    rng = np.random.default_rng(seed)
    ts = sde.time_grid(K)
    sig = sde.schedule_sigmas(ts, eta)
    v = _exact_velocity(m, s)
    x = rng.standard_normal(n)
    for k in range(K):
        x = step(x, v(x, ts[k]), rng.standard_normal(n), ts[k], ts[k + 1], sig[k])
    return x


@pytest.mark.parametrize("eta", [0.0, 0.3, 0.7])
def test_sde_preserves_gaussian_marginals(eta):
    """P4: with the exact velocity of N(m, s^2) data, Eq. 1 maps N(0,1) at t=1 to N(m, s^2) at t=0.

    This fixes the sign of dt in the drift, the sqrt(|dt|) noise scale and the
    sigma clip at t = 1 (a flipped drift sign gives a std far from s).
    """
    m, s = 2.0, 0.5
    x = _integrate(m, s, eta, K=300, n=40000, seed=4)
    assert abs(x.mean() - m) < 0.02
    assert abs(x.std() - s) < 0.02


def test_planted_drift_sign_error_is_caught():
    """A plausible mistake planted in the oracle (drift sign of the sigma term) fails P4."""
    def wrong_step(x, v, eps, t, tn, sigma):
        dt = tn - t
        mean = x + (v - sigma ** 2 / (2 * t) * (x + (1 - t) * v)) * dt
        return mean + sigma * math.sqrt(abs(dt)) * eps
    x = _integrate(2.0, 0.5, 0.7, K=300, n=20000, seed=5, step=wrong_step)
    assert abs(x.std() - 0.5) > 0.1


def test_planted_logprob_scale_error_is_caught():
    """Using sigma^2 instead of sigma^2 |dt| as the variance breaks P2."""
    D, sigma, dt = 10, 0.8, -0.2
    mean = np.zeros((1, D))
    wrong = -0.5 * D * math.log(2 * math.pi * sigma ** 2)
    assert abs(sde.log_prob(mean, mean, sigma, dt)[0] - wrong) > 1.0
