"""Pins of the oracle's training objectives (CPU only): hand examples, closed forms, invariants."""
import json
import math
import os

import numpy as np
import pytest

from oracle import losses as L

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


def test_flow_noise_endpoints_and_velocity():
    """x_t runs from x0 (t = 0) to eps (t = 1); its t-derivative is the target eps - x0, so the exact
    velocity has zero AWM loss (a flipped target sign would not)."""
    rng = np.random.default_rng(0)
    x0, eps = rng.standard_normal((3, 5, 4)), rng.standard_normal((3, 5, 4))
    np.testing.assert_array_equal(L.flow_noise(x0, eps, np.zeros(3)), x0)
    np.testing.assert_array_equal(L.flow_noise(x0, eps, np.ones(3)), eps)
    t, h = np.array([0.2, 0.5, 0.9]), 1e-6
    dxdt = (L.flow_noise(x0, eps, t + h) - L.flow_noise(x0, eps, t - h)) / (2 * h)
    np.testing.assert_allclose(dxdt, eps - x0, rtol=0, atol=1e-8)
    per, loss = L.awm_loss(dxdt, eps, x0, np.array([1.0, -2.0, 0.5]))
    assert np.all(np.abs(per) < 1e-9) and abs(loss) < 1e-9


def test_awm_hand_example():
    g = GOLD["awm_two_samples"]
    per, loss = L.awm_loss(np.array(g["v"]), np.array(g["eps"]), np.array(g["x0"]), np.array(g["adv"]))
    np.testing.assert_allclose(per, g["per_sample"], rtol=0, atol=1e-15)
    assert loss == pytest.approx(g["loss"], abs=1e-15)


def test_awm_is_linear_in_advantage_and_matches_norm():
    rng = np.random.default_rng(1)
    v, eps, x0 = (rng.standard_normal((4, 7)) for _ in range(3))
    per1, _ = L.awm_loss(v, eps, x0, np.ones(4))
    np.testing.assert_allclose(per1, np.linalg.norm(v - (eps - x0), axis=1) ** 2, rtol=1e-14)
    a = rng.standard_normal(4)
    per_a, loss_a = L.awm_loss(v, eps, x0, a)
    np.testing.assert_allclose(per_a, a * per1, rtol=1e-14)
    assert loss_a == pytest.approx(np.mean(a * per1), rel=1e-14)


def test_nft_hand_example_and_limits():
    g = GOLD["nft_two_samples"]
    per, loss = L.nft_loss(np.array(g["v_pos"]), np.array(g["v_neg"]), np.array(g["eps"]), np.array(g["x0"]),
                           np.array(g["r"]))
    np.testing.assert_allclose(per, g["per_sample"], rtol=0, atol=1e-15)
    assert loss == pytest.approx(g["loss"], abs=1e-15)
    rng = np.random.default_rng(2)
    vp, vn, eps, x0 = (rng.standard_normal((3, 6)) for _ in range(4))
    target = eps - x0
    p1, _ = L.nft_loss(vp, vn, eps, x0, np.ones(3))        # r = 1: only the positive term
    np.testing.assert_allclose(p1, np.linalg.norm(vp - target, axis=1) ** 2, rtol=1e-14)
    p0, _ = L.nft_loss(vp, vn, eps, x0, np.zeros(3))       # r = 0: only the negative term
    np.testing.assert_allclose(p0, np.linalg.norm(vn - target, axis=1) ** 2, rtol=1e-14)
    ph, _ = L.nft_loss(vp, vn, eps, x0, np.full(3, 0.5))   # linear in r
    np.testing.assert_allclose(ph, 0.5 * (p0 + p1), rtol=1e-14)


def test_grpo_hand_example():
    g = GOLD["grpo_clip_two"]
    loss, n = L.grpo_loss(np.array(g["logp_new"]), np.array(g["logp_old"]), np.array(g["adv"]), None, g["clip_eps"])
    assert loss == pytest.approx(g["loss"], abs=1e-15)
    assert n == g["n_clipped"]


def test_grpo_on_policy_and_piecewise_form():
    """Equal log-probs give ratio 1 and loss -mean(w A); off-policy, the surrogate equals the
    pessimistic piecewise form min(r, 1 + eps) A for A >= 0 and max(r, 1 - eps) A for A < 0."""
    rng = np.random.default_rng(3)
    S, B, ec = 3, 10, 0.2
    lpo = rng.standard_normal((S, B)) * 50 - 1e5
    A = rng.standard_normal(B)
    w = rng.uniform(0.5, 2.0, S)
    loss, n = L.grpo_loss(lpo, lpo, A, w, ec)
    assert loss == pytest.approx(-np.sum(w[:, None] * A[None, :]) / (S * B), rel=1e-14) and n == 0
    lpn = lpo + rng.uniform(-0.5, 0.5, (S, B))
    r = np.exp(lpn - lpo)
    u = np.where(A[None, :] >= 0, np.minimum(r, 1 + ec) * A[None, :], np.maximum(r, 1 - ec) * A[None, :])
    loss, n = L.grpo_loss(lpn, lpo, A, w, ec)
    assert loss == pytest.approx(-np.sum(w[:, None] * u) / (S * B), rel=1e-13)
    assert n == int(np.sum(np.abs(r - 1) > ec))
    loss_big, _ = L.grpo_loss(lpn, lpo, A, w, 1e9)          # no clipping: the plain ratio objective
    assert loss_big == pytest.approx(-np.sum(w[:, None] * r * A[None, :]) / (S * B), rel=1e-13)
