"""Pins of the oracle's group advantages (CPU only): hand examples and invariants."""
import json
import os

import numpy as np
import pytest

from oracle import advantage as A

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


@pytest.mark.parametrize("key,mode", [("adv_weighted_two", A.MODE_WEIGHTED_SUM),
                                      ("adv_weighted_two_rewards", A.MODE_WEIGHTED_SUM),
                                      ("adv_gdpo_two_rewards", A.MODE_GDPO)])
def test_hand_examples(key, mode):
    g = GOLD[key]
    adv, counts = A.group_advantages(np.array(g["rewards"]), np.array(g["weights"]),
                                     np.array(g["group_id"]), 1, mode)
    np.testing.assert_allclose(adv, g["adv"], rtol=1e-13)
    assert counts.tolist() == [2]


def _case(seed, N=48, K=3, n_groups=6):
    rng = np.random.default_rng(seed)
    r = rng.standard_normal((N, K)) * 3 + 1
    w = rng.uniform(0.2, 2.0, K)
    gid = rng.permutation(np.repeat(np.arange(n_groups), N // n_groups))
    return r, w, gid, n_groups


@pytest.mark.parametrize("mode", [A.MODE_WEIGHTED_SUM, A.MODE_GDPO])
def test_moments_per_group(mode):
    """P12: zero mean per group; weighted-sum variance is (s/(s+eps))^2."""
    r, w, gid, G = _case(0)
    eps = 1e-4
    adv, _ = A.group_advantages(r, w, gid, G, mode, eps)
    for g in range(G):
        m = gid == g
        assert abs(adv[m].mean()) < 1e-12
        if mode == A.MODE_WEIGHTED_SUM:
            s = (r[m] @ w).std()
            assert adv[m].var() == pytest.approx((s / (s + eps)) ** 2, rel=1e-12)


def test_constant_and_singleton_groups_are_zero():
    r = np.array([[2.0], [2.0], [2.0], [5.0]])
    adv, counts = A.group_advantages(r, [1.0], [0, 0, 0, 1], 2)
    np.testing.assert_array_equal(adv, 0.0)
    assert counts.tolist() == [3, 1]


@pytest.mark.parametrize("mode", [A.MODE_WEIGHTED_SUM, A.MODE_GDPO])
def test_affine_invariance_and_permutation_equivariance(mode):
    r, w, gid, G = _case(1)
    adv, _ = A.group_advantages(r, w, gid, G, mode, eps=0.0)
    adv2, _ = A.group_advantages(3.5 * r - 7.0, w, gid, G, mode, eps=0.0)
    np.testing.assert_allclose(adv2, adv, atol=1e-12)
    perm = np.random.default_rng(2).permutation(len(gid))
    adv3, _ = A.group_advantages(r[perm], w, gid[perm], G, mode, eps=0.0)
    np.testing.assert_allclose(adv3, adv[perm], atol=1e-12)


def test_counts_exact_and_empty_group():
    gid = np.array([3, 0, 3, 3, 1, 0], dtype=np.int32)
    _, counts = A.group_advantages(np.ones((6, 1)), [1.0], gid, 5)
    assert counts.dtype == np.int32
    assert counts.tolist() == [2, 1, 0, 3, 0]


def test_gdpo_equals_weighted_sum_for_one_reward():
    r, w, gid, G = _case(3, K=1)
    a, _ = A.group_advantages(r, [1.0], gid, G, A.MODE_WEIGHTED_SUM)
    b, _ = A.group_advantages(r, [1.0], gid, G, A.MODE_GDPO)
    np.testing.assert_allclose(a, b, rtol=1e-14)
