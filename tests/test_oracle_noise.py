"""Pins of the oracle's counter-based noise (CPU only): the generator's published known-answer
vectors, and the Gaussian law of the Box-Muller output."""
import json
import os

import numpy as np
import pytest
from scipy import stats

from oracle import noise as N

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


@pytest.mark.parametrize("case", GOLD["philox4x32_10_kat"]["cases"])
def test_philox_known_answers(case):
    ctr = np.array([int(x, 16) for x in case["ctr"]], dtype=np.uint64)
    key = [int(x, 16) for x in case["key"]]
    got = N.philox4x32_10(ctr, key)
    assert [f"{int(x):08x}" for x in got] == case["out"]


def test_box_muller_is_standard_normal():
    z = N.sde_noise(4, 50000, seed=12345, step=3).ravel()
    assert abs(z.mean()) < 5 * 1 / np.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * np.sqrt(2 / z.size)
    assert stats.kstest(z, "norm").pvalue > 1e-4
    # pairs from one Box-Muller draw are uncorrelated
    zz = N.sde_noise(1, 400000, seed=7, step=0).reshape(-1, 2)
    assert abs(np.corrcoef(zz[:, 0], zz[:, 1])[0, 1]) < 5 / np.sqrt(zz.shape[0])


def test_streams_differ_by_sample_step_and_seed():
    base = N.sde_noise(2, 64, seed=1, step=0)
    assert not np.allclose(base[0], base[1])
    assert not np.allclose(base, N.sde_noise(2, 64, seed=1, step=1))
    assert not np.allclose(base, N.sde_noise(2, 64, seed=2, step=0))
    # a shorter sample is a prefix of a longer one (the layout depends on d only)
    np.testing.assert_array_equal(N.sde_noise(2, 10, seed=1, step=0), base[:, :10])
