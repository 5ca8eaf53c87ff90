"""Group-normalised advantages with multi-reward aggregation (Sec. 2.3), float64.

The paper names two aggregation strategies for several rewards: a weighted sum
of the rewards, and GDPO-style per-reward normalisation.  Readings used where
it gives no formula:
  * normalisation is within each group (the G samples of one prompt): subtract
    the group mean, divide by (population std + eps), eps = 1e-4;
  * weighted sum: r~ = sum_k w_k r_k first, then normalise r~;
  * GDPO: normalise each reward within the group, then take the weighted sum;
    no re-normalisation afterwards;
  * a group of one sample, or with constant rewards, gets advantage 0.
"""
from __future__ import annotations

import numpy as np

MODE_WEIGHTED_SUM = 0
MODE_GDPO = 1


def group_counts(group_id, n_groups: int) -> np.ndarray:
    counts = np.zeros(n_groups, dtype=np.int32)
    for g in np.asarray(group_id).tolist():
        counts[g] += 1
    return counts


def _normalise(values: np.ndarray, group_id: np.ndarray, n_groups: int, eps: float) -> np.ndarray:
    out = np.zeros(values.shape[0], dtype=np.float64)
    for g in range(n_groups):
        members = np.nonzero(group_id == g)[0]
        if members.size == 0:
            continue
        vals = values[members]
        mean = vals.sum() / members.size
        std = np.sqrt(np.sum((vals - mean) ** 2) / members.size)
        out[members] = (vals - mean) / (std + eps)
    return out


def group_advantages(rewards, weights, group_id, n_groups: int, mode: int = MODE_WEIGHTED_SUM,
                     eps: float = 1e-4):
    """Returns (advantages [N] float64, counts [n_groups] int32).

    rewards [N, K], weights [K], group_id [N] in [0, n_groups).
    """
    r = np.asarray(rewards, dtype=np.float64)
    if r.ndim == 1:
        r = r[:, None]
    w = np.asarray(weights, dtype=np.float64).reshape(-1)
    gid = np.asarray(group_id).astype(np.int64)
    if mode == MODE_WEIGHTED_SUM:
        adv = _normalise(r @ w, gid, n_groups, eps)
    elif mode == MODE_GDPO:
        adv = np.zeros(r.shape[0], dtype=np.float64)
        for k in range(r.shape[1]):
            adv += w[k] * _normalise(r[:, k], gid, n_groups, eps)
    else:
        raise ValueError(mode)
    return adv, group_counts(gid, n_groups)
