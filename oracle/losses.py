"""Training objectives that consume the rollout (Sec. 3.1 and 3.2), float64.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
CPU baseline of bench.py, never by the library or its binding.

Readings where the paper is silent (the same for the HIP path):
  * Noising for the decoupled objectives follows the rollout's time convention
    (t = 1 pure noise, t = 0 data): x_t = (1 - t) x_0 + t eps, whose velocity
    d x_t / dt = eps - x_0 is the regression target of Eq. 3.
  * ||.||^2 in Eq. 2 and Eq. 3 is the squared L2 norm over all elements of a
    sample; the expectation is the mean over the samples of the batch (each
    sample carries its own t and eps).
  * Eq. 2's target v is the same forward-process velocity eps - x_0; the
    implicit positive / negative velocities v+ and v- are supplied by the
    caller (the paper does not say how they are formed from the policy).
  * The GRPO policy objective on stored trajectories is the clipped ratio
    surrogate: r = exp(logp_theta - logp_old) per (SDE step, sample),
    u = min(r A, clip(r, 1 - eps_c, 1 + eps_c) A), and the loss is
    -sum_{k,b} w_k u_{k,b} / (S B) over S SDE steps and B samples.  The
    per-step weights w_k carry a timestep-dependent reweighting such as
    GRPO-Guard's (unit weights give the plain mean).  An element counts as
    clipped when r lies outside [1 - eps_c, 1 + eps_c].
"""
from __future__ import annotations

import numpy as np


def flow_noise(x0: np.ndarray, eps: np.ndarray, t: np.ndarray) -> np.ndarray:
    """x_t = (1 - t_b) x_0 + t_b eps for samples b (first axis); t: [B]."""
    x0 = np.asarray(x0, dtype=np.float64)
    eps = np.asarray(eps, dtype=np.float64)
    tb = np.asarray(t, dtype=np.float64).reshape((-1,) + (1,) * (x0.ndim - 1))
    return (1.0 - tb) * x0 + tb * eps


def flow_target(x0: np.ndarray, eps: np.ndarray) -> np.ndarray:
    """The forward-process velocity eps - x_0 (the target of Eq. 2 and Eq. 3)."""
    return np.asarray(eps, dtype=np.float64) - np.asarray(x0, dtype=np.float64)


def _sq_norm_per_sample(d: np.ndarray) -> np.ndarray:
    d = np.asarray(d, dtype=np.float64)
    return np.sum(d.reshape(d.shape[0], -1) ** 2, axis=1)


def awm_loss(v: np.ndarray, eps: np.ndarray, x0: np.ndarray, adv: np.ndarray):
    """Eq. 3: per-sample A_b ||v_b - (eps_b - x0_b)||^2 and their mean over the batch."""
    per = np.asarray(adv, dtype=np.float64) * _sq_norm_per_sample(np.asarray(v, dtype=np.float64) - flow_target(x0, eps))
    return per, float(np.mean(per))


def nft_loss(v_pos: np.ndarray, v_neg: np.ndarray, eps: np.ndarray, x0: np.ndarray, r: np.ndarray):
    """Eq. 2: per-sample r_b ||v+_b - v_b||^2 + (1 - r_b) ||v-_b - v_b||^2, v = eps - x0, and the mean."""
    target = flow_target(x0, eps)
    r = np.asarray(r, dtype=np.float64)
    per = (r * _sq_norm_per_sample(np.asarray(v_pos, dtype=np.float64) - target)
           + (1.0 - r) * _sq_norm_per_sample(np.asarray(v_neg, dtype=np.float64) - target))
    return per, float(np.mean(per))


def grpo_loss(logp_new: np.ndarray, logp_old: np.ndarray, adv: np.ndarray, step_w, clip_eps: float):
    """Clipped ratio surrogate over logp arrays [S, B] (SDE step, sample); adv [B]; step_w [S] or None.

    Returns (loss, number of clipped elements)."""
    lpn = np.asarray(logp_new, dtype=np.float64)
    lpo = np.asarray(logp_old, dtype=np.float64)
    S, B = lpn.shape
    A = np.asarray(adv, dtype=np.float64)[None, :]
    w = np.ones(S) if step_w is None else np.asarray(step_w, dtype=np.float64)
    ratio = np.exp(lpn - lpo)
    clipped_ratio = np.clip(ratio, 1.0 - clip_eps, 1.0 + clip_eps)
    u = np.minimum(ratio * A, clipped_ratio * A)
    loss = -float(np.sum(w[:, None] * u)) / (S * B)
    n_clipped = int(np.sum((ratio < 1.0 - clip_eps) | (ratio > 1.0 + clip_eps)))
    return loss, n_clipped
