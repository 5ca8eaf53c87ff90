"""The K-step Flow-GRPO rollout (Sec. 3.1) with per-step log-probs and advantages, float64.

For k = 0..K-1 on the grid t_k = 1 - k/K:
  v_k = v_theta(x_k, c, t_k)
  SDE steps (MixGRPO may restrict them to a subset S): x_{k+1} = Eq. 1 step,
    log-prob of the stored x_{k+1} under the step's Gaussian transition
  ODE steps: x_{k+1} = x_k + v_k dt, no log-prob
Rewards arrive per sample; advantages are normalised per group of G samples.

``store`` rounds each new latent to the storage precision of the run
(identity for fp64/fp32 comparisons); the log-prob is of the stored value.
"""
from __future__ import annotations

import numpy as np

from . import advantage, dit, sde


def rollout(cfg, W, x0, txt, eps_steps, K: int, eta: float, sde_steps=None, cond=None,
            txt_index=None, grid=(1, 1, 1), store=lambda a: a, sigma_kind: str = "flow"):
    """Returns dict with xs [K+1] latents, vs [K], logp {k: [B]}, ts, sigmas."""
    ts = sde.time_grid(K)
    sigmas = sde.schedule_sigmas(ts, eta, sigma_kind, sde_steps)
    B = x0.shape[0]
    x = np.asarray(x0, dtype=np.float64)
    xs, vs, logp = [x], [], {}
    for k in range(K):
        t, t_next = float(ts[k]), float(ts[k + 1])
        tb = np.full(B, t)
        v = dit.forward(cfg, W, x, txt, t=tb, cond=cond, txt_index=txt_index, grid=grid)
        x_next = store(sde.sde_step(x, v, eps_steps[k], t, t_next, float(sigmas[k])))
        if sigmas[k] > 0.0:
            logp[k] = sde.step_log_prob(x, v, x_next, t, t_next, float(sigmas[k]))
        vs.append(v)
        xs.append(x_next)
        x = np.asarray(x_next, dtype=np.float64)
    return {"xs": xs, "vs": vs, "logp": logp, "ts": ts, "sigmas": sigmas}


def advantages_for(rewards, group: int, weights=None, mode: int = advantage.MODE_WEIGHTED_SUM,
                   eps: float = 1e-4):
    N = rewards.shape[0]
    gid = np.arange(N) // group
    if weights is None:
        weights = np.ones(rewards.shape[1] if rewards.ndim == 2 else 1)
    return advantage.group_advantages(rewards, weights, gid, N // group, mode, eps)
