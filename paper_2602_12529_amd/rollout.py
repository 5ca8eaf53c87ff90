"""The K-step Flow-GRPO rollout driven through the C ABI (Sec. 3.1), and the
objectives that consume it (Sec. 3.1, 3.2).

Host side: the uniform time grid t_k = 1 - k/K, the sigma schedule of Table 1
(Flow-SDE with its t = 1 singularity evaluated with 1 - t_1, Dance-SDE, or
ODE) and the MixGRPO step mask.  Device side (all in libff.so): the DiT
velocity, the SDE step with its per-sample log-probability, the group
advantages; for training, the log-probabilities of a stored trajectory under
the current weights with the clipped-ratio GRPO objective, and the noised
forward pass with the AWM loss (Eq. 3).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import torch

from . import api
from . import configs as C


def time_grid(K: int) -> List[float]:
    return [1.0 - k / K for k in range(K + 1)]


def sigma_schedule(ts: Sequence[float], eta: float, kind: str = "flow", sde_steps=None) -> List[float]:
    """sigma_k of each step k (0 on ODE steps); Table 1."""
    out = []
    for k in range(len(ts) - 1):
        if sde_steps is not None and k not in sde_steps:
            out.append(0.0)
            continue
        t = ts[k]
        if kind == "flow":
            tt = ts[1] if t >= 1.0 else t          # 1 - t is 0 at t = 1: use the next grid point
            out.append(eta * math.sqrt(t / (1.0 - tt)))
        elif kind == "dance":
            out.append(float(eta))
        elif kind == "ode":
            out.append(0.0)
        else:
            raise ValueError(kind)
    return out


@dataclass
class RolloutResult:
    xs: List[torch.Tensor]
    vs: List[torch.Tensor]
    logp: Dict[int, torch.Tensor]
    ts: List[float]
    sigmas: List[float]
    adv: Optional[torch.Tensor] = None
    counts: Optional[torch.Tensor] = None


class Rollout:
    """Holds the model handle and the per-step buffers of one workload."""

    def __init__(self, w: C.Workload, dit: api.Dit, device="cuda", keep_velocities: bool = True,
                 noise_seed: Optional[int] = None):
        """noise_seed: draw each step's noise on the device (Philox4x32-10, counter = (element, sample,
        step), key = noise_key(rollout index)) instead of reading the eps tensors passed to run()."""
        self.w = w
        self.noise_seed = noise_seed
        self.dit = dit
        self.device = device
        self.keep_v = keep_velocities
        m = w.model
        self.dt = api.torch_dtype(m.dtype)
        B = w.batch
        width = m.hidden if m.io_mode == C.IO_HIDDEN else m.in_channels
        self.shape = (B, w.n_img, width)
        n_prompts = B if m.io_mode == C.IO_HIDDEN else w.prompts
        self.ws_dit = api.workspace(dit.workspace_size(B, w.grid, w.n_txt, n_prompts), device)
        self.ws_sde = api.workspace(api.sde_workspace_size(B, w.latent_dim), device)
        if w.fixed_step is not None:
            self.ts = [w.fixed_step[0], w.fixed_step[1]]
        else:
            self.ts = time_grid(w.steps)
        self.sigmas = sigma_schedule(self.ts, w.eta, w.dynamics, w.sde_steps)
        if w.fixed_step is not None:
            t, tn = w.fixed_step
            self.sigmas = [w.eta * math.sqrt(t / (1.0 - t))]
        # group ids (sample b belongs to prompt b // G), unit reward weights, outputs
        self.group_id = torch.tensor([b // w.group for b in range(B)], dtype=torch.int32, device=device)
        self.counts = torch.empty(w.prompts, dtype=torch.int32, device=device)
        self.adv = torch.empty(B, dtype=torch.float32, device=device)
        self.unit_weights = torch.ones(w.n_rewards, dtype=torch.float32, device=device)
        # per-step time vectors t_k for all samples, uploaded once
        self.t_steps = torch.tensor([[t] * B for t in self.ts[:-1]], dtype=torch.float32, device=device)
        self.rollouts_started = 0

    def noise_key(self, rollout_index: int) -> int:
        """The 64-bit Philox key of one rollout's on-device noise: the seed advanced by a Weyl step
        per rollout, so successive rollouts of one object draw independent noise (the counter
        already separates elements, samples and steps within a rollout)."""
        return (int(self.noise_seed) + rollout_index * 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF

    def iter_steps(self, x0, txt, eps_steps, cond=None, txt_index=None, txt_out=None, result=None):
        """The rollout one denoising step at a time: a generator that issues step k (DiT forward,
        then the SDE or ODE step with its log-prob) and yields k.  ``result`` (a RolloutResult with
        empty lists) collects the latents, velocities and log-probs as they are produced."""
        w, m = self.w, self.w.model
        B = w.batch
        x = x0
        res = result if result is not None else RolloutResult(xs=[], vs=[], logp={}, ts=list(self.ts),
                                                               sigmas=list(self.sigmas))
        res.xs.append(x0)
        key = None
        if self.noise_seed is not None:
            key = self.noise_key(self.rollouts_started)
        self.rollouts_started += 1
        # WAN: the text context is fixed along the trajectory, so its per-block cross-attention K / V
        # are prepared once and every step's forward reads them.
        context = None
        if m.model == C.MODEL_WAN:
            context = self.dit.prepare_context(txt, w.grid, B, txt_index=txt_index, ws=self.ws_dit)
        for k in range(len(self.ts) - 1):
            t, tn, sigma = self.ts[k], self.ts[k + 1], self.sigmas[k]
            v = torch.empty(self.shape, dtype=self.dt, device=self.device)
            if context is not None:
                self.dit.forward_ctx(x, context, w.n_txt, w.grid, v, self.t_steps[k], ws=self.ws_dit)
            elif m.io_mode == C.IO_LATENT:
                self.dit.forward(x, txt, w.grid, v, t=self.t_steps[k], cond=cond, txt_index=txt_index,
                                 ws=self.ws_dit)
            else:
                self.dit.forward(x, txt, w.grid, v, cond=cond, txt_out=txt_out, ws=self.ws_dit)
            x_next = torch.empty_like(x)
            lp = None
            if sigma > 0.0:
                lp = torch.empty(B, dtype=torch.float64, device=self.device)
                res.logp[k] = lp
            if key is None:
                api.sde_step(x, v, eps_steps[k], x_next, t, tn, sigma, logp=lp, ws=self.ws_sde)
            else:
                api.sde_step_philox(x, v, x_next, t, tn, sigma, key, k, logp=lp, ws=self.ws_sde)
            if self.keep_v:
                res.vs.append(v)
            res.xs.append(x_next)
            x = x_next
            yield k

    def run(self, x0, txt, eps_steps, cond=None, txt_index=None, txt_out=None) -> RolloutResult:
        res = RolloutResult(xs=[], vs=[], logp={}, ts=list(self.ts), sigmas=list(self.sigmas))
        for _ in self.iter_steps(x0, txt, eps_steps, cond=cond, txt_index=txt_index, txt_out=txt_out, result=res):
            pass
        return res

    def sde_step_ids(self) -> List[int]:
        return [k for k, s in enumerate(self.sigmas) if s > 0.0]

    def policy_logprobs(self, res: RolloutResult, txt, cond=None, txt_index=None, txt_out=None, out=None):
        """Log-probabilities of the stored SDE transitions x_k -> x_{k+1} under the current weights:
        a DiT forward at each stored x_k, then ff_logprob of the stored x_{k+1}.  Returns float64
        [S, B] in SDE-step order."""
        w, m = self.w, self.w.model
        steps = self.sde_step_ids()
        if out is None:
            out = torch.empty((len(steps), w.batch), dtype=torch.float64, device=self.device)
        for i, k in enumerate(steps):
            x = res.xs[k]
            v = torch.empty(self.shape, dtype=self.dt, device=self.device)
            if m.io_mode == C.IO_LATENT:
                self.dit.forward(x, txt, w.grid, v, t=self.t_steps[k], cond=cond, txt_index=txt_index, ws=self.ws_dit)
            else:
                self.dit.forward(x, txt, w.grid, v, cond=cond, txt_out=txt_out, ws=self.ws_dit)
            api.logprob(x, v, res.xs[k + 1], out[i], self.ts[k], self.ts[k + 1], self.sigmas[k], ws=self.ws_sde)
        return out

    def grpo_objective(self, res: RolloutResult, adv, txt, cond=None, txt_index=None, txt_out=None, step_w=None,
                       clip_eps: float = 0.2):
        """Clipped-ratio GRPO objective of a stored rollout: (loss float64 [1], clipped count int32 [1])."""
        new = self.policy_logprobs(res, txt, cond=cond, txt_index=txt_index, txt_out=txt_out)
        old = torch.stack([res.logp[k] for k in self.sde_step_ids()])
        return api.grpo_loss(new, old, adv, step_w, clip_eps)

    def awm_objective(self, x0, eps, t, txt, adv, cond=None, txt_index=None):
        """AWM (Eq. 3) on clean latents x0 noised to x_t = (1 - t) x0 + t eps at per-sample times t
        (float32 [B] on the device): (per-sample float64 [B], loss float64 [1])."""
        w, m = self.w, self.w.model
        if m.io_mode != C.IO_LATENT:
            raise ValueError("the AWM objective needs a latent-space model")
        xt = api.flow_noise(x0, eps, t)
        v = torch.empty(self.shape, dtype=self.dt, device=self.device)
        self.dit.forward(xt, txt, w.grid, v, t=t, cond=cond, txt_index=txt_index, ws=self.ws_dit)
        return api.awm_loss(v, eps, x0, adv)

    def advantages(self, rewards, weights=None, mode: int = 0, eps: float = 1e-4):
        if weights is None:
            weights = self.unit_weights if rewards.shape[1] == self.unit_weights.numel() else \
                torch.ones(rewards.shape[1], dtype=torch.float32, device=self.device)
        api.group_advantage(rewards, weights, self.group_id, self.w.prompts, mode, eps, adv=self.adv,
                            counts=self.counts)
        return self.adv, self.counts
