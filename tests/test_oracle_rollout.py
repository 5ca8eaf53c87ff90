"""Pins of the oracle's K-step rollout loop (Sec. 3.1; CPU only).

The loop is checked on a model whose velocity is known in closed form: a latent DiT whose final
projection has zero weights returns its bias b for every token, sample and time, so that

* an all-ODE rollout moves every latent by b times the summed step sizes: x_K = x_0 - b exactly
  (the grid runs from t = 1 to t = 0);
* on an SDE step the stored latent minus the step's mean is the scaled noise sigma_k sqrt(|dt_k|)
  eps_k of that step, so the step's log-probability is scipy's normal log-density of that noise
  (this fixes which noise tensor, which sigma and which step size the loop pairs with step k);
* a MixGRPO mask restricts log-probabilities to its steps, and the other steps are plain Euler
  steps x_{k+1} = x_k + b dt_k.
"""
import math

import numpy as np
from scipy import stats

from oracle import dit
from oracle import rollout as orollout
from oracle import sde

from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import synth

GRID = (1, 2, 3)


def _model():
    cfg = C.ModelConfig(model=C.MODEL_MMDIT, io_mode=C.IO_LATENT, dtype=C.F32, n_dual=1, n_single=1, hidden=12,
                        heads=2, head_dim=6, mlp_hidden=10, in_channels=3, txt_dim=5, pooled_dim=4, rope_axes=(2, 2, 2))
    rng = np.random.default_rng(31)
    W = {}
    for name, shape, kind in synth.tensor_table(cfg):
        W[name] = rng.standard_normal(shape) * 0.3 + (1.0 if kind == "norm" else 0.0)
    W["final.proj.w"] = np.zeros_like(W["final.proj.w"])
    b = rng.standard_normal(W["final.proj.b"].shape)
    W["final.proj.b"] = b
    return cfg, W, b


def _inputs(cfg, B, K, seed):
    rng = np.random.default_rng(seed)
    n_img = int(np.prod(GRID))
    x0 = rng.standard_normal((B, n_img, cfg.in_channels))
    txt = rng.standard_normal((2, 4, cfg.txt_dim))
    cond = rng.standard_normal((2, cfg.pooled_dim))
    eps = [rng.standard_normal(x0.shape) for _ in range(K)]
    tidx = np.arange(B) % 2
    return x0, txt, cond, eps, tidx


def test_constant_velocity_model():
    cfg, W, b = _model()
    x0, txt, cond, _, tidx = _inputs(cfg, 3, 1, 32)
    v = dit.forward(cfg, W, x0, txt, t=np.full(3, 0.4), cond=cond, txt_index=tidx, grid=GRID)
    np.testing.assert_array_equal(v, np.broadcast_to(b, v.shape))


def test_ode_rollout_moves_by_minus_b():
    cfg, W, b = _model()
    K = 5
    x0, txt, cond, eps, tidx = _inputs(cfg, 3, K, 33)
    res = orollout.rollout(cfg, W, x0, txt, eps, K, 0.0, cond=cond, txt_index=tidx, grid=GRID)
    assert res["logp"] == {}
    np.testing.assert_allclose(res["xs"][-1], x0 - b, rtol=0, atol=1e-14)
    np.testing.assert_allclose(res["ts"], [1.0, 0.8, 0.6, 0.4, 0.2, 0.0], rtol=0, atol=1e-15)


def test_sde_steps_pair_noise_sigma_and_step():
    cfg, W, b = _model()
    K, eta = 4, 0.7
    mask = (1, 2)
    x0, txt, cond, eps, tidx = _inputs(cfg, 3, K, 34)
    res = orollout.rollout(cfg, W, x0, txt, eps, K, eta, sde_steps=mask, cond=cond, txt_index=tidx, grid=GRID)
    ts, sig = res["ts"], res["sigmas"]
    assert sorted(res["logp"]) == list(mask)
    for k in range(K):
        dt = ts[k + 1] - ts[k]
        xk, xn = res["xs"][k], res["xs"][k + 1]
        np.testing.assert_array_equal(res["vs"][k], np.broadcast_to(b, xk.shape))
        if k not in mask:
            assert sig[k] == 0.0
            np.testing.assert_allclose(xn, xk + b * dt, rtol=0, atol=1e-14)
            continue
        # sigma of Table 1's Flow-SDE row at t_k, with t = 1 clipped to the next grid point
        tt = ts[1] if ts[k] == 1.0 else ts[k]
        assert sig[k] == math.sqrt(tt / (1.0 - tt)) * eta
        scale = sig[k] * math.sqrt(-dt)
        noise = xn - sde.sde_mean(xk, res["vs"][k], ts[k], dt, sig[k])
        np.testing.assert_allclose(noise, scale * eps[k], rtol=1e-12, atol=1e-14)
        ref = stats.norm.logpdf(scale * eps[k], loc=0.0, scale=scale).reshape(3, -1).sum(axis=1)
        np.testing.assert_allclose(res["logp"][k], ref, rtol=1e-11)
