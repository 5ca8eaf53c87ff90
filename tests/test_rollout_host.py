"""Host logic of the rollout driver (CPU only: the model and the SDE call are recorded, not run)."""
import torch

from paper_2602_12529_amd import api
from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import rollout as R


class _RecordingDit:
    def workspace_size(self, B, grid, n_txt, n_prompts):
        return 16

    def forward(self, x, txt, grid, v, **kw):
        v.zero_()


def test_successive_rollouts_draw_fresh_device_noise(monkeypatch):
    """Eq. 1 draws a fresh eps ~ N(0, I) for every trajectory: each run() of one Rollout object
    passes the device noise generator a different key, and the same key for every step of a run
    (the step index is part of the counter)."""
    calls = []
    monkeypatch.setattr(api, "sde_workspace_size", lambda B, D: 16)
    monkeypatch.setattr(api, "sde_step_philox",
                        lambda x, v, xn, t, tn, s, key, k, logp=None, ws=None: calls.append((key, k)))
    w = C.Workload(**{**C.TINY.__dict__, "name": "tiny-keys"})
    ro = R.Rollout(w, _RecordingDit(), device="cpu", noise_seed=1234)
    x0 = torch.zeros(w.batch, w.n_img, w.model.in_channels)
    txt = torch.zeros(w.prompts, w.n_txt, w.model.txt_dim)
    ro.run(x0, txt, None)
    ro.run(x0, txt, None)
    assert [k for _, k in calls] == list(range(w.steps)) * 2
    first = {key for key, k in calls[:w.steps]}
    second = {key for key, k in calls[w.steps:]}
    assert len(first) == 1 and len(second) == 1 and first != second
    assert first == {ro.noise_key(0)} and second == {ro.noise_key(1)}
    assert all(0 <= key < 2 ** 64 for key, _ in calls)


def test_iter_steps_yields_each_step_once(monkeypatch):
    """The per-step generator issues the K steps in order (MixGRPO steps {1, 3} with log-probs,
    ODE steps elsewhere) and records one latent per step."""
    w = C.Workload(**{**C.TINY.__dict__, "name": "tiny-steps", "sde_steps": (1, 3)})
    calls = []
    monkeypatch.setattr(api, "sde_workspace_size", lambda B, D: 16)
    monkeypatch.setattr(api, "sde_step",
                        lambda x, v, e, xn, t, tn, s, logp=None, ws=None: calls.append((t, tn, s, logp is not None)))
    ro = R.Rollout(w, _RecordingDit(), device="cpu")
    res = R.RolloutResult(xs=[], vs=[], logp={}, ts=ro.ts, sigmas=ro.sigmas)
    ks = list(ro.iter_steps(torch.zeros(ro.shape), None, [None] * w.steps, result=res))
    assert ks == list(range(w.steps))
    assert len(res.xs) == w.steps + 1 and len(res.vs) == w.steps
    assert sorted(res.logp) == [1, 3]
    assert [c[3] for c in calls] == [False, True, False, True]
    assert [c[0] for c in calls] == ro.ts[:-1]
