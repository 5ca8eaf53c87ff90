"""GPU parity of ff_dit_forward and of the whole rollout against the oracle.

* the tiny float32 workload end to end: 4-step SDE rollout, per-step
  log-probs, advantages;
* small bf16 models exercising the dual-stream block (hidden mode) and the
  latent path with single-stream blocks and the pooled-text embedder;
* the full-size Flux dual-stream block (B=8, 4096 + 512 tokens, H=3072),
  checked on whole samples the oracle computes one at a time.
"""
import math

import numpy as np
import pytest
import torch

from oracle import dit as odit
from oracle import losses as olosses
from oracle import rollout as orollout
from oracle import sde as osde
from paper_2602_12529_amd import api
from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import rollout as R
from paper_2602_12529_amd import synth

from gpu_util import LOGP_ABS, TOL, check, dev, host, model_stages, rel, say

pytestmark = pytest.mark.gpu


def _inputs(w):
    m = w.model
    W = synth.weights(w)
    txt = synth.text_input(w)
    cond = synth.cond_input(w)
    x0 = synth.x0(w)
    eps = [synth.sde_noise(w, k) for k in range(w.steps)]
    return W, txt, cond, x0, eps


def _device(w, W, txt, cond, x0, eps):
    dt = w.model.dtype
    Wd = {k: dev(v, dt) for k, v in W.items()}
    return Wd, dev(txt, dt), (dev(cond, dt) if cond is not None else None), dev(x0, dt), [dev(e, dt) for e in eps]


def test_tiny_rollout_end_to_end(gpu_lib):
    """The tiny float32 workload: 2 dual blocks, 4 SDE steps, log-probs and advantages."""
    w = C.TINY
    m = w.model
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    res = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    rewards = synth.rewards(w)
    adv, counts = ro.advantages(dev(rewards))
    torch.cuda.synchronize()
    ref = orollout.rollout(m, W, x0, txt, eps, w.steps, w.eta, txt_index=synth.txt_index(w), grid=w.grid)
    assert res.ts == pytest.approx(list(ref["ts"]), abs=0)
    assert res.sigmas == pytest.approx(list(ref["sigmas"]), rel=1e-15)
    for k in range(w.steps):
        check(host(res.vs[k]), ref["vs"][k], C.F32, what=f"tiny v step {k}")
        check(host(res.xs[k + 1]), ref["xs"][k + 1], C.F32, what=f"tiny x step {k}")
        assert np.max(np.abs(host(res.logp[k]) - ref["logp"][k])) <= LOGP_ABS
        # the GRPO ratio of the rollout policy to itself is exactly 1
        lp2 = torch.empty_like(res.logp[k])
        api.logprob(res.xs[k], res.vs[k], res.xs[k + 1], lp2, res.ts[k], res.ts[k + 1], res.sigmas[k])
        torch.cuda.synchronize()
        assert torch.equal(torch.exp(lp2 - res.logp[k]), torch.ones_like(lp2))
    ref_adv, ref_cnt = orollout.advantages_for(rewards, w.group)
    np.testing.assert_allclose(host(adv), ref_adv, rtol=1e-5, atol=1e-5)
    assert counts.cpu().tolist() == ref_cnt.tolist()


def test_tiny_rollout_dance_sde_and_mixgrpo(gpu_lib):
    """The tiny workload with Dance-SDE (sigma = eta on every SDE step, Table 1) on steps {1, 3} and ODE
    steps elsewhere (MixGRPO): the whole rollout against the oracle, log-probs only on SDE steps."""
    w = C.Workload(**{**C.TINY.__dict__, "name": "tiny-dance-mix", "dynamics": "dance", "sde_steps": (1, 3)})
    m = w.model
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    ro = R.Rollout(w, api.Dit(m, Wd))
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    res = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    ref = orollout.rollout(m, W, x0, txt, eps, w.steps, w.eta, sde_steps=w.sde_steps, txt_index=synth.txt_index(w),
                           grid=w.grid, sigma_kind="dance")
    assert res.sigmas == pytest.approx(list(ref["sigmas"]), rel=1e-15)
    assert res.sigmas == [0.0, w.eta, 0.0, w.eta]
    assert sorted(res.logp) == sorted(ref["logp"]) == [1, 3]
    for k in range(w.steps):
        check(host(res.xs[k + 1]), ref["xs"][k + 1], C.F32, what=f"tiny dance/mix x step {k}")
    for k in (1, 3):
        assert np.max(np.abs(host(res.logp[k]) - ref["logp"][k])) <= LOGP_ABS


def _small_hidden():
    m = C.ModelConfig(model=C.MODEL_MMDIT, io_mode=C.IO_HIDDEN, dtype=C.BF16, n_dual=1, hidden=256, heads=2,
                      head_dim=128, mlp_hidden=1024, in_channels=64, txt_dim=256, rope_axes=(16, 56, 56))
    return C.Workload(name="small-hidden", index=11, model=m, prompts=1, group=2, grid=(1, 8, 8), n_txt=24, steps=1,
                      fixed_step=(0.6, 0.5))


@pytest.mark.parametrize("n_dual,n_single", [(1, 0), (2, 1), (0, 2)])
def test_bf16_hidden_blocks(gpu_lib, n_dual, n_single):
    w = _small_hidden()
    m = w.model.replace(n_dual=n_dual, n_single=n_single)
    w = C.Workload(**{**w.__dict__, "model": m})
    say("hidden blocks", n_dual, n_single)
    W, txt, cond, x0, _ = _inputs(w)
    Wd, T, Cd, X0, _ = _device(w, W, txt, cond, x0, [])
    dit = api.Dit(m, Wd)
    v = torch.empty_like(X0)
    tout = torch.empty_like(T)
    dit.forward(X0, T, w.grid, v, cond=Cd, txt_out=tout)
    torch.cuda.synchronize()
    img, tx = odit.forward(m, W, x0, txt, cond=cond, grid=w.grid)
    check(host(v), img, C.BF16, model_stages(m), what=f"hidden blocks {n_dual}+{n_single} img")
    check(host(tout), tx, C.BF16, model_stages(m), what=f"hidden blocks {n_dual}+{n_single} txt")
    # the blocks did act on the streams
    assert rel(img, x0) > 1e-3


def test_bf16_latent_with_single_blocks_and_pooled(gpu_lib):
    m = C.ModelConfig(model=C.MODEL_MMDIT, io_mode=C.IO_LATENT, dtype=C.BF16, n_dual=1, n_single=2, hidden=256,
                      heads=2, head_dim=128, mlp_hidden=512, in_channels=64, txt_dim=128, pooled_dim=64,
                      rope_axes=(16, 56, 56))
    w = C.Workload(name="small-latent", index=12, model=m, prompts=2, group=2, grid=(1, 4, 8), n_txt=16, steps=2)
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    res = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    # teacher-forced per step: the oracle evaluates v at the GPU's stored x_k
    for k in range(w.steps):
        xk = host(res.xs[k])
        v_ref = odit.forward(m, W, xk, txt, t=np.full(w.batch, res.ts[k]), cond=cond, txt_index=synth.txt_index(w),
                             grid=w.grid)
        check(host(res.vs[k]), v_ref, C.BF16, model_stages(m), what=f"small latent v step {k}")
        xn_ref = osde.sde_step(xk, host(res.vs[k]), eps[k], res.ts[k], res.ts[k + 1], res.sigmas[k])
        check(host(res.xs[k + 1]), xn_ref, C.BF16, 0, what=f"small latent x step {k}")
        lp_ref = osde.step_log_prob(xk, host(res.vs[k]), host(res.xs[k + 1]), res.ts[k], res.ts[k + 1], res.sigmas[k])
        assert np.max(np.abs(host(res.logp[k]) - lp_ref)) <= LOGP_ABS


@pytest.mark.parametrize("B,n_same", [(24, 6), (8, 8), (66, 4)], ids=["21-classes", "1-class", "B66-no-search"])
def test_modulation_row_classes(gpu_lib, B, n_same):
    """The adaLN GEMVs compute each distinct conditioning row once and write it to every sample of
    its class (Eq. 1's v depends on a sample's c = f(t, prompt) only).  Samples 0 .. n_same - 1 share
    t; the rest have their own t; prompts cycle over three (one prompt when all share t), so the
    classes are not contiguous and with B = 24 there are 21 of them (more than one 16-row pass).  B = 66 is past the class search
    (every row its own class).  Parity against the oracle per sample, and samples with the same
    (x, t, prompt) give bitwise equal velocities."""
    m = C.ModelConfig(model=C.MODEL_MMDIT, io_mode=C.IO_LATENT, dtype=C.BF16, n_dual=1, n_single=1, hidden=256,
                      heads=2, head_dim=128, mlp_hidden=512, in_channels=64, txt_dim=128, pooled_dim=64,
                      rope_axes=(16, 56, 56))
    w = C.Workload(name="small-latent-classes", index=17, model=m, prompts=3, group=B // 3 + (B % 3 > 0),
                   grid=(1, 4, 8), n_txt=16, steps=1)
    say("row classes", B, n_same)
    W = synth.weights(w)
    txt = synth.text_input(w)
    cond = synth.cond_input(w)
    x0 = synth.x0(w)[:B].copy()
    tidx = (np.arange(B) % 3 if n_same < B else np.zeros(B)).astype(np.int32)
    t = np.array([0.6] * n_same + list(np.linspace(0.95, 0.05, B - n_same)), dtype=np.float32)
    x0[3] = x0[0]   # sample 3: same x, t and prompt as sample 0
    Wd = {k: dev(v, m.dtype) for k, v in W.items()}
    dit = api.Dit(m, Wd)
    X = dev(x0, m.dtype)
    v = torch.empty_like(X)
    dit.forward(X, dev(txt, m.dtype), w.grid, v, t=torch.from_numpy(t).cuda(), cond=dev(cond, m.dtype),
                txt_index=torch.from_numpy(tidx).cuda())
    torch.cuda.synchronize()
    got = host(v)
    assert np.array_equal(got[3], got[0])
    ref = odit.forward(m, W, x0, txt, t=t.astype(np.float64), cond=cond, txt_index=tidx, grid=w.grid)
    check(got, ref, C.BF16, model_stages(m), what=f"row classes B={B} shared={n_same}")


def test_modulation_row_classes_hidden_mode(gpu_lib):
    """Hidden mode takes c per sample.  Rows 0, 1 are equal; row 2 equals row 0 except in its last
    column (+3), and row 4 equals row 2: the classes are {0, 1}, {2, 4}, {3}, {5}.  A merge of
    rows that differ anywhere would give samples 2 and 4 the modulation of sample 0."""
    w = _small_hidden()
    m = w.model.replace(n_dual=1, n_single=1)
    w = C.Workload(**{**w.__dict__, "model": m, "group": 6})
    W, txt, cond, x0, _ = _inputs(w)
    cond = cond.copy(); txt = txt.copy(); x0 = x0.copy()
    cond[1] = cond[0]
    cond[2] = cond[0]
    cond[2, -1] += 3.0
    cond[4] = cond[2]
    for a, b in ((1, 0), (4, 2)):
        txt[a] = txt[b]
        x0[a] = x0[b]
    Wd, T, Cd, X0, _ = _device(w, W, txt, cond, x0, [])
    dit = api.Dit(m, Wd)
    v = torch.empty_like(X0)
    tout = torch.empty_like(T)
    dit.forward(X0, T, w.grid, v, cond=Cd, txt_out=tout)
    torch.cuda.synchronize()
    got = host(v)
    assert np.array_equal(got[1], got[0]) and np.array_equal(got[4], got[2])
    img, tx = odit.forward(m, W, x0, txt, cond=cond, grid=w.grid)
    check(got, img, C.BF16, model_stages(m), what="row classes hidden img")
    check(host(tout), tx, C.BF16, model_stages(m), what="row classes hidden txt")
    # the +3 in one column of c does change the result
    assert np.max(np.abs(img[2] - img[0])) > 1e-2


def test_deep_model_modulation_launch_groups(gpu_lib):
    """The forward computes every block's modulation vectors up front, 40 weight matrices per
    launch: 21 dual blocks (42 matrices) and 3 single blocks give two launches with a segment
    boundary inside a block's pair.  float32 tiny widths with per-sample t and two prompts; the
    velocity against the oracle's whole forward."""
    m = C.TINY.model.replace(n_dual=21, n_single=3)
    w = C.Workload(**{**C.TINY.__dict__, "name": "tiny-deep", "index": 18, "model": m})
    say("deep model", m.n_dual, m.n_single)
    W, txt, cond, x0, _ = _inputs(w)
    t = np.linspace(0.9, 0.3, w.batch).astype(np.float32)
    tidx = synth.txt_index(w)
    Wd, T, Cd, X0, _ = _device(w, W, txt, cond, x0, [])
    dit = api.Dit(m, Wd)
    v = torch.empty_like(X0)
    dit.forward(X0, T, w.grid, v, t=torch.from_numpy(t).cuda(), cond=Cd, txt_index=torch.from_numpy(tidx).cuda())
    torch.cuda.synchronize()
    ref = odit.forward(m, W, x0, txt, t=t.astype(np.float64), cond=cond, txt_index=tidx, grid=w.grid)
    check(host(v), ref, C.F32, what="deep model (21 dual + 3 single) v")


def _small_latent_stack():
    m = C.ModelConfig(model=C.MODEL_MMDIT, io_mode=C.IO_LATENT, dtype=C.BF16, n_dual=1, n_single=1, hidden=256,
                      heads=2, head_dim=128, mlp_hidden=512, in_channels=64, txt_dim=128, pooled_dim=64,
                      rope_axes=(16, 56, 56))
    return C.Workload(name="small-latent-grpo", index=16, model=m, prompts=2, group=2, grid=(1, 4, 8), n_txt=16,
                      steps=3, sde_steps=(0, 2))


def test_grpo_policy_update_forward(gpu_lib):
    """The GRPO update forward on a stored rollout (MixGRPO steps {0, 2}): recomputed with the
    rollout's own weights every log-prob is bitwise the stored one (ratio 1, nothing clipped,
    loss = -mean A).  With perturbed weights, per SDE step the recomputed velocity matches the
    oracle's at the stored latent, the log-prob matches the oracle's density of the stored next
    latent given that velocity (teacher-forced, as in the rollout tests), the driver's output is
    bitwise the explicit forward + ff_logprob, and the objective matches the oracle's on those
    log-probs."""
    w = _small_latent_stack()
    m = w.model
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    ro = R.Rollout(w, api.Dit(m, Wd))
    res = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    adv = torch.from_numpy(np.array([0.5, -1.5, 1.0, 0.25], dtype=np.float32)).cuda()
    loss, n = ro.grpo_objective(res, adv, T, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    assert int(n.cpu()[0]) == 0
    assert host(loss)[0] == pytest.approx(-float(np.mean(host(adv))), rel=1e-12)
    # a slightly different policy
    W2 = {k: synth.bf16_round((v + synth.normal(500 + i, v.shape, C.F32, 0.002)).astype(np.float32))
          for i, (k, v) in enumerate(W.items())}
    ro2 = R.Rollout(w, api.Dit(m, {k: dev(v, C.BF16) for k, v in W2.items()}))
    step_w = torch.from_numpy(np.array([1.5, 0.5], dtype=np.float32)).cuda()
    new = ro2.policy_logprobs(res, T, cond=Cd, txt_index=tidx)
    loss2, n2 = gpu_lib.grpo_loss(new, torch.stack([res.logp[k] for k in ro2.sde_step_ids()]), adv, step_w, 0.2)
    torch.cuda.synchronize()
    lp_new = host(new)
    for i, k in enumerate(ro2.sde_step_ids()):
        v = torch.empty_like(res.xs[k])
        ro2.dit.forward(res.xs[k], T, w.grid, v, t=ro2.t_steps[k], cond=Cd, txt_index=tidx)
        lp = torch.empty(w.batch, dtype=torch.float64, device="cuda")
        gpu_lib.logprob(res.xs[k], v, res.xs[k + 1], lp, res.ts[k], res.ts[k + 1], res.sigmas[k])
        torch.cuda.synchronize()
        assert torch.equal(lp, new[i])
        xk, xk1 = host(res.xs[k]), host(res.xs[k + 1])
        v_ref = odit.forward(m, W2, xk, txt, t=np.full(w.batch, res.ts[k]), cond=cond,
                             txt_index=synth.txt_index(w), grid=w.grid)
        check(host(v), v_ref, C.BF16, model_stages(m), what=f"grpo recompute v step {k}")
        lp_ref = osde.step_log_prob(xk, host(v), xk1, res.ts[k], res.ts[k + 1], res.sigmas[k])
        assert np.max(np.abs(lp_new[i] - lp_ref)) <= LOGP_ABS
    old = np.stack([host(res.logp[k]) for k in ro2.sde_step_ids()])
    ref_loss, ref_n = olosses.grpo_loss(lp_new, old, host(adv), host(step_w), 0.2)
    assert host(loss2)[0] == pytest.approx(ref_loss, rel=1e-12, abs=1e-15)
    assert int(n2.cpu()[0]) == ref_n


def test_awm_training_forward(gpu_lib):
    """AWM (Eq. 3) through the model: noising, the DiT forward at per-sample t, the loss; each
    stage against the oracle on the GPU's stored inputs, and the fused driver bit-equal to the
    staged calls."""
    w = _small_latent_stack()
    m = w.model
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    ro = R.Rollout(w, api.Dit(m, Wd))
    e = synth.normal(600, x0.shape, C.BF16)
    Ed = dev(e, C.BF16)
    t = np.array([0.1, 0.4, 0.7, 0.95], dtype=np.float32)
    Td = torch.from_numpy(t).cuda()
    adv = np.array([1.0, -0.5, 2.0, 0.0], dtype=np.float32)
    Ad = torch.from_numpy(adv).cuda()
    per, loss = ro.awm_objective(X0, Ed, Td, T, Ad, cond=Cd, txt_index=tidx)
    xt = gpu_lib.flow_noise(X0, Ed, Td)
    v = torch.empty_like(X0)
    ro.dit.forward(xt, T, w.grid, v, t=Td, cond=Cd, txt_index=tidx)
    per2, loss2 = gpu_lib.awm_loss(v, Ed, X0, Ad)
    torch.cuda.synchronize()
    assert torch.equal(per, per2) and torch.equal(loss, loss2)
    check(host(xt), olosses.flow_noise(x0, e, t.astype(np.float64)), C.BF16, 0, what="awm noised x_t")
    v_ref = odit.forward(m, W, host(xt), txt, t=t.astype(np.float64), cond=cond, txt_index=synth.txt_index(w),
                         grid=w.grid)
    check(host(v), v_ref, C.BF16, model_stages(m), what="awm v")
    ref_per, ref_loss = olosses.awm_loss(host(v), e, x0, adv)
    np.testing.assert_allclose(host(per), ref_per, rtol=1e-5, atol=1e-9)
    assert host(loss)[0] == pytest.approx(ref_loss, rel=1e-5)


@pytest.mark.timeout(900)
def test_flux_dual_block_full_size(gpu_lib):
    """One Flux-shaped dual-stream block at full size (B=8, 4096 img + 512 txt, H=3072, bf16),
    one SDE step t=0.6 -> 0.5 with log-prob, as timed by the benchmark; the oracle
    recomputes two whole samples.  A second run on the same inputs is bitwise the first."""
    w = C.FLUX_BLOCK
    m = w.model
    say("full flux block: generating inputs")
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    res = ro.run(X0, T, E, cond=Cd)
    torch.cuda.synchronize()
    v = host(res.vs[0])
    xn = host(res.xs[1])
    lp = host(res.logp[0])
    say("full flux block: repeat run")
    res2 = ro.run(X0, T, E, cond=Cd)
    torch.cuda.synchronize()
    assert torch.equal(res2.vs[0], res.vs[0]) and torch.equal(res2.xs[1], res.xs[1])
    assert torch.equal(res2.logp[0], res.logp[0])
    del res2
    t, tn, sigma = res.ts[0], res.ts[1], res.sigmas[0]
    assert sigma == pytest.approx(0.7 * math.sqrt(1.5), rel=1e-15)
    for b in (0, 5):
        say("oracle sample", b)
        img, _ = odit.forward(m, W, x0[b:b + 1], txt[b:b + 1], cond=cond[b:b + 1], grid=w.grid)
        check(v[b:b + 1], img, C.BF16, model_stages(m), what=f"flux block v sample {b}")
        xr = osde.sde_step(x0[b:b + 1], v[b:b + 1], eps[0][b:b + 1], t, tn, sigma)
        check(xn[b:b + 1], xr, C.BF16, 0, what=f"flux block x' sample {b}")
        lr = osde.step_log_prob(x0[b:b + 1], v[b:b + 1], xn[b:b + 1], t, tn, sigma)
        assert abs(lp[b] - lr[0]) <= LOGP_ABS


@pytest.mark.timeout(900)
@pytest.mark.parametrize("shape", ["qwen", "flux-stack"])
def test_dual_block_full_size_other_shapes(gpu_lib, shape):
    """One dual-stream block at the other headline shapes, hidden 3072, 24 heads, MLP 12288, bf16:
    the Qwen-Image stack's (B=8, 4096 image + 256 text tokens) and the Flux stack's (B=16, 1024 +
    512), one SDE step; the fused QKV epilogue runs; the oracle recomputes two whole samples.  Both
    shapes split the last round of the K = 12288 projection along K (1632 and 1152 tiles on 256 CUs):
    a second run is bitwise the first, the partial sums being added in a fixed order."""
    base = C.FLUX_BLOCK
    if shape == "qwen":
        kw = dict(group=8, grid=(1, 64, 64), n_txt=256, index=18)
    else:
        kw = dict(group=16, grid=(1, 32, 32), n_txt=512, index=19)
    w = C.Workload(**{**base.__dict__, "name": f"dual-block-{shape}", **kw})
    m = w.model
    say(shape, "dual block: generating inputs")
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    api.profile_reset()
    api.profile_enable(True)
    try:
        res = ro.run(X0, T, E, cond=Cd)
        torch.cuda.synchronize()
    finally:
        api.profile_enable(False)
    prof = api.profile_read()
    api.profile_reset()
    assert prof.get("gemm_bf16_qkv", {}).get("launches", 0) == 1, sorted(prof)
    res2 = ro.run(X0, T, E, cond=Cd)
    torch.cuda.synchronize()
    assert torch.equal(res2.vs[0], res.vs[0]) and torch.equal(res2.xs[1], res.xs[1])
    del res2
    v = host(res.vs[0])
    for b in (0, w.batch - 1):
        say("oracle sample", b)
        img, _ = odit.forward(m, W, x0[b:b + 1], txt[b:b + 1], cond=cond[b:b + 1], grid=w.grid)
        check(v[b:b + 1], img, C.BF16, model_stages(m), what=f"{w.name} v sample {b}")


@pytest.mark.parametrize("n_dual,n_single,kernel", [(1, 0, "gemm_bf16_qkv"), (0, 1, "gemm_bf16_qkv_gelu")])
def test_fused_qkv_epilogue_ragged_streams(gpu_lib, n_dual, n_single, kernel):
    """A dual-stream block (text and image QKV projections grouped in one launch) or a single-stream
    block (Q, K, V and the MLP input from one projection, GELU from column 3H) whose QKV projection
    takes the fused QK norm / rotation / relayout epilogue.  264 text tokens per sample: 64-token
    waves straddle two samples, and in the single-stream block also the text / image boundary where
    the rotation starts; the last row tile is ragged.  Checked against the oracle on whole samples."""
    m = C.ModelConfig(model=C.MODEL_MMDIT, io_mode=C.IO_HIDDEN, dtype=C.BF16, n_dual=n_dual, n_single=n_single,
                      hidden=1536, heads=12, head_dim=128, mlp_hidden=3072, in_channels=64, txt_dim=1536,
                      rope_axes=(16, 56, 56))
    w = C.Workload(name="fused-qkv-ragged", index=17, model=m, prompts=4, group=1, grid=(1, 32, 32), n_txt=264,
                   steps=1, fixed_step=(0.6, 0.5))
    say("fused qkv:", kernel, "generating inputs")
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    api.profile_reset()
    api.profile_enable(True)
    try:
        res = ro.run(X0, T, E, cond=Cd, txt_out=torch.empty_like(T))
        torch.cuda.synchronize()
    finally:
        api.profile_enable(False)
    prof = api.profile_read()
    api.profile_reset()
    assert prof.get(kernel, {}).get("launches", 0) == 1, sorted(prof)
    assert "qk_norm_rope" not in prof
    v = host(res.vs[0])
    for b in (0, 3):
        say("oracle sample", b)
        img, _ = odit.forward(m, W, x0[b:b + 1], txt[b:b + 1], cond=cond[b:b + 1], grid=w.grid)
        check(v[b:b + 1], img, C.BF16, model_stages(m), what=f"{w.name} v sample {b}")


@pytest.mark.timeout(900)
def test_flux_single_block_full_width(gpu_lib):
    """One Flux-shaped single-stream block at full width (H=3072, fused H -> 3H + F projection,
    two-source [attention | MLP] -> H projection with 15360 inputs) on B=4 samples of 1024 image
    + 512 text tokens: both projections run on the 256 x 256 GEMM tile, the second one switching
    its A source mid-K.  The oracle recomputes two whole samples."""
    base = C.FLUX_BLOCK
    m = base.model.replace(n_dual=0, n_single=1)
    w = C.Workload(**{**base.__dict__, "name": "flux-single-block-B4", "index": 15, "model": m, "group": 4,
                      "grid": (1, 32, 32)})
    say("full-width single block: generating inputs")
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    res = ro.run(X0, T, E, cond=Cd, txt_out=torch.empty_like(T))
    torch.cuda.synchronize()
    v = host(res.vs[0])
    for b in (0, 3):
        say("oracle sample", b)
        img, _ = odit.forward(m, W, x0[b:b + 1], txt[b:b + 1], cond=cond[b:b + 1], grid=w.grid)
        check(v[b:b + 1], img, C.BF16, model_stages(m), what=f"{w.name} v sample {b}")


def _small_wan(dtype):
    if dtype == C.BF16:
        m = C.ModelConfig(model=C.MODEL_WAN, io_mode=C.IO_LATENT, dtype=C.BF16, n_wan=2, hidden=256, heads=2,
                          head_dim=128, mlp_hidden=512, in_channels=64, txt_dim=128, norm_kind=C.NORM_LN,
                          rope_axes=(44, 42, 42))
        return C.Workload(name="small-wan-bf16", index=13, model=m, prompts=1, group=2, grid=(3, 4, 4), n_txt=16,
                          steps=2)
    m = C.ModelConfig(model=C.MODEL_WAN, io_mode=C.IO_LATENT, dtype=C.F32, n_wan=2, hidden=64, heads=4,
                      head_dim=16, mlp_hidden=128, in_channels=16, txt_dim=32, norm_kind=C.NORM_LN,
                      rope_axes=(4, 6, 6))
    return C.Workload(name="small-wan-f32", index=14, model=m, prompts=2, group=1, grid=(2, 3, 4), n_txt=8, steps=2)


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
def test_wan_rollout_teacher_forced(gpu_lib, dt):
    """WAN blocks (3D RoPE, full-width QK norm, cross-attention, LN modulation) in a 2-step rollout."""
    w = _small_wan(dt)
    m = w.model
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    res = ro.run(X0, T, E, txt_index=tidx)
    torch.cuda.synchronize()
    for k in range(w.steps):
        xk = host(res.xs[k])
        v_ref = odit.forward(m, W, xk, txt, t=np.full(w.batch, res.ts[k]), txt_index=synth.txt_index(w), grid=w.grid)
        check(host(res.vs[k]), v_ref, dt, model_stages(m), what=f"{w.name} v step {k}")
        lp_ref = osde.step_log_prob(xk, host(res.vs[k]), host(res.xs[k + 1]), res.ts[k], res.ts[k + 1], res.sigmas[k])
        assert np.max(np.abs(host(res.logp[k]) - lp_ref)) <= LOGP_ABS


@pytest.mark.parametrize("dt", [C.F32, C.BF16])
def test_wan_prepared_context_matches_forward(gpu_lib, dt):
    """The per-block cross-attention K / V prepared once from the text (ff_dit_prepare_context) give
    ff_dit_forward_ctx exactly the velocities of ff_dit_forward, with prompts shared by samples."""
    w = _small_wan(dt)
    m = w.model
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    t = torch.full((w.batch,), 0.75, dtype=torch.float32, device="cuda")
    v_ref = torch.empty_like(X0)
    dit.forward(X0, T, w.grid, v_ref, t=t, txt_index=tidx)
    ctx = dit.prepare_context(T, w.grid, w.batch, txt_index=tidx)
    assert ctx.numel() == dit.context_size(w.batch, w.n_txt)
    v = torch.empty_like(X0)
    dit.forward_ctx(X0, ctx, w.n_txt, w.grid, v, t)
    torch.cuda.synchronize()
    assert torch.equal(v, v_ref)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("path", ["forward", "forward_ctx"])
def test_wan_block_full_size_sampled_rows(gpu_lib, path):
    """One WAN block at full size (B=1, 21x30x52 = 32760 video tokens, 512 text tokens, H=1536, bf16),
    through ff_dit_forward or through the path the WAN rollout takes (the text context's cross K / V
    prepared once by ff_dit_prepare_context, then ff_dit_forward_ctx); the oracle's sampled-row forward
    recomputes keys and values for all tokens and everything else for 48 query tokens."""
    base = C.WAN_STACK
    m = base.model.replace(n_wan=1)
    w = C.Workload(**{**base.__dict__, "model": m, "steps": 1})
    say("full wan block", path, ": generating inputs")
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    dit = api.Dit(m, Wd)
    v = torch.empty_like(X0)
    t = torch.full((1,), 0.6, dtype=torch.float32, device="cuda")
    tidx = torch.zeros(1, dtype=torch.int32, device="cuda")
    if path == "forward":
        dit.forward(X0, T, w.grid, v, t=t, txt_index=tidx)
    else:
        ctx = dit.prepare_context(T, w.grid, 1, txt_index=tidx)
        dit.forward_ctx(X0, ctx, w.n_txt, w.grid, v, t)
    torch.cuda.synchronize()
    rows = np.linspace(0, w.n_img - 1, 48).astype(int)
    say("  oracle rows")
    v_ref = odit.forward(m, W, x0, txt, t=np.array([0.6]), txt_index=np.zeros(1, dtype=np.int64), grid=w.grid,
                         rows=rows)
    check(host(v)[:, rows], v_ref, C.BF16, model_stages(m), what=f"wan block full size ({path}) sampled rows")


@pytest.mark.timeout(900)
def test_qwen_shaped_latent_rollout_mixgrpo(gpu_lib):
    """The Qwen-Image stack's latent model at full width (hidden 3072, 24 heads, MLP 12288, text width
    3584) cut to 2 dual blocks and 1024 + 256 tokens, B = 2, in its 10-step rollout with SDE only on
    1-indexed steps 2-4 (0-indexed {1, 2, 3}, MixGRPO): the sigma schedule and the log-prob steps
    against the oracle's schedule; per step the next latent against Eq. 1 (or the ODE step) on the
    GPU's own velocity and noise, and the log-prob of the stored latent; the velocity itself against
    the oracle's forward at the GPU's stored x_k (teacher-forced) on the steps either side of the SDE
    block and inside it."""
    base = C.QWEN_STACK
    m = base.model.replace(n_dual=2)
    w = C.Workload(**{**base.__dict__, "name": "qwen-2dual-1024img", "index": 20, "model": m, "group": 2,
                      "grid": (1, 32, 32)})
    say("qwen-shaped latent rollout: generating inputs")
    W, txt, cond, x0, eps = _inputs(w)
    Wd, T, Cd, X0, E = _device(w, W, txt, cond, x0, eps)
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    ro = R.Rollout(w, api.Dit(m, Wd))
    res = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    ref_sig = osde.schedule_sigmas(osde.time_grid(w.steps), w.eta, "flow", w.sde_steps)
    assert res.sigmas == pytest.approx(list(ref_sig), rel=1e-15)
    assert [k for k, s in enumerate(res.sigmas) if s > 0] == [1, 2, 3]
    assert sorted(res.logp) == [1, 2, 3]
    for k in range(w.steps):
        xk, vk = host(res.xs[k]), host(res.vs[k])
        xn_ref = osde.sde_step(xk, vk, eps[k], res.ts[k], res.ts[k + 1], res.sigmas[k])
        check(host(res.xs[k + 1]), xn_ref, C.BF16, 0, what=f"qwen-shaped x step {k}")
        if k in res.logp:
            lp_ref = osde.step_log_prob(xk, vk, host(res.xs[k + 1]), res.ts[k], res.ts[k + 1], res.sigmas[k])
            assert np.max(np.abs(host(res.logp[k]) - lp_ref)) <= LOGP_ABS
    for k in (0, 1, 3, 4):
        say("  oracle forward, step", k)
        v_ref = odit.forward(m, W, host(res.xs[k])[1:], txt, t=np.full(1, res.ts[k]), cond=cond,
                             txt_index=synth.txt_index(w)[1:], grid=w.grid)
        check(host(res.vs[k])[1:], v_ref, C.BF16, model_stages(m), what=f"qwen-shaped v step {k} sample 1")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("stack", ["QWEN_STACK", "FLUX_STACK", "WAN_STACK"])
def test_stack_bench_configuration(gpu_lib, stack):
    """The benchmark's stack workloads as they run there, weights drawn on the device: the
    Qwen-Image-shaped stack (60 dual blocks, B = 8 of 4096 + 256 tokens, SDE on 1-indexed steps 2-4),
    the Flux stack (19 dual + 38 single blocks, B = 16 of 1024 + 512 tokens) and WAN (30 blocks,
    32760 tokens, cross-attention to 512), bf16, whole rollouts.  The oracle cannot run such stacks,
    so the final projection's weights are zeroed and the velocity is its bias b for every token:
    every velocity must be exactly b (a non-finite value anywhere in the blocks would reach it, 0 x
    NaN being NaN), every stored latent must match the oracle's SDE or ODE step from the previous
    stored latent element by element, every log-prob the oracle's, and a second rollout is bitwise
    the first.  On the Flux stack also the GRPO update and AWM forwards the benchmark times there."""
    w = getattr(C, stack)
    m = w.model
    say(stack, "drawing weights on the device")
    g = torch.Generator(device="cuda")
    g.manual_seed(1000 + w.index)
    Wd = {}
    for name, shape, kind in synth.tensor_table(m):
        t = torch.randn(shape, device="cuda", generator=g, dtype=torch.float32).mul_(0.02)
        if kind == "norm":
            t.add_(1.0)
        Wd[name] = t.to(torch.bfloat16)
    Wd["final.proj.w"].zero_()
    b = host(Wd["final.proj.b"])
    txt, cond, x0 = synth.text_input(w), synth.cond_input(w), synth.x0(w)
    eps = [synth.sde_noise(w, k) for k in range(w.steps)]
    T, X0 = dev(txt, C.BF16), dev(x0, C.BF16)
    Cd = dev(cond, C.BF16) if cond is not None else None
    E = [dev(e, C.BF16) for e in eps]
    tidx = torch.from_numpy(synth.txt_index(w)).cuda()
    ro = R.Rollout(w, api.Dit(m, Wd))
    say(stack, "rollout")
    res = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    assert sorted(res.logp) == [k for k, sg in enumerate(res.sigmas) if sg > 0]
    for k in range(w.steps):
        xk, vk = host(res.xs[k]), host(res.vs[k])
        assert np.array_equal(vk, np.broadcast_to(b, vk.shape)), f"velocity of step {k}"
        xn_ref = osde.sde_step(xk, vk, host(E[k]), res.ts[k], res.ts[k + 1], res.sigmas[k])
        check(host(res.xs[k + 1]), xn_ref, C.BF16, 0, what=f"{stack} x step {k}")
        if k in res.logp:
            lp_ref = osde.step_log_prob(xk, vk, host(res.xs[k + 1]), res.ts[k], res.ts[k + 1], res.sigmas[k])
            assert np.max(np.abs(host(res.logp[k]) - lp_ref)) <= LOGP_ABS
    say(stack, "repeat")
    res2 = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    assert torch.equal(res2.xs[-1], res.xs[-1])
    assert all(torch.equal(res2.logp[k], res.logp[k]) for k in res.logp)
    del res2
    if stack != "FLUX_STACK":
        return
    # The training forwards the benchmark times on this stack.  GRPO update on the stored rollout:
    # recomputed with the rollout's own weights every log-prob is bitwise the stored one, so the
    # ratio is 1, nothing is clipped and the objective is -mean(A).  AWM (Eq. 3) at per-sample t:
    # with v = b the per-sample loss is the oracle's on b, the noise and x_0.
    say(stack, "GRPO and AWM forwards")
    adv = torch.from_numpy(np.linspace(-1.5, 1.5, w.batch).astype(np.float32)).cuda()
    new = ro.policy_logprobs(res, T, cond=Cd, txt_index=tidx)
    loss, n = ro.grpo_objective(res, adv, T, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    assert torch.equal(new, torch.stack([res.logp[k] for k in ro.sde_step_ids()]))
    assert int(n.cpu()[0]) == 0
    assert host(loss)[0] == pytest.approx(-float(np.mean(host(adv))), rel=1e-12)
    e = synth.normal(700, x0.shape, C.BF16)
    t = np.linspace(0.05, 0.95, w.batch).astype(np.float32)
    per, aloss = ro.awm_objective(X0, dev(e, C.BF16), torch.from_numpy(t).cuda(), T, adv, cond=Cd, txt_index=tidx)
    torch.cuda.synchronize()
    ref_per, ref_loss = olosses.awm_loss(np.broadcast_to(b, x0.shape), e, host(X0), host(adv))
    np.testing.assert_allclose(host(per), ref_per, rtol=1e-5, atol=1e-9)
    assert host(aloss)[0] == pytest.approx(ref_loss, rel=1e-5)
