"""GPU parity of ff_sde_step / ff_logprob / ff_group_advantage against the oracle."""
import math

import numpy as np
import pytest
import torch

from oracle import advantage as oadv
from oracle import sde as osde
from paper_2602_12529_amd import configs as C

from gpu_util import LOGP_ABS, TOL, check, dev, host, normal, rel, say, tdt

pytestmark = pytest.mark.gpu

SHAPES = [(8, 256), (3, 1000), (1, 1), (2, 7), (5, 12345), (4, 65536), (2, 8 * 2048 + 8)]
STEPS = [(1.0, 0.75, 0.7 * math.sqrt(1 / 0.25)), (0.6, 0.5, 0.7 * math.sqrt(1.5)), (0.25, 0.0, 0.4)]


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("B,D", SHAPES)
@pytest.mark.parametrize("t,tn,sigma", STEPS)
def test_sde_step_parity(gpu_lib, dt, B, D, t, tn, sigma):
    say("sde", dt, B, D, t, tn, sigma)
    x, v, e = (normal(100 + i, (B, D), dt) for i in range(3))
    X, V, E = dev(x, dt), dev(v, dt), dev(e, dt)
    Xn = torch.empty_like(X)
    lp = torch.empty(B, dtype=torch.float64, device="cuda")
    gpu_lib.sde_step(X, V, E, Xn, t, tn, sigma, logp=lp)
    lp2 = torch.empty_like(lp)
    gpu_lib.logprob(X, V, Xn, lp2, t, tn, sigma)
    Xn2 = torch.empty_like(X)
    lp3 = torch.empty_like(lp)
    gpu_lib.sde_step(X, V, E, Xn2, t, tn, sigma, logp=lp3)
    torch.cuda.synchronize()
    ref = osde.sde_step(x, v, e, t, tn, sigma)
    got = host(Xn)
    check(got, ref, dt, 0, 3, what=f"sde step {B}x{D} t={t}")
    if dt == C.F32:
        assert np.max(np.abs(got - ref)) <= 1e-5 * (1 + np.max(np.abs(ref)))
    # the log-prob of the stored next latent (its rounding is part of the stored value)
    lp_ref = osde.step_log_prob(x, v, got, t, tn, sigma)
    assert np.max(np.abs(host(lp) - lp_ref)) <= LOGP_ABS
    # recomputation and repetition are bitwise identical
    assert torch.equal(lp, lp2) and torch.equal(lp, lp3) and torch.equal(Xn, Xn2)


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
def test_ode_step_and_no_logprob(gpu_lib, dt):
    x, v = normal(7, (4, 999), dt), normal(8, (4, 999), dt)
    X, V = dev(x, dt), dev(v, dt)
    Xn = torch.empty_like(X)
    gpu_lib.sde_step(X, V, X, Xn, 0.7, 0.6, 0.0)
    torch.cuda.synchronize()
    check(host(Xn), osde.sde_step(x, v, None, 0.7, 0.6, 0.0), dt, 0, 2, what="ode step")
    with pytest.raises(gpu_lib.FFError):
        gpu_lib.sde_step(X, V, X, Xn, 0.7, 0.6, 0.0, logp=torch.empty(4, dtype=torch.float64, device="cuda"))


def test_logprob_at_mean_matches_closed_form(gpu_lib):
    """x_next = mean exactly (eps = 0 in f32): logp = -D/2 log(2 pi sigma^2 |dt|) per sample."""
    B, D = 3, 40000
    x, v = normal(11, (B, D)), normal(12, (B, D))
    X, V = dev(x), dev(v)
    Xn = torch.empty_like(X)
    lp = torch.empty(B, dtype=torch.float64, device="cuda")
    t, tn, s = 0.8, 0.7, 1.1
    gpu_lib.sde_step(X, V, torch.zeros_like(X), Xn, t, tn, s, logp=lp)
    torch.cuda.synchronize()
    closed = -0.5 * D * math.log(2 * math.pi * s * s * (t - tn))
    assert np.max(np.abs(host(lp) - closed)) <= LOGP_ABS


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
def test_empty_samples_and_empty_batch(gpu_lib, dt):
    """Degenerate sizes: samples with no elements have log-density 0 (the oracle's empty sum) from
    every step entry point and from the recomputation; an empty batch is a no-op."""
    say("empty samples", dt)
    B = 5
    X = torch.empty((B, 0), dtype=tdt(dt), device="cuda")
    ref = osde.step_log_prob(np.zeros((B, 0)), np.zeros((B, 0)), np.zeros((B, 0)), 0.6, 0.5, 0.9)
    assert np.all(ref == 0.0)
    calls = {
        "sde_step": lambda lp: gpu_lib.sde_step(X, X, X, torch.empty_like(X), 0.6, 0.5, 0.9, logp=lp),
        "logprob": lambda lp: gpu_lib.logprob(X, X, X, lp, 0.6, 0.5, 0.9),
        "sde_step_philox": lambda lp: gpu_lib.sde_step_philox(X, X, torch.empty_like(X), 0.6, 0.5, 0.9, 7, 1, logp=lp),
        "sde_step_noalloc": lambda lp: gpu_lib.sde_step_noalloc(X, X, X, torch.empty_like(X), 0.6, 0.5, 0.9, logp=lp),
    }
    for name, f in calls.items():
        lp = torch.full((B,), float("nan"), dtype=torch.float64, device="cuda")
        f(lp)
        torch.cuda.synchronize()
        assert np.array_equal(host(lp), ref), name
    # B = 0: nothing is written (the sentinel behind the empty view stays)
    lp = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
    Z = torch.empty((0, 16), dtype=tdt(dt), device="cuda")
    gpu_lib.sde_step(Z, Z, Z, torch.empty_like(Z), 0.6, 0.5, 0.9, logp=lp[:0])
    gpu_lib.logprob(Z, Z, Z, lp[:0], 0.6, 0.5, 0.9)
    torch.cuda.synchronize()
    assert torch.isnan(lp).all()


def test_sde_full_size_flux_block_shape(gpu_lib):
    """The 1024^2 Flux hidden-state reading of the SDE step: B=8, D=4096*3072, bf16."""
    B, D = 8, 4096 * 3072
    t, tn = 0.6, 0.5
    sigma = 0.7 * math.sqrt(t / (1 - t))
    say("sde full size", B, D)
    x, v, e = (normal(200 + i, (B, D), C.BF16) for i in range(3))
    X, V, E = dev(x, C.BF16), dev(v, C.BF16), dev(e, C.BF16)
    Xn = torch.empty_like(X)
    lp = torch.empty(B, dtype=torch.float64, device="cuda")
    gpu_lib.sde_step(X, V, E, Xn, t, tn, sigma, logp=lp)
    torch.cuda.synchronize()
    got = host(Xn)
    check(got, osde.sde_step(x, v, e, t, tn, sigma), C.BF16, 0, 3, what="sde step full size 8x12.58M")
    lp_ref = osde.step_log_prob(x, v, got, t, tn, sigma)
    assert np.max(np.abs(host(lp) - lp_ref)) <= LOGP_ABS


# ------------------------------------------------------------------ advantages
ADV_CASES = [
    # N, K, n_groups, mode
    (8, 1, 2, 0), (16, 1, 1, 0), (64, 3, 8, 0), (64, 3, 8, 1), (1000, 4, 100, 1), (1, 1, 1, 0), (4096, 1, 4096, 0),
]


@pytest.mark.parametrize("N,K,G,mode", ADV_CASES)
def test_group_advantage_parity(gpu_lib, N, K, G, mode):
    say("adv", N, K, G, mode)
    rng = np.random.default_rng(N * 31 + K)
    r = rng.uniform(0, 1, (N, K)).astype(np.float32)
    w = rng.uniform(0.5, 2, K).astype(np.float32)
    gid = rng.permutation(np.arange(N) % G).astype(np.int32)
    adv = gpu_lib.group_advantage(dev(r), dev(w), torch.from_numpy(gid).cuda(), G, mode,
                                  counts=(cnt := torch.empty(G, dtype=torch.int32, device="cuda")))
    torch.cuda.synchronize()
    ref, ref_cnt = oadv.group_advantages(r, w, gid, G, mode)
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    np.testing.assert_allclose(host(adv), ref, rtol=1e-5, atol=1e-5)


def test_group_advantage_edge_cases(gpu_lib):
    r = np.array([[2.0], [2.0], [2.0], [5.0], [1.0], [3.0]], dtype=np.float32)
    gid = np.array([0, 0, 0, 1, 3, 9], dtype=np.int32)       # group 2 empty; id 9 out of range
    cnt = torch.empty(4, dtype=torch.int32, device="cuda")
    adv = gpu_lib.group_advantage(dev(r), dev(np.ones(1)), torch.from_numpy(gid).cuda(), 4, 0, counts=cnt)
    torch.cuda.synchronize()
    a = adv.cpu().numpy()
    assert cnt.cpu().tolist() == [3, 1, 0, 1]
    assert np.all(a[:5] == 0.0) and np.isnan(a[5])
    # no samples: every group is empty
    cnt = torch.full((3,), -1, dtype=torch.int32, device="cuda")
    gpu_lib.group_advantage(torch.empty((0, 2), device="cuda"), dev(np.ones(2)), torch.empty(0, dtype=torch.int32, device="cuda"),
                            3, 1, counts=cnt)
    torch.cuda.synchronize()
    assert cnt.cpu().tolist() == [0, 0, 0]


# ------------------------------------------------------------------ counter-based noise
from oracle import noise as onoise  # noqa: E402


def _u32(t):
    return t.cpu().numpy().view(np.uint32)


def test_philox_known_answers_on_device(gpu_lib):
    import json
    import os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))
    for case in gold["philox4x32_10_kat"]["cases"]:
        c = [int(x, 16) for x in case["ctr"]]
        k = [int(x, 16) for x in case["key"]]
        w = gpu_lib.philox4x32(1, c[0] | (c[1] << 32), c[2], c[3], k[0] | (k[1] << 32))
        torch.cuda.synchronize()
        assert [f"{int(x):08x}" for x in _u32(w)[0]] == case["out"]


def test_philox_words_match_oracle_bit_exact(gpu_lib):
    n, base, c2, c3, key = 100003, (1 << 32) - 17, 5, 9, 0x0123456789ABCDEF
    w = _u32(gpu_lib.philox4x32(n, base, c2, c3, key))
    i = np.arange(n, dtype=np.uint64) + np.uint64(base)
    ctr = np.stack([i & np.uint64(0xFFFFFFFF), i >> np.uint64(32), np.full(n, c2, np.uint64),
                    np.full(n, c3, np.uint64)], axis=-1)
    ref = onoise.philox4x32_10(ctr, (key & 0xFFFFFFFF, key >> 32))
    assert np.array_equal(w, ref)


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("B,D", [(3, 1000), (2, 7), (4, 65536), (1, 8 * 2048 + 8)])
def test_philox_normal_matches_oracle(gpu_lib, dt, B, D):
    seed, step = 0x5EED0000ABCD, 4
    z = gpu_lib.philox_normal((B, D), seed, step, dtype=torch.bfloat16 if dt == C.BF16 else torch.float32)
    torch.cuda.synchronize()
    ref = onoise.sde_noise(B, D, seed, step)
    got = host(z)
    # float32 Box-Muller: log, sqrt, sin/cos to a few ulp of |z| <= ~6.7; bf16 adds half an ulp
    bound = (2.0 ** -8 * np.abs(ref) if dt == C.BF16 else 0.0) + 2e-5
    assert np.all(np.abs(got - ref) <= bound)


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("B,D", [(8, 256), (3, 1000), (2, 7), (4, 65536)])
def test_sde_step_philox_parity(gpu_lib, dt, B, D):
    t, tn, sigma, seed, step = 0.6, 0.5, 0.7 * math.sqrt(1.5), 987654321, 2
    x, v = normal(200, (B, D), dt), normal(201, (B, D), dt)
    X, V = dev(x, dt), dev(v, dt)
    Xn = torch.empty_like(X)
    lp = torch.empty(B, dtype=torch.float64, device="cuda")
    gpu_lib.sde_step_philox(X, V, Xn, t, tn, sigma, seed, step, logp=lp)
    lp2 = torch.empty_like(lp)
    gpu_lib.logprob(X, V, Xn, lp2, t, tn, sigma)
    torch.cuda.synchronize()
    eps = onoise.sde_noise(B, D, seed, step)
    ref = osde.sde_step(x, v, eps, t, tn, sigma)
    got = host(Xn)
    assert rel(got, ref) <= TOL[dt]
    # element-wise on the kernel's own float32 noise (which matches the oracle's Box-Muller to 2e-5
    # absolute, test_philox_normal_matches_oracle): near-zero outputs would otherwise see that difference
    # times sigma sqrt|dt| against a bound scaled by their own magnitude
    e32 = host(gpu_lib.philox_normal((B, D), seed, step))
    check(got, osde.sde_step(x, v, e32, t, tn, sigma), dt, 0, 3, what=f"sde step philox {B}x{D}")
    assert np.max(np.abs(host(lp) - osde.step_log_prob(x, v, got, t, tn, sigma))) <= LOGP_ABS
    assert torch.equal(lp, lp2)   # the recompute of the fused step's log-prob is bitwise identical
    if dt == C.F32:
        # the fused step equals the step on the materialised noise, bit for bit
        E = gpu_lib.philox_normal((B, D), seed, step)
        Xn2 = torch.empty_like(X)
        lp3 = torch.empty_like(lp)
        gpu_lib.sde_step(X, V, E, Xn2, t, tn, sigma, logp=lp3)
        torch.cuda.synchronize()
        assert torch.equal(Xn, Xn2) and torch.equal(lp, lp3)
