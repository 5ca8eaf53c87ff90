"""Throughput of the Flow-GRPO rollout hot path on one MI355X.

Default workload: the Qwen-Image-shaped stack (60 dual-stream blocks, hidden 3072, 24 heads x 128,
MLP 12288, B = 8 samples of 4096 image + 256 text tokens, bf16) in its 10-step rollout on the
uniform grid with the SDE step only on 1-indexed steps 2-4 (MixGRPO) and ODE steps elsewhere.

One step = one denoising step of the whole batch: the DiT velocity forward (embedders, the 60
blocks, the final layer), then the SDE step with its per-sample log-probability (or the ODE step),
and, on the step that ends a rollout, the group-normalised advantages.  --steps K times exactly K
such steps, walking through successive rollouts (20 steps = two rollouts' worth, every window of
10 consecutive steps holds the three SDE steps).  Weights are drawn on the device (N(0, 0.02^2),
norm weights 1 + N(0, 0.02^2)); prompt embeddings, x_1 and the SDE noise are seeded host draws;
everything is resident in HBM before timing starts.

Prints one JSON line: steps/s (and latent tokens/s), the roofline of the dominant kernel measured
with HIP events on its launch stream over the timed region, and the plain CPU oracle.  The
per-kernel breakdown comes from an untimed pass of one rollout in which every launch is bracketed
by events; in the timed region only the dominant kernel's launches are, since events around
every launch cost about 1% of a step.

The CPU oracle (float64 numpy) is timed on the host in the same run.  For the stacks it times one
block of each kind at full shape with one sample (WAN: sampled query rows, extrapolated linearly
in the row count), the embedders and final layer, the SDE step and log-prob at full size and the
advantages, and extrapolates to a batch step by block count x samples; the line says
"extrapolated".  The one-block and tiny workloads are timed in full.

Other workloads (--workload): flux-block (one Flux-shaped dual-stream block, B = 8, 4096 + 512
tokens, one SDE step t = 0.6 -> 0.5 on the block's hidden state), qwen-block (the same with the
Qwen stack's block shape, 4096 + 256 tokens: its launches are the stack's), flux-stack (19 dual + 38 single
blocks, B = 16, 1024 + 512 tokens, 10 SDE steps), wan (30 WAN blocks, B = 1, 32760 + 512 tokens,
8 steps), tiny, and two training-side workloads on the Flux stack: grpo-flux-stack (the GRPO
policy-update forward over a stored rollout; a step is one recomputed SDE step) and
awm-flux-stack (noising, DiT forward, Eq. 3 loss; a step is one forward of the batch).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time


def _host_threads() -> int:
    """Host threads for the oracle: the CPUs this process may run on, capped by an OMP_NUM_THREADS
    the environment already sets (a shared box's per-GPU CPU share)."""
    n = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS", "")
    if share.isdigit() and int(share) > 0:
        n = min(n, int(share))
    return n


# The BLAS thread pools are sized when numpy is first imported, so this runs before any import
# that loads it (torch does).
HOST_THREADS = _host_threads()
for _var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ[_var] = str(HOST_THREADS)

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SDE rollout steps/sec and latent tokens/sec per GPU; % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
TARGET_MFMA, TARGET_HBM = 0.50, 0.70

# workload name -> (configs attribute, default timed steps, default warmup steps)
WORKLOADS = {"qwen-stack": ("QWEN_STACK", 20, 5), "flux-block": ("FLUX_BLOCK", 20, 5), "tiny": ("TINY", 20, 5),
             "qwen-block": ("QWEN_BLOCK", 20, 5),
             "flux-stack": ("FLUX_STACK", 20, 5), "wan": ("WAN_STACK", 16, 4),
             "grpo-flux-stack": ("FLUX_STACK", 2, 1), "awm-flux-stack": ("FLUX_STACK", 10, 2)}
DEVICE_DRAWN = ("flux-stack", "qwen-stack", "wan", "grpo-flux-stack", "awm-flux-stack")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="qwen-stack", choices=list(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--noise", default="stored", choices=["stored", "philox"],
                    help="read each step's noise from HBM (default) or draw it in the SDE kernel")
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def main() -> int:
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the rollout would shard by prompt groups with no communication until the advantages).",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2602_12529_amd import api
    from paper_2602_12529_amd import configs as C
    from paper_2602_12529_amd import profiling
    from paper_2602_12529_amd import rollout as R
    from paper_2602_12529_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    api.load()
    attr, def_steps, def_warmup = WORKLOADS[args.workload]
    w = getattr(C, attr)
    args.steps = def_steps if args.steps is None else args.steps
    args.warmup = def_warmup if args.warmup is None else args.warmup
    m = w.model
    dt = api.torch_dtype(m.dtype)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda().to(dt)
    log(f"workload {w.name}: generating inputs")
    device_drawn = args.workload in DEVICE_DRAWN
    if device_drawn:
        W = None
        Wd = device_weights(m, 1000 + w.index, dt)
    else:
        W = synth.weights(w)
        Wd = {k: dev(v) for k, v in W.items()}
    txt, cond, x0 = synth.text_input(w), synth.cond_input(w), synth.x0(w)
    eps = [synth.sde_noise(w, k) for k in range(len(R.time_grid(w.steps)) - 1)]
    T, Cd, X0 = dev(txt), (dev(cond) if cond is not None else None), dev(x0)
    E = [dev(e) for e in eps]
    rewards = torch.from_numpy(synth.rewards(w)).cuda()
    tidx = torch.from_numpy(synth.txt_index(w)).cuda() if m.io_mode == C.IO_LATENT else None
    dit = api.Dit(m, Wd)
    ro = R.Rollout(w, dit, keep_velocities=False, noise_seed=(3000 + w.index) if args.noise == "philox" else None)
    txt_out = torch.empty_like(T) if m.io_mode == C.IO_HIDDEN else None
    K = len(ro.sigmas)                  # denoising steps of one rollout
    steps_per_rollout = K
    state = {"it": None}

    def step():
        """One denoising step of the batch, continuing the current rollout (a new one starts after the
        last step; the step that ends a rollout also computes the advantages)."""
        if state["it"] is None:
            state["it"] = ro.iter_steps(X0, T, E, cond=Cd, txt_index=tidx, txt_out=txt_out)
        k = next(state["it"])
        if k == K - 1:
            ro.advantages(rewards)
            state["it"] = None

    timed_unit = "denoising step of the batch (DiT forward, SDE/ODE step with log-prob; advantages at rollout end)"
    if args.workload == "grpo-flux-stack":
        log("storing one rollout for the policy update")
        stored = ro.run(X0, T, E, cond=Cd, txt_index=tidx)
        ro.advantages(rewards)
        adv_stored = ro.adv.clone()
        steps_per_rollout = len(ro.sde_step_ids())
        step_w = torch.ones(steps_per_rollout, dtype=torch.float32, device="cuda")
        timed_unit = "GRPO update forward over a stored rollout (a step is one recomputed SDE step)"

        def step():  # noqa: F811 -- the timed unit of this workload: a whole update, counted as its SDE steps
            return ro.grpo_objective(stored, adv_stored, T, cond=Cd, txt_index=tidx, step_w=step_w)
    elif args.workload == "awm-flux-stack":
        g = torch.Generator(device="cuda")
        g.manual_seed(2000 + w.index)
        t_awm = torch.rand(w.batch, generator=g, device="cuda", dtype=torch.float32)
        eps_awm = torch.randn(X0.shape, generator=g, device="cuda", dtype=torch.float32).to(dt)
        adv_awm = torch.randn(w.batch, generator=g, device="cuda", dtype=torch.float32)
        steps_per_rollout = 1
        timed_unit = "AWM training forward of the batch"

        def step():  # noqa: F811 -- the timed unit of this workload
            return ro.awm_objective(X0, eps_awm, t_awm, T, adv_awm, cond=Cd, txt_index=tidx)
    calls_per_step = steps_per_rollout if args.workload == "grpo-flux-stack" else 1
    n_calls = max(1, args.steps // calls_per_step) if calls_per_step > 1 else args.steps
    n_warm = max(1, args.warmup // calls_per_step) if calls_per_step > 1 else args.warmup

    log(f"warmup {args.warmup} steps")
    for _ in range(n_warm):
        step()
    torch.cuda.synchronize()
    # Per-kernel breakdown: an untimed pass over one rollout's worth of steps with every launch
    # bracketed by HIP events (the events cost ~1% of a step, so the timed region below brackets
    # the dominant kernel only).
    bd_calls = 1 if calls_per_step > 1 else max(K, 1)
    api.profile_filter(None)
    api.profile_reset()
    api.profile_enable(True)
    for _ in range(bd_calls):
        step()
    torch.cuda.synchronize()
    api.profile_enable(False)
    prof = api.profile_read()
    bd_steps = bd_calls * calls_per_step
    dominant = max(prof, key=lambda n: prof[n]["ms"])
    # Timed region: events around the dominant kernel's launches only.
    api.profile_reset()
    api.profile_filter(dominant)
    api.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(n_calls):
        step()
        if (i + 1) % 10 == 0:
            log(f"{i + 1}/{n_calls} issued")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    api.profile_enable(False)
    prof_timed = api.profile_read()
    api.profile_filter(None)
    n_steps = n_calls * calls_per_step
    log(f"timed {n_steps} steps in {elapsed:.3f} s")

    ms_per_step = 1e3 * elapsed / n_steps
    steps_per_s = n_steps / elapsed
    latent_tok_s = steps_per_s * w.batch * w.n_img
    peak_mfma = PEAK_BF16_TFLOPS if m.dtype == C.BF16 else PEAK_FP32_TFLOPS

    # Per-kernel achieved rates from the breakdown pass's HIP events.
    kernels = {}
    for name, p in prof.items():
        avg_ms = p["ms"] / max(p["launches"], 1)
        k = {"launches_per_step": p["launches"] / bd_steps, "avg_us": 1e3 * avg_ms,
             "ms_per_step": p["ms"] / bd_steps}
        if p["flops"] > 0 and name.startswith(("gemm", "attn")):
            k["tflops"] = p["flops"] / (p["ms"] * 1e-3) / 1e12
            k["mfma_frac"] = k["tflops"] / peak_mfma
        elif p["bytes"] > 0:
            k["gbs"] = p["bytes"] / (p["ms"] * 1e-3) / 1e9
            k["hbm_frac"] = k["gbs"] / PEAK_HBM_GBS
        kernels[name] = k
    model_flops = sum(p["flops"] for n, p in prof.items() if n.startswith(("gemm", "attn"))) / bd_steps
    dp = prof_timed[dominant]   # the dominant kernel, timed live over the timed region
    per_launch = {"flops": dp["flops"] / dp["launches"], "algorithmic_bytes": dp["bytes"] / dp["launches"],
                  "avg_us": 1e3 * dp["ms"] / dp["launches"], "launches_timed": dp["launches"]}
    # HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary of this kernel on this
    # workload, null when there is none or the kernel's sources have changed since it was taken.
    rec = profiling.lookup_traffic(dominant, w.name)
    traffic = rec["traffic_bytes_per_launch"] if rec else None
    if rec:
        per_launch["traffic_source"] = rec["summary"]
    if dp["flops"] > 0 and dominant.startswith(("gemm", "attn")):
        achieved = dp["flops"] / (dp["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak_mfma, "unit": "TFLOP/s",
                "frac": achieved / peak_mfma, "traffic": traffic, "kernel": dominant, "per_launch": per_launch}
    else:
        achieved = dp["bytes"] / (dp["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS, "traffic": traffic, "kernel": dominant, "per_launch": per_launch}

    # Each kernel family against its own bar: MFMA kernels >= 50% of the bf16 peak, the HBM-bound
    # SDE / log-prob kernels >= 70% of 8 TB/s.  A miss is reported as a miss.
    def family(prefix, key):
        sel = {n: p for n, p in prof.items() if n.startswith(prefix)}
        tot_ms = sum(p["ms"] for p in sel.values())
        if not sel or tot_ms <= 0:
            return None
        if key == "flops":
            frac = sum(p["flops"] for p in sel.values()) / (tot_ms * 1e-3) / 1e12 / peak_mfma
            return {"frac_of_peak": frac, "target": TARGET_MFMA, "met": frac >= TARGET_MFMA,
                    "share_of_step": tot_ms / bd_steps / ms_per_step}
        frac = sum(p["bytes"] for p in sel.values()) / (tot_ms * 1e-3) / 1e9 / PEAK_HBM_GBS
        return {"frac_of_peak": frac, "target": TARGET_HBM, "met": frac >= TARGET_HBM,
                "share_of_step": tot_ms / bd_steps / ms_per_step}
    targets = {"gemm": family("gemm", "flops"), "attention": family("attn", "flops"),
               "sde_step": family("sde_step", "bytes"),
               "model_mfma_frac": model_flops / (ms_per_step * 1e-3) / 1e12 / peak_mfma}
    if targets["sde_step"] is not None:
        # below ~64 MB per call the step is launch-latency bound (~10-20 us) and fits the 256 MB MALL;
        # its bandwidth bar applies to calls of hundreds of MB (the size sweep under profiles/)
        targets["sde_step"]["bytes_per_call"] = w.batch * w.latent_dim * 4 * (2 if m.dtype == C.BF16 else 4)

    cpu = None
    if not args.no_cpu_baseline and args.workload not in ("grpo-flux-stack", "awm-flux-stack"):
        cpu = cpu_baseline(w, W)

    out = {
        "metric": METRIC,
        "value": steps_per_s,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": n_steps,
        "warmup": n_warm * calls_per_step,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if m.dtype == C.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "img_tokens": w.n_img, "txt_tokens": w.n_txt,
                   "hidden": m.hidden, "heads": m.heads, "head_dim": m.head_dim, "mlp_hidden": m.mlp_hidden,
                   "dual_blocks": m.n_dual, "single_blocks": m.n_single, "wan_blocks": m.n_wan,
                   "denoising_steps_per_rollout": K, "sde_steps_per_rollout": sum(1 for s in ro.sigmas if s > 0),
                   "sde_step_ids": [k for k, s in enumerate(ro.sigmas) if s > 0],
                   "timed_unit": timed_unit,
                   "weights": "device-drawn N(0,0.02)" if device_drawn else "host-drawn N(0,0.02), seeded",
                   "noise": "Philox4x32-10 in the SDE kernel" if args.noise == "philox" else "stored eps tensors"},
        "latent_tokens_per_s": latent_tok_s,
        "sample_steps_per_s": steps_per_s * w.batch,
        "model_tflops": model_flops / (ms_per_step * 1e-3) / 1e12,
        "model_mfma_frac": targets["model_mfma_frac"],
        "roofline": roof,
        "targets": targets,
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


def device_weights(m, seed: int, dt):
    """Random weights of the model drawn on the device: N(0, 0.02^2), norm weights 1 + N(0, 0.02^2)."""
    import torch

    from paper_2602_12529_amd import synth

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    out = {}
    for name, shape, kind in synth.tensor_table(m):
        t = torch.randn(shape, device="cuda", generator=g, dtype=torch.float32).mul_(0.02)
        if kind == "norm":
            t.add_(1.0)
        out[name] = t.to(dt)
    return out


def _timed(fn):
    t0 = time.perf_counter()
    r = fn()
    return time.perf_counter() - t0, r


def cpu_baseline(w, W):
    """The oracle (as it stands, float64 numpy) on the host cores.  One-block and tiny workloads: the
    whole step.  Stacks: one block of each kind at full shape with one sample, the embedders and
    final layer, the SDE step, log-prob and advantages at full size; extrapolated to a batch step."""
    import numpy as np

    from oracle import dit as odit
    from oracle import rollout as orollout
    from oracle import sde as osde
    from paper_2602_12529_amd import configs as C
    from paper_2602_12529_amd import rollout as R
    from paper_2602_12529_amd import synth

    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        blas_threads = HOST_THREADS
    m = w.model
    ts = [w.fixed_step[0], w.fixed_step[1]] if w.fixed_step else R.time_grid(w.steps)
    if w.fixed_step:
        sigmas = [w.eta * math.sqrt(ts[0] / (1 - ts[0]))]
    else:
        sigmas = R.sigma_schedule(ts, w.eta, w.dynamics, w.sde_steps)
    K = len(sigmas)
    txt, cond, x0 = synth.text_input(w), synth.cond_input(w), synth.x0(w)
    x0d = x0.astype(np.float64)
    eps0 = synth.sde_noise(w, 0)
    log(f"cpu baseline: oracle on {HOST_THREADS} host threads ({blas_threads} BLAS threads)")

    # the SDE / ODE step (and log-prob on SDE steps) and the advantages at full size
    t_sde = 0.0
    for k in range(K):
        tk, tn, s = ts[k], ts[k + 1], sigmas[k]
        dt_, xn = _timed(lambda: osde.sde_step(x0d, x0d, eps0, tk, tn, s))
        t_sde += dt_
        if s > 0:
            t_sde += _timed(lambda: osde.step_log_prob(x0d, x0d, xn, tk, tn, s))[0]
    t_adv = _timed(lambda: orollout.advantages_for(synth.rewards(w), w.group))[0]
    update_per_step = t_sde / K + t_adv / K

    if W is not None:
        # one-block / tiny workloads: the whole step (or rollout) on the full batch
        def full():
            x = x0d
            tidx = synth.txt_index(w)
            for k in range(K):
                if m.io_mode == C.IO_HIDDEN:
                    v, _ = odit.forward(m, W, x, txt, cond=cond, grid=w.grid)
                else:
                    v = odit.forward(m, W, x, txt, t=np.full(w.batch, ts[k]), cond=cond, txt_index=tidx, grid=w.grid)
                xn = osde.sde_step(x, v, synth.sde_noise(w, k), ts[k], ts[k + 1], sigmas[k])
                if sigmas[k] > 0:
                    osde.step_log_prob(x, v, xn, ts[k], ts[k + 1], sigmas[k])
                x = xn
            orollout.advantages_for(synth.rewards(w), w.group)
        el = _timed(full)[0]
        per_step = el / K
        return {"value": 1.0 / per_step, "unit": "steps/s", "cores": HOST_THREADS, "kind": "oracle",
                "extrapolated": False,
                "sample": f"the whole {'step' if K == 1 else f'{K}-step rollout'} of the batch ({w.batch} samples: "
                          f"DiT forward, SDE steps, log-probs, advantages) in float64, {el:.1f} s measured"}

    # stacks: one block of each kind at full shape, B = 1, on seeded host weights of block 0
    one = {"n_dual": 1 if m.n_dual else 0, "n_single": 1 if m.n_single else 0, "n_wan": 1 if m.n_wan else 0}
    w1 = C.Workload(**{**w.__dict__, "model": m.replace(**one), "prompts": 1, "group": 1})
    W1 = synth.weights(w1)
    x1 = x0d[:1]
    tid = np.zeros(1, dtype=np.int64)
    t_mid = np.array([ts[1]])
    ang = odit.rope_angles(odit.grid_positions(w.grid), m.rope_axes, m.rope_theta)
    parts = {}
    if m.model == C.MODEL_MMDIT:
        c = odit.mlp2(odit.timestep_sinusoid(t_mid), W1, "temb.fc1", "temb.fc2", odit.silu)
        if m.pooled_dim:
            c = c + odit.mlp2(odit.f64(cond)[tid], W1, "pooled.fc1", "pooled.fc2", odit.silu)
        x_img = odit.linear(x1, W1, "x_in")
        x_txt = odit.linear(txt, W1, "txt_in")[tid]
        t_edge = _timed(lambda: odit.forward(w1.model.replace(n_dual=0, n_single=0), W1, x1, txt, t=t_mid,
                                             cond=cond, txt_index=tid, grid=w.grid))[0]
        if m.n_dual:
            parts["dual"] = (_timed(lambda: odit.dual_block(x_img, x_txt, c, W1, 0, m, ang))[0], m.n_dual)
        if m.n_single:
            xj = np.concatenate([x_txt, x_img], axis=1)
            parts["single"] = (_timed(lambda: odit.single_block(xj, c, W1, 0, m, w.n_txt, ang))[0], m.n_single)
        how = "one block of each kind timed in full"
    else:
        temb = odit.mlp2(odit.timestep_sinusoid(t_mid), W1, "temb.fc1", "temb.fc2", odit.silu)
        e6 = odit.linear(odit.silu(temb), W1, "temb.proj").reshape(1, 6, -1)
        ctx = odit.mlp2(txt, W1, "txt_in.fc1", "txt_in.fc2", odit.gelu_tanh)[tid]
        xh = odit.linear(x1, W1, "x_in")
        t_edge = _timed(lambda: odit.final_layer(xh, temb, W1, m))[0]
        t_edge += _timed(lambda: odit.linear(x1, W1, "x_in"))[0]
        # the sampled-row block is linear in the row count: keys / values of all tokens plus each row
        r1, r2 = 64, 192
        rows1 = np.linspace(0, w.n_img - 1, r1).astype(np.int64)
        rows2 = np.linspace(0, w.n_img - 1, r2).astype(np.int64)
        ta = _timed(lambda: odit.wan_block(xh, ctx, e6, W1, 0, m, ang, rows=rows1))[0]
        tb = _timed(lambda: odit.wan_block(xh, ctx, e6, W1, 0, m, ang, rows=rows2))[0]
        per_row = max(tb - ta, 0.0) / (r2 - r1)
        t_block = ta + per_row * (w.n_img - r1)
        parts["wan"] = (t_block, m.n_wan)
        how = (f"one WAN block on {r1} and {r2} sampled query rows ({ta:.1f} s, {tb:.1f} s), "
               f"extrapolated linearly to {w.n_img} rows")
    per_step = w.batch * (t_edge + sum(t * n for t, n in parts.values())) + update_per_step
    detail = ", ".join(f"{k} block {t:.2f} s x {n}" for k, (t, n) in parts.items())
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": HOST_THREADS, "kind": "oracle",
            "extrapolated": True,
            "sample": f"float64 oracle, one sample: {detail} ({how}); embedders + final layer {t_edge:.2f} s; "
                      f"x {w.batch} samples; plus SDE/ODE steps, log-probs and advantages at full size "
                      f"({update_per_step * 1e3:.1f} ms per step); extrapolated to {per_step:.0f} s per batch step"}


if __name__ == "__main__":
    sys.exit(main())
