"""Throughput of the Flow-GRPO rollout hot path on one MI355X.

One step = one pass of the whole hot path over one batch: the DiT velocity
forward (here one Flux-shaped dual-stream block, B = 8 samples of 4096 image
+ 512 text tokens, hidden 3072, bf16), the SDE step with its per-sample
log-probability, and the group-normalised advantages.  Inputs are synthetic
(seeded, N(0, 0.02) weights, N(0, 1) activations) and resident in HBM before
timing starts.

Prints one JSON line: steps/s (and latent tokens/s), the roofline of the
dominant kernel measured with HIP events on its launch stream over the timed
region, and the plain CPU oracle timed on a bounded sample of the same work.
The per-kernel breakdown comes from an untimed pass in which every launch is
bracketed by events; in the timed region only the dominant kernel's launches
are, since events around every launch cost about 1% of a step.

The other workloads (--workload flux-stack | qwen-stack | wan) run whole
rollouts of the full model: 19 dual + 38 single Flux blocks (B = 16, 1024 +
512 tokens, 10 SDE steps), 60 Qwen-Image-shaped dual blocks (B = 8, 4096 +
256 tokens, 10 steps with SDE on steps 2-4) or 30 WAN blocks (B = 1, 32760 +
512 tokens, 8 steps).  Their weights are drawn on the device (N(0, 0.02),
norm weights 1 + N(0, 0.02)); a step is one denoising step of the batch, and
--steps / --warmup count whole rollouts.  Two training-side workloads run on
the Flux stack: grpo-flux-stack times the GRPO policy-update forward over a
stored rollout (a DiT forward and a log-prob recompute per SDE step, then the
clipped-ratio objective; a step is one recomputed SDE step), awm-flux-stack
the AWM training forward (noising at per-sample t, DiT forward, Eq. 3 loss; a
step is one forward of the batch).  The oracle is timed on the default
workload only.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
                       [--workload flux-block|flux-stack|qwen-stack|wan|tiny]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SDE rollout steps/sec and latent tokens/sec per GPU; % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E

# workload name -> (configs attribute, default timed units, default warmup units); the one-block
# and tiny workloads time single steps, the stacks whole rollouts.
WORKLOADS = {"flux-block": ("FLUX_BLOCK", 20, 3), "tiny": ("TINY", 20, 3), "flux-stack": ("FLUX_STACK", 2, 1),
             "qwen-stack": ("QWEN_STACK", 1, 1), "wan": ("WAN_STACK", 2, 1),
             "grpo-flux-stack": ("FLUX_STACK", 2, 1), "awm-flux-stack": ("FLUX_STACK", 10, 2)}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="flux-block", choices=list(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--noise", default="stored", choices=["stored", "philox"],
                    help="read each step's noise from HBM (default) or draw it in the SDE kernel")
    ap.add_argument("--cpu-samples", type=int, default=3, help="samples of the batch the oracle times")
    return ap.parse_args()


def main() -> int:
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
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
    print(f"[bench] workload {w.name}: generating inputs", file=sys.stderr, flush=True)
    device_drawn = args.workload in ("flux-stack", "qwen-stack", "wan", "grpo-flux-stack", "awm-flux-stack")
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
    steps_per_unit = len(ro.sigmas)     # denoising steps in one timed unit (a rollout, or the one step)

    def step():
        res = ro.run(X0, T, E, cond=Cd, txt_index=tidx, txt_out=txt_out)
        ro.advantages(rewards)
        return res

    if args.workload == "grpo-flux-stack":
        print("[bench] storing one rollout for the policy update", file=sys.stderr, flush=True)
        stored = step()
        adv_stored = ro.adv.clone()
        steps_per_unit = len(ro.sde_step_ids())
        step_w = torch.ones(steps_per_unit, dtype=torch.float32, device="cuda")

        def step():  # noqa: F811 -- the timed unit of this workload
            return ro.grpo_objective(stored, adv_stored, T, cond=Cd, txt_index=tidx, step_w=step_w)
    elif args.workload == "awm-flux-stack":
        g = torch.Generator(device="cuda")
        g.manual_seed(2000 + w.index)
        t_awm = torch.rand(w.batch, generator=g, device="cuda", dtype=torch.float32)
        eps_awm = torch.randn(X0.shape, generator=g, device="cuda", dtype=torch.float32).to(dt)
        adv_awm = torch.randn(w.batch, generator=g, device="cuda", dtype=torch.float32)
        steps_per_unit = 1

        def step():  # noqa: F811 -- the timed unit of this workload
            return ro.awm_objective(X0, eps_awm, t_awm, T, adv_awm, cond=Cd, txt_index=tidx)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Per-kernel breakdown: an untimed pass with every launch bracketed by HIP events (the events
    # cost ~1% of a step, so the timed region below brackets the dominant kernel only).
    bd_units = 1 if steps_per_unit > 1 else min(args.steps, 5)
    api.profile_filter(None)
    api.profile_reset()
    api.profile_enable(True)
    for _ in range(bd_units):
        step()
    torch.cuda.synchronize()
    api.profile_enable(False)
    prof = api.profile_read()
    bd_steps = bd_units * steps_per_unit
    dominant = max(prof, key=lambda n: prof[n]["ms"])
    # Timed region: events around the dominant kernel's launches only.
    api.profile_reset()
    api.profile_filter(dominant)
    api.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
        if steps_per_unit > 1:
            print(f"[bench] rollout {i + 1}/{args.steps} issued", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    api.profile_enable(False)
    prof_timed = api.profile_read()
    api.profile_filter(None)
    print(f"[bench] timed {args.steps} steps in {elapsed:.3f} s", file=sys.stderr, flush=True)

    n_steps = args.steps * steps_per_unit
    ms_per_step = 1e3 * elapsed / n_steps
    steps_per_s = n_steps / elapsed
    latent_tok_s = steps_per_s * w.batch * w.n_img

    # Per-kernel achieved rates from the breakdown pass's HIP events.
    kernels = {}
    for name, p in prof.items():
        avg_ms = p["ms"] / max(p["launches"], 1)
        k = {"launches_per_step": p["launches"] / bd_steps, "avg_us": 1e3 * avg_ms,
             "ms_per_step": p["ms"] / bd_steps}
        if p["flops"] > 0 and name.startswith(("gemm", "attn")):
            k["tflops"] = p["flops"] / (p["ms"] * 1e-3) / 1e12
            k["mfma_frac"] = k["tflops"] / (PEAK_BF16_TFLOPS if m.dtype == C.BF16 else PEAK_FP32_TFLOPS)
        elif p["bytes"] > 0:
            k["gbs"] = p["bytes"] / (p["ms"] * 1e-3) / 1e9
            k["hbm_frac"] = k["gbs"] / PEAK_HBM_GBS
        kernels[name] = k
    block_flops = sum(p["flops"] for n, p in prof.items() if n.startswith(("gemm", "attn"))) / bd_steps
    dp = prof_timed[dominant]   # the dominant kernel, timed live over the timed region
    per_launch = {"flops": dp["flops"] / dp["launches"], "algorithmic_bytes": dp["bytes"] / dp["launches"],
                  "avg_us": 1e3 * dp["ms"] / dp["launches"]}
    # HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary of this kernel,
    # null when there is none or the kernel's sources have changed since it was taken.
    rec = profiling.lookup_traffic(dominant)
    traffic = rec["traffic_bytes_per_launch"] if rec else None
    if rec:
        per_launch["traffic_source"] = rec["summary"]
    compute_bound = dp["flops"] > 0 and dominant.startswith(("gemm", "attn"))
    if compute_bound:
        peak = PEAK_BF16_TFLOPS if m.dtype == C.BF16 else PEAK_FP32_TFLOPS
        achieved = dp["flops"] / (dp["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": traffic, "kernel": dominant, "per_launch": per_launch}
    else:
        achieved = dp["bytes"] / (dp["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS, "traffic": traffic, "kernel": dominant, "per_launch": per_launch}

    cpu = None
    if not args.no_cpu_baseline and W is not None:
        cpu = cpu_baseline(w, W, txt, cond, x0, eps, args.cpu_samples)

    out = {
        "metric": METRIC,
        "value": steps_per_s,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": n_steps,
        "warmup": args.warmup * steps_per_unit,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if m.dtype == C.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "img_tokens": w.n_img, "txt_tokens": w.n_txt,
                   "hidden": m.hidden, "heads": m.heads, "head_dim": m.head_dim, "mlp_hidden": m.mlp_hidden,
                   "dual_blocks": m.n_dual, "single_blocks": m.n_single, "wan_blocks": m.n_wan,
                   "denoising_steps": len(ro.sigmas), "sde_steps": sum(1 for s in ro.sigmas if s > 0),
                   "timed_unit": {"grpo-flux-stack": "GRPO update forward over a stored rollout",
                                  "awm-flux-stack": "AWM training forward of the batch"}.get(
                       args.workload, "rollout" if steps_per_unit > 1 else "step"),
                   "weights": "device-drawn N(0,0.02)" if device_drawn else "host-drawn N(0,0.02), seeded",
                   "noise": "Philox4x32-10 in the SDE kernel" if args.noise == "philox" else "stored eps tensors",
                   "t": ro.ts[0], "t_next": ro.ts[1], "sigma": ro.sigmas[0]},
        "latent_tokens_per_s": latent_tok_s,
        "sample_steps_per_s": steps_per_s * w.batch,
        "model_tflops": block_flops / (ms_per_step * 1e-3) / 1e12,
        "model_mfma_frac": block_flops / (ms_per_step * 1e-3) / 1e12 /
                           (PEAK_BF16_TFLOPS if m.dtype == C.BF16 else PEAK_FP32_TFLOPS),
        "roofline": roof,
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


def cpu_baseline(w, W, txt, cond, x0, eps, n_samples: int):
    """The oracle (as it stands) on a bounded sample of the step: n_samples of the batch's samples
    through the DiT forward, the SDE step and its log-prob, plus the advantages; scaled to steps/s."""
    import numpy as np

    from oracle import dit as odit
    from oracle import rollout as orollout
    from oracle import sde as osde
    from paper_2602_12529_amd import configs as C
    from paper_2602_12529_amd import rollout as R
    from paper_2602_12529_amd import synth

    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        threads = 1
    m = w.model
    ts = [w.fixed_step[0], w.fixed_step[1]] if w.fixed_step else R.time_grid(w.steps)
    n = min(n_samples, w.batch)
    print(f"[bench] cpu baseline: oracle on {n} of {w.batch} samples, {threads} threads", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    x = x0[:n].astype(np.float64)
    tidx = synth.txt_index(w)[:n]
    for k in range(len(ts) - 1):
        t, tn = ts[k], ts[k + 1]
        sigma = (w.eta * math.sqrt(t / (1 - t))) if w.fixed_step else R.sigma_schedule(ts, w.eta, w.dynamics, w.sde_steps)[k]
        if m.io_mode == C.IO_HIDDEN:
            v, _ = odit.forward(m, W, x, txt[:n], cond=cond[:n], grid=w.grid)
        else:
            v = odit.forward(m, W, x, txt, t=np.full(n, t), cond=cond, txt_index=tidx, grid=w.grid)
        xn = osde.sde_step(x, v, eps[k][:n], t, tn, sigma)
        if sigma > 0:
            osde.step_log_prob(x, v, xn, t, tn, sigma)
        x = xn
    orollout.advantages_for(synth.rewards(w), w.group)
    el = time.perf_counter() - t0
    per_step = el * (w.batch / n)
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} of {w.batch} samples of one step (DiT forward fp64, SDE step, log-prob, advantages), "
                      f"{el:.1f} s measured, scaled by {w.batch}/{n} to the full batch"}


if __name__ == "__main__":
    sys.exit(main())
