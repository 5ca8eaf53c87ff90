"""rocprofv3 summaries for the rollout's kernels, and the HBM traffic lookup of bench.py.

Subcommands (python -m paper_2602_12529_amd.profiling ...):

  copy --bytes N --reps R
      A plain device-to-device copy of N bytes, R times: the calibration kernel
      whose FETCH_SIZE / WRITE_SIZE counters are compared with the known N.
  ceiling OUT --title T --cmd C [--reps R]
      The HBM streaming ceiling (ff_stream_probe: read, write, copy over 1 GiB, non-temporal or
      not, a sweep of grid sizes) beside a torch copy and the rollout's HBM-bound kernels at
      full size, in one process -> markdown table.
  sde-sweep OUT --title T --cmd C [--reps R]
      The SDE step with log-prob over 1 MB .. 2 GB of traffic, warm and cold (rotating
      buffer sets beyond the MALL), per-launch HIP events -> markdown table.
  linear --M --N --K --precision bf16|fp8 [--gelu] --reps R
      One linear layer on random device data, R times, timed per launch by the
      library's events (fp8: the activation quantiser and the FP8 GEMM).
  stats CSV OUT --title T --cmd C
      kernel_stats.csv of `rocprofv3 --kernel-trace --stats` -> markdown table.
  counter CSV OUT --counter NAME --title T --cmd C [--note N]
      one counter of a `rocprofv3 --pmc` run (e.g. the derived MfmaUtil) per kernel.
  traffic --fetch CSV --write CSV --copy-fetch CSV --copy-write CSV --copy-bytes N
          --workload W --key NAME=PATTERN OUT --title T --cmd C [--cmd C ...]
      counter_collection.csv files of four `rocprofv3 --pmc` runs (FETCH_SIZE,
      then WRITE_SIZE, over the workload and over the copy) -> per-kernel HBM
      bytes per launch.  Each counter is scaled by N / (its value for the copy),
      so the numbers are in the copy's units: bytes that crossed the HBM
      interface.  NAME is the library's profiler name of the kernel the bench
      reports (gemm_bf16_gated, attn_bf16, ...), PATTERN a substring of
      rocprofv3's kernel name; the summary stores NAME's traffic per launch
      with the workload's name and the hash of the sources the kernel is built
      from, and bench.py reports it for that workload only while that hash
      still matches.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys
from collections import defaultdict
from typing import Dict, List, Optional

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_12529_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")

# Source files each kernel family is compiled from (beside the shared headers).
_FAMILY_SOURCES = {
    "gemm": ["gemm.hip"],
    "attn": ["attention.hip"],
    "sde": ["sde.hip"],
    "logp": ["sde.hip"],
    "group_adv": ["sde.hip"],
}
_SHARED = ["dev.h", "ff_internal.h"]


def sources_of(kernel: str) -> List[str]:
    fam = next((v for k, v in _FAMILY_SOURCES.items() if kernel.startswith(k)), ["ops.hip", "dit.hip"])
    return [os.path.join(CSRC, f) for f in fam + _SHARED]


def sources_sha256(kernel: str) -> str:
    h = hashlib.sha256()
    for path in sources_of(kernel):
        with open(path, "rb") as f:
            h.update(os.path.basename(path).encode() + b"\0" + f.read())
    return h.hexdigest()


def short_name(name: str) -> str:
    s = name.replace("void ", "").replace("ff::(anonymous namespace)::", "")
    s = s.replace("(anonymous namespace)::", "")
    depth, out = 0, []
    for ch in s:                     # drop the argument list
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    s = "".join(out)
    return s if len(s) <= 70 else s[:67] + "..."


# ---------------------------------------------------------------------------- copy calibration
def run_copy(nbytes: int, reps: int) -> None:
    import torch

    if not torch.cuda.is_available():
        raise SystemExit("copy calibration needs a GPU")
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    src.random_(0, 255)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def run_linear(M: int, N: int, K: int, precision: str, gelu: bool, reps: int) -> dict:
    """Times one linear layer (bf16 ff_linear, or fp8 ff_quantize_fp8 of the activations plus
    ff_linear_fp8) on random device data with the library's own per-launch events."""
    import torch

    from . import api

    if not torch.cuda.is_available():
        raise SystemExit("linear timing needs a GPU")
    g = torch.Generator(device="cuda").manual_seed(0)
    x = torch.randn((M, K), device="cuda", generator=g).to(torch.bfloat16)
    w = (torch.randn((N, K), device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    b = (torch.randn((N,), device="cuda", generator=g) * 0.1).to(torch.bfloat16)
    out = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
    epi = api.EPI_GELU if gelu else api.EPI_BIAS
    if precision == "fp8":
        wq, wd = api.quantize_fp8(w)
        xq = torch.empty((M, K), device="cuda", dtype=torch.uint8)
        xd = torch.empty((M,), device="cuda", dtype=torch.float32)

        def step():
            api.quantize_fp8(x, xq, xd)
            api.linear_fp8(xq, xd, wq, wd, b, out, epi=epi)
    else:
        def step():
            api.linear(x, w, b, out, epi=epi)
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    api.profile_reset()
    api.profile_enable(True)
    for _ in range(reps):
        step()
    torch.cuda.synchronize()
    api.profile_enable(False)
    prof = api.profile_read()
    res = {"M": M, "N": N, "K": K, "precision": precision, "gelu": gelu, "reps": reps, "kernels": {}}
    peak = 5000.0 if precision == "fp8" else 2500.0
    for name, r in prof.items():
        k = {"avg_us": 1e3 * r["ms"] / r["launches"]}
        if r["flops"] > 0:
            k["tflops"] = r["flops"] / (r["ms"] * 1e-3) / 1e12
            k["frac_of_dense_peak"] = k["tflops"] / peak
        elif r["bytes"] > 0:
            k["gbs"] = r["bytes"] / (r["ms"] * 1e-3) / 1e9
        res["kernels"][name] = k
    print(json.dumps(res), flush=True)
    return res


def run_sde_sweep(out_md: str, title: str, cmds: List[str], reps: int = 20) -> List[dict]:
    """The SDE step with log-prob (ff_sde_step, bf16, B = 8) over sizes of 1 MB to 2 GB of algorithmic
    traffic (x, v, eps read, x' written: 8 bytes per element), each timed per launch with HIP events
    (median of `reps`): warm, re-running on one buffer set (the 256 MB MALL holds the small ones),
    and cold, rotating over enough buffer sets to cover at least twice the MALL (at least four)."""
    import statistics

    import torch

    from . import api

    if not torch.cuda.is_available():
        raise SystemExit("the SDE size sweep needs a GPU")
    B, mall = 8, 256 << 20
    rows = []
    sizes = [1 << 20, 4 << 20, 16 << 20, 64 << 20, 256 << 20, 805306368, 1 << 30, 2 << 30]
    g = torch.Generator(device="cuda").manual_seed(0)
    for total in sizes:
        D = max(2048, total // (8 * B) // 2048 * 2048)
        nbytes = 8 * B * D
        sets = max(4, -(-2 * mall // nbytes))
        bufs = []
        for _ in range(sets):
            x = torch.randn((B, D), device="cuda", generator=g).to(torch.bfloat16)
            v = torch.randn((B, D), device="cuda", generator=g).to(torch.bfloat16)
            e = torch.randn((B, D), device="cuda", generator=g).to(torch.bfloat16)
            bufs.append((x, v, e, torch.empty_like(x), torch.empty(B, dtype=torch.float64, device="cuda")))
        ws = api.workspace(api.sde_workspace_size(B, D))
        res = {"bytes": nbytes, "elements_per_sample": D, "cold_sets": sets}
        for mode in ("warm", "cold"):
            times = []
            for i in range(reps + 3):
                x, v, e, xn, lp = bufs[0] if mode == "warm" else bufs[i % sets]
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                api.sde_step(x, v, e, xn, 0.6, 0.5, 0.9, logp=lp, ws=ws)
                e1.record()
                e1.synchronize()
                if i >= 3:
                    times.append(e0.elapsed_time(e1) * 1e-3)
            med = statistics.median(times)
            res[mode + "_us"] = med * 1e6
            res[mode + "_tbs"] = nbytes / med / 1e12
        rows.append(res)
        print(json.dumps(res), flush=True)
        del bufs
        torch.cuda.empty_cache()
    out = _header(title, cmds)
    out += ["ff_sde_step with its log-prob, bf16, B = 8; median of %d launches, each bracketed by HIP events "
            "on the launch stream. Warm: one buffer set re-run; cold: rotating over the stated number of "
            "sets (together at least twice the 256 MB MALL). Peak HBM 8 TB/s." % reps, "",
            "| bytes per launch | elements per sample | warm µs | warm TB/s | cold sets | cold µs | cold TB/s | cold / 8 TB/s |",
            "|---|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {r['bytes'] / 1e6:.1f} MB | {r['elements_per_sample']} | {r['warm_us']:.1f} | "
                   f"{r['warm_tbs']:.2f} | {r['cold_sets']} | {r['cold_us']:.1f} | {r['cold_tbs']:.2f} | "
                   f"{r['cold_tbs'] / 8.0:.2f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(out) + "\n")
    return rows


def run_ceiling(out_md: str, title: str, cmds: List[str], reps: int = 10) -> List[dict]:
    """Streaming ceiling of HBM on the box: ff_stream_probe read-only, write-only and copy over 1 GiB
    (four times the 256 MB MALL), non-temporal or not, over a sweep of grid sizes, the best of
    each; beside them, in the same process, a plain torch copy and the rollout's HBM-bound kernels
    at full size (the SDE step with log-prob of the one-block workload, 8 x 12.58 M bf16; the norm
    + modulate of a 32768 x 3072 image stream; the adaLN GEMV of one stream, B = 8, 6H x H).
    Each entry is the median of `reps` launches timed with the library's HIP events."""
    import statistics

    import torch

    from . import api

    if not torch.cuda.is_available():
        raise SystemExit("the streaming ceiling needs a GPU")

    def timed(fn, name):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        times = []
        for _ in range(reps):
            api.profile_filter(name)
            api.profile_reset()
            api.profile_enable(True)
            fn()
            torch.cuda.synchronize()
            api.profile_enable(False)
            r = api.profile_read()[name]
            times.append(r["ms"] * 1e-3 / r["launches"])
        api.profile_filter(None)
        return statistics.median(times)

    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.random_(0, 255)
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    rows, best = [], {}
    for mode, label in ((0, "read"), (1, "write"), (2, "copy")):
        moved = n * (2 if mode == 2 else 1)
        for nt in (True, False):
            for blocks in (1024, 2048, 4096, 8192, 16384):
                t = timed(lambda: api.stream_probe(mode, src, dst, n, blocks, nt), "stream_probe")
                r = {"what": f"probe {label}", "nt": nt, "blocks": blocks, "bytes": moved, "us": t * 1e6,
                     "tbs": moved / t / 1e12}
                rows.append(r)
                if label not in best or r["tbs"] > best[label]["tbs"]:
                    best[label] = r
                print(json.dumps(r), flush=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        dst.copy_(src)
    times = []
    for _ in range(reps):
        e0.record()
        dst.copy_(src)
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1) * 1e-3)
    t = statistics.median(times)
    kern = [{"what": "torch copy_", "bytes": 2 * n, "us": t * 1e6, "tbs": 2 * n / t / 1e12, "ref": "copy"}]
    del src, dst
    torch.cuda.empty_cache()
    g = torch.Generator(device="cuda").manual_seed(0)
    B, D = 8, 4096 * 3072
    x, v, e = (torch.randn((B, D), device="cuda", generator=g).to(torch.bfloat16) for _ in range(3))
    xn = torch.empty_like(x)
    lp = torch.empty(B, dtype=torch.float64, device="cuda")
    ws = api.workspace(api.sde_workspace_size(B, D))
    t = timed(lambda: api.sde_step(x, v, e, xn, 0.6, 0.5, 0.9, logp=lp, ws=ws), "sde_step")
    kern.append({"what": "sde_step (x, v, eps read, x' written), 8 x 12.58 M bf16", "bytes": 8 * B * D, "us": t * 1e6,
                 "tbs": 8 * B * D / t / 1e12, "ref": "copy"})
    del x, v, e, xn
    torch.cuda.empty_cache()
    R, H = 32768, 3072
    X = torch.randn((R, H), device="cuda", generator=g).to(torch.bfloat16)
    Y = torch.empty_like(X)
    mod = torch.randn((8, 6 * H), device="cuda", generator=g)
    t = timed(lambda: api.norm_modulate(X, Y, shift=mod, scale=mod[:, H:], mod_ld=6 * H, rows_per_sample=R // 8),
              "norm_modulate")
    kern.append({"what": "norm_modulate (x read, y written), 32768 x 3072 bf16", "bytes": 4 * R * H, "us": t * 1e6,
                 "tbs": 4 * R * H / t / 1e12, "ref": "copy"})
    del X, Y
    cin = torch.randn((8, H), device="cuda", generator=g)
    Wm = (torch.randn((6 * H, H), device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    bm = torch.zeros(6 * H, device="cuda").to(torch.bfloat16)
    out = torch.empty((8, 6 * H), device="cuda")
    t = timed(lambda: api.skinny_linear(cin, Wm, bm, out, act_in=1), "skinny_linear")
    kern.append({"what": "skinny_linear (weights read), B = 8, 18432 x 3072 bf16", "bytes": 2 * 6 * H * H,
                 "us": t * 1e6, "tbs": 2 * 6 * H * H / t / 1e12, "ref": "read"})
    for k in kern:
        print(json.dumps(k), flush=True)
    out = _header(title, cmds)
    out += ["Streaming probes over 1 GiB (4x the 256 MB MALL; cold), median of %d launches timed with the "
            "library's HIP events; 16-byte accesses, four in flight per thread, 256-thread workgroups in a "
            "grid-stride loop. TB/s counts bytes read plus bytes written. Peak HBM 8 TB/s." % reps, "",
            "| probe | non-temporal | workgroups | µs | TB/s | / 8 TB/s |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {r['what']} | {'yes' if r['nt'] else 'no'} | {r['blocks']} | {r['us']:.1f} | {r['tbs']:.2f} | "
                   f"{r['tbs'] / 8.0:.2f} |")
    out += ["", "Best of each: " + ", ".join(f"{k} {v['tbs']:.2f} TB/s" for k, v in best.items()) + ".", "",
            "The rollout's HBM-bound kernels in the same process (algorithmic bytes only):", "",
            "| kernel | MB per launch | µs | TB/s | / 8 TB/s | / best probe of its kind |", "|---|---|---|---|---|---|"]
    for k in kern:
        ref = best[k["ref"]]["tbs"]
        out.append(f"| {k['what']} | {k['bytes'] / 1e6:.1f} | {k['us']:.1f} | {k['tbs']:.2f} | {k['tbs'] / 8.0:.2f} | "
                   f"{k['tbs'] / ref:.2f} ({k['ref']}) |")
    with open(out_md, "w") as f:
        f.write("\n".join(out) + "\n")
    return rows + kern


# ---------------------------------------------------------------------------- summaries
def _header(title: str, cmds: List[str]) -> List[str]:
    out = [f"# {title}", "", "Commands (run from the repository root on one MI355X):", "", "```"]
    out += cmds
    out += ["```", ""]
    return out


def stats_md(csv_path: str, out_md: str, title: str, cmds: List[str]) -> None:
    rows = list(csv.DictReader(open(csv_path)))
    out = _header(title, cmds)
    out += ["rocprofv3 kernel statistics (all launches of the run, warmup included):", "",
            "| kernel | calls | total ms | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['MinNs']) / 1e3:.1f} | "
                   f"{float(r['MaxNs']) / 1e3:.1f} | {float(r['Percentage']):.2f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(out) + "\n")


def _counter_per_kernel(path: str, counter: str) -> Dict[str, List[float]]:
    """Kernel name -> per-dispatch values (KiB) of `counter`, summed over a dispatch's rows."""
    per_dispatch: Dict[tuple, float] = defaultdict(float)
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        per_dispatch[(r["Kernel_Name"], int(r["Dispatch_Id"]))] += float(r["Counter_Value"])
    out: Dict[str, List[float]] = defaultdict(list)
    for (name, _), v in sorted(per_dispatch.items(), key=lambda kv: kv[0][1]):
        out[name].append(v)
    return out


def _copy_factor(path: str, counter: str, nbytes: int) -> float:
    """Bytes per counter unit: nbytes / the median counter of the copy kernel's dispatches."""
    vals = sorted(v for name, vs in _counter_per_kernel(path, counter).items() if "copy" in name.lower() for v in vs)
    if not vals:
        raise SystemExit(f"{path}: no {counter} values of a copy kernel")
    return nbytes / vals[len(vals) // 2]


def traffic_md(fetch_csv: str, write_csv: str, copy_fetch_csv: str, copy_write_csv: str, copy_bytes: int,
               keys: Dict[str, str], out_md: str, title: str, cmds: List[str], workload: str) -> dict:
    ff_ = _copy_factor(copy_fetch_csv, "FETCH_SIZE", copy_bytes)
    fw_ = _copy_factor(copy_write_csv, "WRITE_SIZE", copy_bytes)
    fetch = _counter_per_kernel(fetch_csv, "FETCH_SIZE")
    write = _counter_per_kernel(write_csv, "WRITE_SIZE")
    out = _header(title, cmds)
    out += [f"Copy calibration: a {copy_bytes} B device copy reads FETCH_SIZE = {copy_bytes / ff_ / 1024:.1f} KiB "
            f"and WRITE_SIZE = {copy_bytes / fw_ / 1024:.1f} KiB, so one counter KiB is {ff_:.1f} B fetched and "
            f"{fw_:.1f} B written.", "",
            "Per kernel, averaged over its launches (warmup included), scaled by those factors:", "",
            "| kernel | launches | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM read MB | HBM write MB | total MB / launch |",
            "|---|---|---|---|---|---|---|"]
    rows = []
    for name in sorted(set(fetch) | set(write), key=lambda n: -sum(fetch.get(n, [0.0]))):
        fv, wv = fetch.get(name, []), write.get(name, [])
        if not fv or not wv:
            continue
        af, aw = sum(fv) / len(fv), sum(wv) / len(wv)
        rb, wb = af * ff_, aw * fw_
        rows.append((name, len(fv), af, aw, rb, wb))
        out.append(f"| `{short_name(name)}` | {len(fv)} | {af:.0f} | {aw:.0f} | {rb / 1e6:.1f} | {wb / 1e6:.1f} | "
                   f"{(rb + wb) / 1e6:.1f} |")
    records = []
    for lib_name, pattern in keys.items():
        match = [r for r in rows if pattern in r[0]]
        if len(match) != 1:
            raise SystemExit(f"pattern {pattern!r} matches {len(match)} kernels")
        name, n, af, aw, rb, wb = match[0]
        records.append({"kernel": lib_name, "workload": workload, "rocprof_kernel": short_name(name), "launches": n,
                        "fetch_bytes_per_launch": rb, "write_bytes_per_launch": wb,
                        "traffic_bytes_per_launch": rb + wb, "copy_factor_fetch": ff_, "copy_factor_write": fw_,
                        "sources_sha256": sources_sha256(lib_name)})
    out += ["", "Traffic records read by bench.py (valid while the kernel's sources hash the same):", "",
            "```json", json.dumps(records, indent=1), "```"]
    with open(out_md, "w") as f:
        f.write("\n".join(out) + "\n")
    return {"records": records}


def counter_md(csv_path: str, counters: List[str], out_md: str, title: str, cmds: List[str], note: str = "") -> None:
    """Counters of a rocprofv3 --pmc run (e.g. the derived MfmaUtil), per kernel: dispatches and, per
    counter, the mean over dispatches (the first counter also min and max)."""
    vals = {c: _counter_per_kernel(csv_path, c) for c in counters}
    first = vals[counters[0]]
    out = _header(title, cmds)
    if note:
        out += [note, ""]
    head = ["kernel", "dispatches", f"mean {counters[0]}", "min", "max"] + [f"mean {c}" for c in counters[1:]]
    out += ["| " + " | ".join(head) + " |", "|" + "---|" * len(head)]
    for name, v in sorted(first.items(), key=lambda kv: -sum(kv[1]) / max(len(kv[1]), 1)):
        cells = [f"`{short_name(name)}`", str(len(v)), f"{sum(v) / len(v):.1f}", f"{min(v):.1f}", f"{max(v):.1f}"]
        for c in counters[1:]:
            w = vals[c].get(name, [])
            cells.append(f"{sum(w) / len(w):.1f}" if w else "")
        out.append("| " + " | ".join(cells) + " |")
    with open(out_md, "w") as f:
        f.write("\n".join(out) + "\n")


def lookup_traffic(kernel: str, workload: str) -> Optional[dict]:
    """The committed traffic record of `kernel` on `workload` whose sources still hash the same, else None."""
    if not os.path.isdir(PROFILES):
        return None
    want = sources_sha256(kernel)
    for fn in sorted(os.listdir(PROFILES)):
        if not fn.endswith(".md"):
            continue
        text = open(os.path.join(PROFILES, fn)).read()
        for block in re.findall(r"```json\n(.*?)```", text, flags=re.S):
            try:
                recs = json.loads(block)
            except ValueError:
                continue
            for r in recs if isinstance(recs, list) else []:
                if r.get("kernel") == kernel and r.get("workload") == workload and r.get("sources_sha256") == want:
                    return dict(r, summary=os.path.join("profiles", fn))
    return None


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(prog="python -m paper_2602_12529_amd.profiling")
    sub = ap.add_subparsers(dest="action", required=True)
    c = sub.add_parser("copy")
    c.add_argument("--bytes", type=int, default=1 << 30)
    c.add_argument("--reps", type=int, default=4)
    li = sub.add_parser("linear")
    li.add_argument("--M", type=int, default=36864)
    li.add_argument("--N", type=int, default=12288)
    li.add_argument("--K", type=int, default=3072)
    li.add_argument("--precision", choices=["bf16", "fp8"], default="fp8")
    li.add_argument("--gelu", action="store_true")
    li.add_argument("--reps", type=int, default=20)
    sw = sub.add_parser("sde-sweep")
    sw.add_argument("out")
    sw.add_argument("--title", required=True)
    sw.add_argument("--cmd", action="append", required=True)
    sw.add_argument("--reps", type=int, default=20)
    ce = sub.add_parser("ceiling")
    ce.add_argument("out")
    ce.add_argument("--title", required=True)
    ce.add_argument("--cmd", action="append", required=True)
    ce.add_argument("--reps", type=int, default=10)
    cn = sub.add_parser("counter")
    cn.add_argument("csv")
    cn.add_argument("out")
    cn.add_argument("--counter", action="append", required=True)
    cn.add_argument("--title", required=True)
    cn.add_argument("--cmd", action="append", required=True)
    cn.add_argument("--note", default="")
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("out")
    s.add_argument("--title", required=True)
    s.add_argument("--cmd", action="append", required=True)
    t = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy_fetch", "copy_write"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--workload", required=True, help="workload name the records belong to")
    t.add_argument("--key", action="append", default=[], help="NAME=PATTERN")
    t.add_argument("out")
    t.add_argument("--title", required=True)
    t.add_argument("--cmd", action="append", required=True)
    a = ap.parse_args(argv)
    if a.action == "copy":
        run_copy(a.bytes, a.reps)
    elif a.action == "linear":
        run_linear(a.M, a.N, a.K, a.precision, a.gelu, a.reps)
    elif a.action == "sde-sweep":
        run_sde_sweep(a.out, a.title, a.cmd, a.reps)
    elif a.action == "ceiling":
        run_ceiling(a.out, a.title, a.cmd, a.reps)
    elif a.action == "counter":
        counter_md(a.csv, a.counter, a.out, a.title, a.cmd, a.note)
    elif a.action == "stats":
        stats_md(a.csv, a.out, a.title, a.cmd)
    else:
        keys = dict(kv.split("=", 1) for kv in a.key)
        traffic_md(a.fetch, a.write, a.copy_fetch, a.copy_write, a.copy_bytes, keys, a.out, a.title, a.cmd,
                   a.workload)
    return 0


if __name__ == "__main__":
    sys.exit(main())
