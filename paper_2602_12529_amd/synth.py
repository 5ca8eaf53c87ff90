"""Seeded synthetic inputs for the rollout workloads.

This module holds no arithmetic of the method: it only names the model's
parameter tensors, draws seeded random values for them and for the inputs
(prompt embeddings, initial noise, per-step SDE noise, rewards), and rounds
them to the storage dtype.  Both the oracle (via the tests and the CPU
baseline) and the GPU path consume exactly these values.

Seeding: every tensor or input stream gets its own numpy PCG64 generator,
keyed by ``SeedSequence(1000 + workload.index, spawn_key=(stream_id,))`` so any
tensor can be drawn without drawing the ones before it.

Distributions (the synthetic stand-in for the paper's FLUX.1-dev / PickScore
workload, whose data and weights are not available):
  * linear weights and biases: N(0, 0.02^2)
  * norm weights: 1 + N(0, 0.02^2)
  * prompt embeddings, conditioning vectors, x_0 and SDE noise: N(0, 1)
  * rewards: U(0, 1) or N(0, 1) per workload
bf16 workloads round every drawn value to bf16 (round to nearest even) once,
here, so both sides see identical bf16 values.
"""
from __future__ import annotations

from typing import Dict, Iterator, List, Tuple

import numpy as np

from . import configs as C

# Stream ids for the non-parameter inputs; parameters use ids 0..n_tensors-1.
_STREAM_TXT = 1 << 20
_STREAM_COND = (1 << 20) + 1
_STREAM_X0 = (1 << 20) + 2
_STREAM_REWARD = (1 << 20) + 3
_STREAM_EPS = 1 << 21          # + step index


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """The upper 16 bits of float32 values that are already bf16-representable."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


def _rng(workload_index: int, stream: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=1000 + workload_index, spawn_key=(stream,))
    return np.random.Generator(np.random.PCG64(ss))


# --------------------------------------------------------------------------
# Parameter table: names, shapes and init kinds, in a fixed order.
# kind: "w" = N(0, 0.02^2), "norm" = 1 + N(0, 0.02^2)
# --------------------------------------------------------------------------

def _lin(name: str, out_f: int, in_f: int) -> List[Tuple[str, Tuple[int, ...], str]]:
    return [(name + ".w", (out_f, in_f), "w"), (name + ".b", (out_f,), "w")]


def tensor_table(m: C.ModelConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    H, F, d = m.hidden, m.mlp_hidden, m.head_dim
    t: List[Tuple[str, Tuple[int, ...], str]] = []
    latent = m.io_mode == C.IO_LATENT
    if m.model == C.MODEL_MMDIT:
        if latent:
            t += _lin("temb.fc1", H, 256) + _lin("temb.fc2", H, H)
            if m.pooled_dim:
                t += _lin("pooled.fc1", H, m.pooled_dim) + _lin("pooled.fc2", H, H)
            t += _lin("x_in", H, m.in_channels) + _lin("txt_in", H, m.txt_dim)
        for i in range(m.n_dual):
            for s in ("img", "txt"):
                p = f"dual.{i}.{s}."
                t += _lin(p + "mod", 6 * H, H) + _lin(p + "qkv", 3 * H, H)
                t += [(p + "q_norm.w", (d,), "norm"), (p + "k_norm.w", (d,), "norm")]
                t += _lin(p + "o", H, H) + _lin(p + "mlp1", F, H) + _lin(p + "mlp2", H, F)
        for j in range(m.n_single):
            p = f"single.{j}."
            t += _lin(p + "mod", 3 * H, H) + _lin(p + "lin1", 3 * H + F, H)
            t += [(p + "q_norm.w", (d,), "norm"), (p + "k_norm.w", (d,), "norm")]
            t += _lin(p + "lin2", H, H + F)
        if latent:
            t += _lin("final.mod", 2 * H, H) + _lin("final.proj", m.in_channels, H)
    elif m.model == C.MODEL_WAN:
        if latent:
            t += _lin("temb.fc1", H, 256) + _lin("temb.fc2", H, H) + _lin("temb.proj", 6 * H, H)
            t += _lin("x_in", H, m.in_channels)
            t += _lin("txt_in.fc1", H, m.txt_dim) + _lin("txt_in.fc2", H, H)
        for i in range(m.n_wan):
            p = f"wan.{i}."
            t += [(p + "mod", (6, H), "w")]
            t += _lin(p + "sa.qkv", 3 * H, H)
            t += [(p + "sa.q_norm.w", (H,), "norm"), (p + "sa.k_norm.w", (H,), "norm")]
            t += _lin(p + "sa.o", H, H)
            t += [(p + "ca.norm.w", (H,), "norm"), (p + "ca.norm.b", (H,), "w")]
            t += _lin(p + "ca.q", H, H) + _lin(p + "ca.kv", 2 * H, H)
            t += [(p + "ca.q_norm.w", (H,), "norm"), (p + "ca.k_norm.w", (H,), "norm")]
            t += _lin(p + "ca.o", H, H) + _lin(p + "ffn1", F, H) + _lin(p + "ffn2", H, F)
        if latent:
            t += _lin("final.mod", 2 * H, H) + _lin("final.proj", m.in_channels, H)
    else:
        raise ValueError(f"unknown model kind {m.model}")
    return t


def _store(a: np.ndarray, dtype: int) -> np.ndarray:
    return bf16_round(a) if dtype == C.BF16 else a.astype(np.float32)


def iter_weights(w: C.Workload) -> Iterator[Tuple[str, np.ndarray]]:
    """Yield (name, float32 array holding storage-dtype values) in table order."""
    m = w.model
    for i, (name, shape, kind) in enumerate(tensor_table(m)):
        a = _rng(w.index, i).standard_normal(shape, dtype=np.float32) * np.float32(0.02)
        if kind == "norm":
            a = a + np.float32(1.0)
        yield name, _store(a, m.dtype)


def weights(w: C.Workload) -> Dict[str, np.ndarray]:
    return dict(iter_weights(w))


def _normal(w: C.Workload, stream: int, shape) -> np.ndarray:
    return _store(_rng(w.index, stream).standard_normal(shape, dtype=np.float32), w.model.dtype)


def text_input(w: C.Workload) -> np.ndarray:
    """LATENT: cached prompt embeddings [P, N_txt, txt_dim]; HIDDEN: text-stream hidden [B, N_txt, H]."""
    m = w.model
    if m.io_mode == C.IO_HIDDEN:
        return _normal(w, _STREAM_TXT, (w.batch, w.n_txt, m.hidden))
    return _normal(w, _STREAM_TXT, (w.prompts, w.n_txt, m.txt_dim))


def cond_input(w: C.Workload):
    """HIDDEN: the conditioning vector c [B, H]; LATENT: pooled text [P, pooled_dim] or None."""
    m = w.model
    if m.io_mode == C.IO_HIDDEN:
        return _normal(w, _STREAM_COND, (w.batch, m.hidden))
    if m.model == C.MODEL_MMDIT and m.pooled_dim:
        return _normal(w, _STREAM_COND, (w.prompts, m.pooled_dim))
    return None


def x0(w: C.Workload) -> np.ndarray:
    """Initial latent x at t = 1: [B, N_img, C] (LATENT) or the image hidden [B, N_img, H] (HIDDEN)."""
    m = w.model
    width = m.hidden if m.io_mode == C.IO_HIDDEN else m.in_channels
    return _normal(w, _STREAM_X0, (w.batch, w.n_img, width))


def sde_noise(w: C.Workload, step: int) -> np.ndarray:
    """The SDE noise eps_k of step k, same shape as x0."""
    m = w.model
    width = m.hidden if m.io_mode == C.IO_HIDDEN else m.in_channels
    return _normal(w, _STREAM_EPS + step, (w.batch, w.n_img, width))


def txt_index(w: C.Workload) -> np.ndarray:
    """Sample b belongs to prompt b // G (int32)."""
    return (np.arange(w.batch, dtype=np.int32) // np.int32(w.group)).astype(np.int32)


def rewards(w: C.Workload) -> np.ndarray:
    """Synthetic rewards [B, n_rewards] float32."""
    g = _rng(w.index, _STREAM_REWARD)
    shape = (w.batch, w.n_rewards)
    if w.reward_kind == "normal":
        return g.standard_normal(shape, dtype=np.float32)
    return g.random(shape, dtype=np.float32)


def normal(seed: int, shape, dtype: int = C.F32, scale: float = 1.0) -> np.ndarray:
    """Free-standing seeded N(0, scale^2) draw for tests (storage-dtype values)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy=seed)))
    return _store(g.standard_normal(shape, dtype=np.float32) * np.float32(scale), dtype)
