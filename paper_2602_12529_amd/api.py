"""Thin Python binding of libff.so over torch device tensors.

Argument marshalling only: every step runs in the library's HIP kernels.
torch supplies device memory (including the workspaces the library asks for)
and the current HIP stream.
"""
from __future__ import annotations

import ctypes
from ctypes import byref, c_double, c_int32, c_int64, c_size_t, c_void_p
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import _lib
from . import configs as C
from ._lib import FFError, check  # noqa: F401

EPI_BIAS, EPI_GELU, EPI_GATED = 0, 1, 2
ACT_NONE, ACT_SILU, ACT_GELU = 0, 1, 2


def load():
    return _lib.load()


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return c_void_p(t.data_ptr())


def _stream():
    return c_void_p(torch.cuda.current_stream().cuda_stream)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return C.BF16
    if t.dtype == torch.float32:
        return C.F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def torch_dtype(code: int):
    return torch.bfloat16 if code == C.BF16 else torch.float32


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ------------------------------------------------------------------ SDE step / log-prob

def _bd(t) -> tuple:
    """(B, D) of a [B, ...] tensor: samples, and elements per sample (also for B = 0)."""
    d = 1
    for n in t.shape[1:]:
        d *= int(n)
    return int(t.shape[0]), d


def sde_workspace_size(B: int, D: int) -> int:
    n = c_size_t()
    check(load().ff_sde_workspace_size(B, D, byref(n)), "ff_sde_workspace_size")
    return n.value


def sde_step(x, v, eps, x_next, t: float, t_next: float, sigma: float, logp=None, ws=None):
    B, D = _bd(x)
    if ws is None and logp is not None:
        ws = workspace(sde_workspace_size(B, D), x.device)
    check(load().ff_sde_step(_p(x), _p(v), _p(eps), _p(x_next), _p(logp), B, D, t, t_next, sigma,
                             dtype_code(x), _p(ws), ws.numel() if ws is not None else 0, _stream()),
          "ff_sde_step")


def logprob(x, v, x_next, logp, t: float, t_next: float, sigma: float, ws=None):
    B, D = _bd(x)
    if ws is None:
        ws = workspace(sde_workspace_size(B, D), x.device)
    check(load().ff_logprob(_p(x), _p(v), _p(x_next), _p(logp), B, D, t, t_next, sigma, dtype_code(x), _p(ws),
                            ws.numel(), _stream()), "ff_logprob")


def sde_step_noalloc(x, v, eps, x_next, t: float, t_next: float, sigma: float, logp=None):
    """ff_sde_step without a workspace: the library's own device scratch holds the partial sums."""
    B, D = _bd(x)
    check(load().ff_sde_step_noalloc(_p(x), _p(v), _p(eps), _p(x_next), _p(logp), B, D, t, t_next, sigma,
                                     dtype_code(x), _stream()), "ff_sde_step_noalloc")


def sde_step_philox(x, v, x_next, t: float, t_next: float, sigma: float, seed: int, step: int, logp=None, ws=None):
    """The SDE step with its noise drawn on the device (Philox4x32-10, Box-Muller)."""
    B, D = _bd(x)
    if ws is None and logp is not None:
        ws = workspace(sde_workspace_size(B, D), x.device)
    check(load().ff_sde_step_philox(_p(x), _p(v), _p(x_next), _p(logp), B, D, t, t_next, sigma, seed, step,
                                    dtype_code(x), _p(ws), ws.numel() if ws is not None else 0, _stream()),
          "ff_sde_step_philox")


def philox_normal(shape, seed: int, step: int, dtype=torch.float32, device="cuda"):
    """The noise of ff_sde_step_philox for a [B, ...] latent, materialised."""
    out = torch.empty(shape, dtype=dtype, device=device)
    B, D = _bd(out)
    check(load().ff_philox_normal(_p(out), B, D, seed, step, dtype_code(out), _stream()), "ff_philox_normal")
    return out


def philox4x32(n: int, ctr_base: int, c2: int, c3: int, key: int, device="cuda"):
    """Raw Philox4x32-10 words, int32 tensor [n, 4] holding the uint32 bit patterns."""
    out = torch.empty((n, 4), dtype=torch.int32, device=device)
    check(load().ff_philox4x32(_p(out), n, ctr_base, c2, c3, key, _stream()), "ff_philox4x32")
    return out


def group_advantage(rewards, weights, group_id, n_groups: int, mode: int = 0, eps: float = 1e-4, adv=None,
                    counts=None):
    N = rewards.shape[0]
    K = rewards.shape[1] if rewards.dim() == 2 else 1
    if adv is None:
        adv = torch.empty(N, dtype=torch.float32, device=rewards.device)
    check(load().ff_group_advantage(_p(rewards), _p(weights), _p(group_id), N, K, n_groups, mode, eps, _p(adv),
                                    _p(counts), _stream()), "ff_group_advantage")
    return adv


# ------------------------------------------------------------------ objectives that consume the rollout
def flow_noise(x0, eps, t, xt=None):
    """x_t = (1 - t) x0 + t eps per sample; t: float32 [B] on the device."""
    B, D = _bd(x0)
    if xt is None:
        xt = torch.empty_like(x0)
    check(load().ff_flow_noise(_p(x0), _p(eps), _p(t), _p(xt), B, D, dtype_code(x0), _stream()), "ff_flow_noise")
    return xt


def loss_workspace_size(B: int, D: int) -> int:
    n = c_size_t()
    check(load().ff_loss_workspace_size(B, D, byref(n)), "ff_loss_workspace_size")
    return n.value


def awm_loss(v, eps, x0, adv, per_sample=None, loss=None, ws=None):
    """Eq. 3; returns (per_sample float64 [B], loss float64 [1]) on the device."""
    B, D = _bd(v)
    per_sample = torch.empty(B, dtype=torch.float64, device=v.device) if per_sample is None else per_sample
    loss = torch.empty(1, dtype=torch.float64, device=v.device) if loss is None else loss
    ws = workspace(loss_workspace_size(B, D), v.device) if ws is None else ws
    check(load().ff_awm_loss(_p(v), _p(eps), _p(x0), _p(adv), B, D, dtype_code(v), _p(per_sample), _p(loss), _p(ws),
                             ws.numel(), _stream()), "ff_awm_loss")
    return per_sample, loss


def nft_loss(v_pos, v_neg, eps, x0, r, per_sample=None, loss=None, ws=None):
    """Eq. 2; returns (per_sample float64 [B], loss float64 [1]) on the device."""
    B, D = _bd(v_pos)
    per_sample = torch.empty(B, dtype=torch.float64, device=v_pos.device) if per_sample is None else per_sample
    loss = torch.empty(1, dtype=torch.float64, device=v_pos.device) if loss is None else loss
    ws = workspace(loss_workspace_size(B, D), v_pos.device) if ws is None else ws
    check(load().ff_nft_loss(_p(v_pos), _p(v_neg), _p(eps), _p(x0), _p(r), B, D, dtype_code(v_pos), _p(per_sample),
                             _p(loss), _p(ws), ws.numel(), _stream()), "ff_nft_loss")
    return per_sample, loss


def grpo_loss(logp_new, logp_old, adv, step_w=None, clip_eps: float = 0.2, loss=None, n_clipped=None):
    """Clipped ratio objective over float64 [S, B] log-probs; returns (loss float64 [1], n_clipped int32 [1])."""
    S, B = logp_new.shape
    loss = torch.empty(1, dtype=torch.float64, device=logp_new.device) if loss is None else loss
    n_clipped = torch.empty(1, dtype=torch.int32, device=logp_new.device) if n_clipped is None else n_clipped
    check(load().ff_grpo_loss(_p(logp_new), _p(logp_old), _p(adv), _p(step_w), B, S, clip_eps, _p(loss),
                              _p(n_clipped), _stream()), "ff_grpo_loss")
    return loss, n_clipped


# ------------------------------------------------------------------ kernel-level ops
def linear_workspace_size() -> int:
    n = c_size_t()
    check(load().ff_linear_workspace_size(byref(n)), "ff_linear_workspace_size")
    return n.value


def linear(A, W, bias, out, epi=EPI_BIAS, gelu_from=0, gate=None, gate_ld=0, resid=None, rows_per_sample=0, ws=None):
    """ws: optional workspace (linear_workspace_size bytes) that lets the last round split along K."""
    M, K = A.shape
    N = W.shape[0]
    check(load().ff_linear(_p(A), A.stride(0), _p(W), _p(bias), _p(out), out.stride(0), M, N, K, epi, gelu_from,
                           _p(gate), gate_ld, _p(resid), resid.stride(0) if resid is not None else 0,
                           rows_per_sample, dtype_code(A), _p(ws), ws.numel() if ws is not None else 0, _stream()),
          "ff_linear")
    return out


def quantize_fp8(x, q=None, d=None):
    """Rows of x [R, C] (bf16 or f32) -> (E4M3 codes uint8 [R, C], float32 scales [R])."""
    R, Cn = x.shape
    if q is None:
        q = torch.empty((R, Cn), dtype=torch.uint8, device=x.device)
    if d is None:
        d = torch.empty((R,), dtype=torch.float32, device=x.device)
    check(load().ff_quantize_fp8(_p(x), x.stride(0), _p(q), q.stride(0), _p(d), R, Cn, dtype_code(x), _stream()),
          "ff_quantize_fp8")
    return q, d


def linear_fp8(A, d_a, W, d_w, bias, out, epi=EPI_BIAS, gelu_from=0):
    """out [M, N] bf16 = epi(d_a[m] d_w[n] (A W^T)[m, n] + bias) on E4M3 codes A [M, K], W [N, K]."""
    M, K = A.shape
    N = W.shape[0]
    check(load().ff_linear_fp8(_p(A), A.stride(0), _p(d_a), _p(W), W.stride(0), _p(d_w), _p(bias), _p(out),
                               out.stride(0), M, N, K, epi, gelu_from, _stream()), "ff_linear_fp8")
    return out


def stream_probe(mode: int, src, dst, nbytes: int, blocks: int, nontemporal: bool = True):
    """HBM streaming probe (0 read, 1 write, 2 copy) over nbytes; measurement only."""
    check(load().ff_stream_probe(mode, 1 if nontemporal else 0, _p(src), _p(dst), nbytes, blocks, _stream()),
          "ff_stream_probe")


def attention(Q, K, V, out):
    B, h, n_q, d = Q.shape
    n_kv = K.shape[2]
    check(load().ff_attention(_p(Q), _p(K), _p(V), _p(out), B, h, n_q, n_kv, d, dtype_code(Q), _stream()),
          "ff_attention")
    return out


def norm_modulate(x, y, shift=None, scale=None, mod_ld=0, rows_per_sample=0, norm_kind=C.NORM_RMS, eps=1e-6):
    rows, H = x.shape
    check(load().ff_norm_modulate(_p(x), _p(y), rows, H, _p(shift), _p(scale), mod_ld, rows_per_sample, norm_kind,
                                  eps, dtype_code(x), _stream()), "ff_norm_modulate")
    return y


def qk_norm_rope(qkv, heads, head_dim, q_w, k_w, Q, K, V, n_joint, tok_offset, rope=None, eps=1e-6):
    B, n_tok, _ = qkv.shape
    check(load().ff_qk_norm_rope(_p(qkv), B, n_tok, heads, head_dim, _p(q_w), _p(k_w), eps, _p(rope), _p(Q),
                                 _p(K), _p(V), n_joint, tok_offset, dtype_code(qkv), _stream()),
          "ff_qk_norm_rope")


def rope_table(grid: Sequence[int], head_dim: int, axes: Sequence[int], theta: float = 10000.0, device="cuda"):
    N = int(np.prod(grid))
    out = torch.empty((N, head_dim // 2, 2), dtype=torch.float32, device=device)
    g = (c_int32 * 3)(*grid)
    a = (c_int32 * 3)(*axes)
    check(load().ff_rope_table(_p(out), g, head_dim, a, theta, _stream()), "ff_rope_table")
    return out


def skinny_linear(inp, W, bias, out, act_in=ACT_NONE, act_out=ACT_NONE, classes=None):
    B, K = inp.shape
    N = W.shape[0]
    check(load().ff_skinny_linear(_p(inp), _p(W), _p(bias), _p(out), B, N, K, act_in, act_out, dtype_code(W),
                                  _p(classes), _stream()), "ff_skinny_linear")
    return out


def row_classes(c, out=None):
    """Classes of bitwise-equal rows of c (float32 [B, H]): the int32 map ff_row_classes documents."""
    B, H = c.shape
    if out is None:
        out = torch.empty(2 + 3 * B, dtype=torch.int32, device=c.device)
    check(load().ff_row_classes(_p(c), B, H, _p(out), _stream()), "ff_row_classes")
    return out


# ------------------------------------------------------------------ DiT
def dit_config(m: C.ModelConfig) -> _lib.DitConfig:
    c = _lib.DitConfig()
    for f in ("model", "io_mode", "dtype", "n_dual", "n_single", "n_wan", "hidden", "heads", "head_dim",
              "mlp_hidden", "in_channels", "txt_dim", "pooled_dim", "norm_kind"):
        setattr(c, f, int(getattr(m, f)))
    c.rope_axes = (c_int32 * 3)(*m.rope_axes)
    c.rope_theta = float(m.rope_theta)
    c.norm_eps = float(m.norm_eps)
    return c


def tensor_table(m: C.ModelConfig):
    """The library's parameter table: [(name, shape)] in ff_dit_tensor_info order."""
    lib = load()
    cfg = dit_config(m)
    n = c_int64()
    check(lib.ff_dit_num_tensors(byref(cfg), byref(n)), "ff_dit_num_tensors")
    out = []
    buf = ctypes.create_string_buffer(256)
    s0, s1 = c_int64(), c_int64()
    for i in range(n.value):
        check(lib.ff_dit_tensor_info(byref(cfg), i, buf, 256, byref(s0), byref(s1)), "ff_dit_tensor_info")
        out.append((buf.value.decode(), (s0.value,) if s1.value == 0 else (s0.value, s1.value)))
    return out


class Dit:
    """A model handle over caller-owned device weights (dict name -> tensor)."""

    def __init__(self, m: C.ModelConfig, weights: Dict[str, torch.Tensor]):
        self.cfg = m
        self._cfg = dit_config(m)
        self.weights = weights
        table = tensor_table(m)
        ptrs = (c_void_p * len(table))()
        for i, (name, shape) in enumerate(table):
            w = weights[name]
            if tuple(w.shape) != tuple(shape):
                raise ValueError(f"{name}: shape {tuple(w.shape)} != {shape}")
            if not w.is_contiguous() or w.dtype != torch_dtype(m.dtype):
                raise ValueError(f"{name}: must be contiguous {torch_dtype(m.dtype)}")
            ptrs[i] = w.data_ptr()
        h = c_void_p()
        check(load().ff_dit_create(byref(self._cfg), ptrs, len(table), byref(h)), "ff_dit_create")
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            try:
                load().ff_dit_destroy(h)
            except Exception:
                pass
            self._h = None

    def workspace_size(self, B: int, grid: Sequence[int], n_txt: int, n_prompts: int) -> int:
        n = c_size_t()
        g = (c_int32 * 3)(*grid)
        check(load().ff_dit_workspace_size(self._h, B, g, n_txt, n_prompts, byref(n)), "ff_dit_workspace_size")
        return n.value

    def forward(self, x, txt, grid, v_out, t=None, cond=None, txt_index=None, txt_out=None, ws=None):
        B = x.shape[0]
        n_txt = txt.shape[1]
        n_prompts = txt.shape[0]
        if ws is None:
            ws = workspace(self.workspace_size(B, grid, n_txt, n_prompts), x.device)
        g = (c_int32 * 3)(*grid)
        check(load().ff_dit_forward(self._h, _p(x), _p(txt), _p(txt_index), n_prompts, _p(cond), _p(t), g, B, n_txt,
                                    _p(v_out), _p(txt_out), _p(ws), ws.numel(), _stream()), "ff_dit_forward")
        return v_out

    # WAN: the per-block cross-attention K / V of a fixed text context, prepared once per rollout.
    def context_size(self, B: int, n_txt: int) -> int:
        n = c_size_t()
        check(load().ff_dit_context_size(self._h, B, n_txt, byref(n)), "ff_dit_context_size")
        return n.value

    def prepare_context(self, txt, grid, B, txt_index=None, ws=None, context=None):
        n_prompts, n_txt = txt.shape[0], txt.shape[1]
        if context is None:
            context = workspace(self.context_size(B, n_txt), txt.device)
        if ws is None:
            ws = workspace(self.workspace_size(B, grid, n_txt, n_prompts), txt.device)
        g = (c_int32 * 3)(*grid)
        check(load().ff_dit_prepare_context(self._h, _p(txt), _p(txt_index), n_prompts, g, B, n_txt, _p(context),
                                            context.numel(), _p(ws), ws.numel(), _stream()), "ff_dit_prepare_context")
        return context

    def forward_ctx(self, x, context, n_txt, grid, v_out, t, ws=None):
        B = x.shape[0]
        if ws is None:
            ws = workspace(self.workspace_size(B, grid, n_txt, 1), x.device)
        g = (c_int32 * 3)(*grid)
        check(load().ff_dit_forward_ctx(self._h, _p(x), _p(context), context.numel(), _p(t), g, B, n_txt, _p(v_out),
                                        _p(ws), ws.numel(), _stream()), "ff_dit_forward_ctx")
        return v_out


def upload_weights(w: C.Workload, device="cuda") -> Dict[str, torch.Tensor]:
    from . import synth
    dt = torch_dtype(w.model.dtype)
    return {name: torch.from_numpy(a).to(device=device).to(dt) for name, a in synth.iter_weights(w)}


# ------------------------------------------------------------------ profiling
def profile_enable(on: bool = True):
    check(load().ff_profile_enable(1 if on else 0), "ff_profile_enable")


def profile_filter(name: Optional[str] = None):
    """Time only the launches of kernel `name` (None: every kernel)."""
    check(load().ff_profile_filter(name.encode() if name else None), "ff_profile_filter")


def profile_reset():
    check(load().ff_profile_reset(), "ff_profile_reset")


def profile_read() -> Dict[str, dict]:
    lib = load()
    n = c_int32()
    check(lib.ff_profile_count(byref(n)), "ff_profile_count")
    out = {}
    buf = ctypes.create_string_buffer(128)
    launches, ms, fl, by = c_int64(), c_double(), c_double(), c_double()
    for i in range(n.value):
        check(lib.ff_profile_read(i, buf, 128, byref(launches), byref(ms), byref(fl), byref(by)), "ff_profile_read")
        out[buf.value.decode()] = {"launches": launches.value, "ms": ms.value, "flops": fl.value, "bytes": by.value}
    return out
