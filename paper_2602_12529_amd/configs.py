"""Model and workload shapes for the Flow-GRPO rollout of a flow-matching DiT.

These are plain shape descriptions (no arithmetic of the method).  They are
shared by the seeded input generator, the C-ABI binding, the tests and the
benchmark.  The oracle receives these objects duck-typed (attribute access
only) and never imports this module.

The paper names FLUX.1-dev, Qwen-Image and WAN as supported backbones
(Experimental Setup, Sec. 4.1) but gives no architecture; the block
structure (adaLN-modulated RMSNorm, QKV with 2D/3D RoPE, joint text+image
attention, adaLN-gated GELU MLP) is the reading used throughout.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional, Tuple

# Model kinds: a stack of dual-stream (MMDiT) blocks followed by optional
# single-stream blocks (Flux, Qwen-Image), or a WAN-style video DiT.
MODEL_MMDIT = 0
MODEL_WAN = 1

# Input/output modes of the DiT forward.
IO_LATENT = 0   # x is a latent [B, N_img, C]; v is [B, N_img, C]
IO_HIDDEN = 1   # x is the image-stream hidden [B, N_img, H]; v is the block stack's image output

NORM_RMS = 0
NORM_LN = 1

F32 = 0
BF16 = 1


@dataclass(frozen=True)
class ModelConfig:
    model: int = MODEL_MMDIT
    io_mode: int = IO_LATENT
    dtype: int = F32
    n_dual: int = 0
    n_single: int = 0
    n_wan: int = 0
    hidden: int = 64
    heads: int = 4
    head_dim: int = 16
    mlp_hidden: int = 256
    in_channels: int = 16
    txt_dim: int = 64
    pooled_dim: int = 0
    norm_kind: int = NORM_RMS
    rope_axes: Tuple[int, int, int] = (4, 6, 6)
    rope_theta: float = 10000.0
    norm_eps: float = 1e-6

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


@dataclass(frozen=True)
class Workload:
    """One rollout workload: the model, the batch and the SDE schedule."""
    name: str
    index: int                      # seed = 1000 + index
    model: ModelConfig
    prompts: int                    # P
    group: int                      # G samples per prompt; B = P * G
    grid: Tuple[int, int, int]      # (frames, rows, cols) of latent tokens; N_img = product
    n_txt: int
    steps: int                      # K
    eta: float = 0.7
    sde_steps: Optional[Tuple[int, ...]] = None   # 0-indexed SDE steps; None = all
    dynamics: str = "flow"          # sigma schedule of Table 1: "flow" (Flow-SDE), "dance" (Dance-SDE), "ode"
    reward_kind: str = "uniform"    # "uniform" U(0,1) or "normal" N(0,1)
    n_rewards: int = 1
    # A single fixed step (t, t_next) instead of the uniform grid (one-block workloads).
    fixed_step: Optional[Tuple[float, float]] = None

    @property
    def batch(self) -> int:
        return self.prompts * self.group

    @property
    def n_img(self) -> int:
        f, r, c = self.grid
        return f * r * c

    @property
    def latent_dim(self) -> int:
        """Elements of one sample's latent: D of the SDE step."""
        m = self.model
        width = m.hidden if m.io_mode == IO_HIDDEN else m.in_channels
        return self.n_img * width


TINY = Workload(
    name="tiny-fp32-2dual-h64",
    index=0,
    model=ModelConfig(model=MODEL_MMDIT, io_mode=IO_LATENT, dtype=F32, n_dual=2, n_single=0,
                      hidden=64, heads=4, head_dim=16, mlp_hidden=256, in_channels=16, txt_dim=64,
                      rope_axes=(4, 6, 6)),
    prompts=2, group=4, grid=(1, 4, 4), n_txt=8, steps=4, eta=0.7, reward_kind="uniform",
)

FLUX_BLOCK = Workload(
    name="flux-dual-block-bf16-B8-4096img-512txt",
    index=1,
    model=ModelConfig(model=MODEL_MMDIT, io_mode=IO_HIDDEN, dtype=BF16, n_dual=1, n_single=0,
                      hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, in_channels=64,
                      txt_dim=3072, rope_axes=(16, 56, 56)),
    prompts=1, group=8, grid=(1, 64, 64), n_txt=512, steps=1, eta=0.7,
    reward_kind="uniform", fixed_step=(0.6, 0.5),
)

FLUX_STACK = Workload(
    name="flux-19dual-38single-bf16-B16-1024img-512txt",
    index=2,
    model=ModelConfig(model=MODEL_MMDIT, io_mode=IO_LATENT, dtype=BF16, n_dual=19, n_single=38,
                      hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, in_channels=64,
                      txt_dim=4096, pooled_dim=768, rope_axes=(16, 56, 56)),
    prompts=1, group=16, grid=(1, 32, 32), n_txt=512, steps=10, eta=0.7, reward_kind="normal",
)

# One dual-stream block of the Qwen-Image-shaped stack on its hidden state (B=8, 4096 image + 256
# text tokens, one SDE step): the block's GEMM, attention and norm launches have exactly the stack's
# shapes, so their per-launch counters stand for the stack's.
QWEN_BLOCK = Workload(
    name="qwen-dual-block-bf16-B8-4096img-256txt",
    index=5,
    model=ModelConfig(model=MODEL_MMDIT, io_mode=IO_HIDDEN, dtype=BF16, n_dual=1, n_single=0,
                      hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, in_channels=64,
                      txt_dim=3072, rope_axes=(16, 56, 56)),
    prompts=1, group=8, grid=(1, 64, 64), n_txt=256, steps=1, eta=0.7,
    reward_kind="uniform", fixed_step=(0.6, 0.5),
)

QWEN_STACK = Workload(
    name="qwen-60dual-bf16-B8-4096img-256txt",
    index=3,
    model=ModelConfig(model=MODEL_MMDIT, io_mode=IO_LATENT, dtype=BF16, n_dual=60, n_single=0,
                      hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, in_channels=64,
                      txt_dim=3584, rope_axes=(16, 56, 56)),
    prompts=1, group=8, grid=(1, 64, 64), n_txt=256, steps=10, eta=0.7, sde_steps=(1, 2, 3),
    reward_kind="uniform",
)

WAN_STACK = Workload(
    name="wan-30blocks-bf16-B1-32760tok-512txt",
    index=4,
    model=ModelConfig(model=MODEL_WAN, io_mode=IO_LATENT, dtype=BF16, n_wan=30, hidden=1536,
                      heads=12, head_dim=128, mlp_hidden=8960, in_channels=64, txt_dim=4096,
                      norm_kind=NORM_LN, rope_axes=(44, 42, 42)),
    prompts=1, group=1, grid=(21, 30, 52), n_txt=512, steps=8, eta=0.7, reward_kind="uniform",
)

WORKLOADS = (TINY, FLUX_BLOCK, FLUX_STACK, QWEN_STACK, WAN_STACK)
