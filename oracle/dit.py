"""The DiT velocity field v_theta(x_t, c, t) of the rollout, float64, plain numpy.

The paper gives no architecture: it names FLUX.1-dev, Qwen-Image and WAN as
backbones (Sec. 4.1) and writes the velocity as v_theta(x_t, t) (Eq. 1) or
v_theta(x_t, c, t) (Eq. 2).  Everything below is the reading of the block
structure ("adaLN-modulated RMSNorm, QKV projection with 2D/3D RoPE, joint
text+image attention, gated MLP") used for both the oracle and the GPU path:

  Norm_RMS(x) = x / sqrt(mean(x^2) + eps);  Norm_LN(x) = (x - mean) / sqrt(var + eps)
  Mod(x; shift, scale) = Norm(x) * (1 + scale) + shift

  Dual-stream block, per stream s in {txt, img} with its own weights:
    (sh1, sc1, g1, sh2, sc2, g2) = split6(W_mod,s SiLU(c) + b)
    [Q K V]_s = Mod(X_s; sh1, sc1) W_qkv,s^T + b, split into heads of width d
    Q_s, K_s <- RoPE(RMSNorm_d(.) * w_{q,k,s})      (text tokens: position 0)
    O = softmax(Q K^T / sqrt(d)) V over the joint sequence [txt; img]
    X_s += g1 * (O_s W_o,s^T + b)
    X_s += g2 * (GELU_tanh(Mod(X_s; sh2, sc2) W_1,s^T + b) W_2,s^T + b)

  Single-stream block on X = [txt; img]:
    (sh, sc, g) = split3(W_mod SiLU(c) + b);  [QKV | U] = Mod(X; sh, sc) W_1^T + b
    X += g * ([O | GELU_tanh(U)] W_2^T + b)

  WAN block: LN modulation from E_block + e(t); self-attention with RMSNorm
  over the full width before 3D RoPE; cross-attention to the text context with
  an affine LN on the queries; GELU_tanh FFN.

Attention is the plain definition (scores materialised, then softmax), in
query-row chunks only to bound memory.  Matrix products use numpy matmul.
"""
from __future__ import annotations

import math

import numpy as np

MODEL_MMDIT = 0
MODEL_WAN = 1
IO_LATENT = 0
IO_HIDDEN = 1
NORM_RMS = 0
NORM_LN = 1


def f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------- elementwise

def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    """GELU, tanh approximation: x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x * x * x)))


def rms_norm(x, eps: float):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def layer_norm(x, eps: float):
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def norm(x, kind: int, eps: float):
    return rms_norm(x, eps) if kind == NORM_RMS else layer_norm(x, eps)


def modulate(xn, shift, scale):
    """xn * (1 + scale) + shift, with shift/scale [B, H] broadcast over tokens."""
    return xn * (1.0 + scale[:, None, :]) + shift[:, None, :]


def linear(x, W, name: str):
    return f64(x) @ f64(W[name + ".w"]).T + f64(W[name + ".b"])


# ----------------------------------------------------------------- positions

def grid_positions(grid) -> np.ndarray:
    """Integer (frame, row, col) of each latent token, row-major over the grid."""
    f, r, c = (int(g) for g in grid)
    n = np.arange(f * r * c, dtype=np.int64)
    return np.stack([n // (r * c), (n // c) % r, n % c], axis=1)


def rope_angles(positions: np.ndarray, axes, theta: float) -> np.ndarray:
    """Rotation angle of every adjacent pair (2i, 2i+1): [N, d/2].

    The head dimension is split into three axis bands of widths ``axes``; the
    pair i of band a turns by pos_a * theta^(-2i / axes[a]).
    """
    cols = []
    for a, width in enumerate(axes):
        if width % 2:
            raise ValueError("rope axis widths must be even")
        inv = theta ** (-np.arange(0, width, 2, dtype=np.float64) / width)
        cols.append(positions[:, a:a + 1].astype(np.float64) * inv[None, :])
    return np.concatenate(cols, axis=1)


def apply_rope(x, angles):
    """Rotate each adjacent pair (x_{2i}, x_{2i+1}) of the last axis by angles[..., i].

    x [..., N, d]; angles [N, d/2].
    """
    x = f64(x)
    x0 = x[..., 0::2]
    x1 = x[..., 1::2]
    cos = np.cos(angles)
    sin = np.sin(angles)
    out = np.empty_like(x)
    out[..., 0::2] = x0 * cos - x1 * sin
    out[..., 1::2] = x0 * sin + x1 * cos
    return out


# ----------------------------------------------------------------- attention

def attention(q, k, v, chunk: int = 256):
    """softmax(q k^T / sqrt(d)) v, non-causal, no mask.  q [..., Nq, d], k/v [..., Nk, d]."""
    q, k, v = f64(q), f64(k), f64(v)
    d = q.shape[-1]
    out = np.empty(q.shape[:-1] + (v.shape[-1],), dtype=np.float64)
    kt = np.swapaxes(k, -1, -2)
    for s in range(0, q.shape[-2], chunk):
        scores = (q[..., s:s + chunk, :] @ kt) / math.sqrt(d)
        scores = scores - scores.max(axis=-1, keepdims=True)
        p = np.exp(scores)
        p = p / p.sum(axis=-1, keepdims=True)
        out[..., s:s + chunk, :] = p @ v
    return out


def split_heads(x, heads: int):
    """[B, N, h*d] -> [B, h, N, d]."""
    B, N, HD = x.shape
    return x.reshape(B, N, heads, HD // heads).transpose(0, 2, 1, 3)


def merge_heads(x):
    """[B, h, N, d] -> [B, N, h*d]."""
    B, h, N, d = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, N, h * d)


# ----------------------------------------------------------------- embedders

def timestep_sinusoid(t, dim: int = 256):
    """[cos | sin] of 1000 t * 10000^(-j / (dim/2)), j = 0..dim/2-1: [B, dim]."""
    t = f64(t).reshape(-1)
    half = dim // 2
    freqs = 10000.0 ** (-np.arange(half, dtype=np.float64) / half)
    arg = 1000.0 * t[:, None] * freqs[None, :]
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=1)


def mlp2(x, W, p1: str, p2: str, act):
    return linear(act(linear(x, W, p1)), W, p2)


# ----------------------------------------------------------------- blocks

def _chunks(m, n: int):
    H = m.shape[-1] // n
    return [m[:, i * H:(i + 1) * H] for i in range(n)]


def dual_block(x_img, x_txt, c, W, i: int, cfg, img_angles):
    """One dual-stream (MMDiT) block; returns the updated (x_img, x_txt)."""
    h, eps, nk = cfg.heads, cfg.norm_eps, cfg.norm_kind
    xs = {"img": f64(x_img).copy(), "txt": f64(x_txt).copy()}
    mods, qs, ks, vs = {}, {}, {}, {}
    for s in ("txt", "img"):
        p = f"dual.{i}.{s}."
        mods[s] = _chunks(linear(silu(f64(c)), W, p + "mod"), 6)
        sh1, sc1 = mods[s][0], mods[s][1]
        y = modulate(norm(xs[s], nk, eps), sh1, sc1)
        qkv = linear(y, W, p + "qkv")
        H = qkv.shape[-1] // 3
        q = split_heads(qkv[..., :H], h)
        k = split_heads(qkv[..., H:2 * H], h)
        v = split_heads(qkv[..., 2 * H:], h)
        q = rms_norm(q, eps) * f64(W[p + "q_norm.w"])
        k = rms_norm(k, eps) * f64(W[p + "k_norm.w"])
        if s == "img":
            q = apply_rope(q, img_angles)
            k = apply_rope(k, img_angles)
        qs[s], ks[s], vs[s] = q, k, v
    n_txt = xs["txt"].shape[1]
    q = np.concatenate([qs["txt"], qs["img"]], axis=2)
    k = np.concatenate([ks["txt"], ks["img"]], axis=2)
    v = np.concatenate([vs["txt"], vs["img"]], axis=2)
    o = merge_heads(attention(q, k, v))
    outs = {"txt": o[:, :n_txt], "img": o[:, n_txt:]}
    for s in ("txt", "img"):
        p = f"dual.{i}.{s}."
        _, _, g1, sh2, sc2, g2 = mods[s]
        xs[s] = xs[s] + g1[:, None, :] * linear(outs[s], W, p + "o")
        z = modulate(norm(xs[s], nk, eps), sh2, sc2)
        xs[s] = xs[s] + g2[:, None, :] * linear(gelu_tanh(linear(z, W, p + "mlp1")), W, p + "mlp2")
    return xs["img"], xs["txt"]


def single_block(x, c, W, j: int, cfg, n_txt: int, img_angles):
    """One single-stream block on the joint sequence x = [txt; img]."""
    h, eps, nk, F = cfg.heads, cfg.norm_eps, cfg.norm_kind, cfg.mlp_hidden
    x = f64(x)
    p = f"single.{j}."
    sh, sc, g = _chunks(linear(silu(f64(c)), W, p + "mod"), 3)
    y = modulate(norm(x, nk, eps), sh, sc)
    h1 = linear(y, W, p + "lin1")
    H = x.shape[-1]
    q = rms_norm(split_heads(h1[..., :H], h), eps) * f64(W[p + "q_norm.w"])
    k = rms_norm(split_heads(h1[..., H:2 * H], h), eps) * f64(W[p + "k_norm.w"])
    v = split_heads(h1[..., 2 * H:3 * H], h)
    q = np.concatenate([q[:, :, :n_txt], apply_rope(q[:, :, n_txt:], img_angles)], axis=2)
    k = np.concatenate([k[:, :, :n_txt], apply_rope(k[:, :, n_txt:], img_angles)], axis=2)
    o = merge_heads(attention(q, k, v))
    u = gelu_tanh(h1[..., 3 * H:3 * H + F])
    return x + g[:, None, :] * linear(np.concatenate([o, u], axis=-1), W, p + "lin2")


def wan_block(x, ctx, e6, W, i: int, cfg, angles, rows=None):
    """One WAN block.  x [B, N, H]; ctx [B, N_txt, H]; e6 [B, 6, H] time modulation.

    With ``rows`` (token indices) the keys and values of the self-attention are still taken
    over all N tokens, but only the listed query rows are carried through the block: the
    result is x_out[:, rows], the same values as those rows of the whole block (every other
    step is row-local), at a fraction of the cost on long sequences.
    """
    h, eps = cfg.heads, cfg.norm_eps
    x = f64(x)
    p = f"wan.{i}."
    sel = slice(None) if rows is None else np.asarray(rows, dtype=np.int64)
    mod = f64(W[p + "mod"])[None, :, :] + f64(e6)
    sh1, sc1, g1, sh2, sc2, g2 = (mod[:, n, :] for n in range(6))
    y = modulate(layer_norm(x, eps), sh1, sc1)
    qkv = linear(y, W, p + "sa.qkv")
    H = x.shape[-1]
    q = rms_norm(qkv[..., :H], eps) * f64(W[p + "sa.q_norm.w"])
    k = rms_norm(qkv[..., H:2 * H], eps) * f64(W[p + "sa.k_norm.w"])
    v = qkv[..., 2 * H:]
    q = apply_rope(split_heads(q, h), angles)[:, :, sel]
    k = apply_rope(split_heads(k, h), angles)
    o = merge_heads(attention(q, k, split_heads(v, h)))
    x = x[:, sel] + g1[:, None, :] * linear(o, W, p + "sa.o")
    y = layer_norm(x, eps) * f64(W[p + "ca.norm.w"]) + f64(W[p + "ca.norm.b"])
    q = rms_norm(linear(y, W, p + "ca.q"), eps) * f64(W[p + "ca.q_norm.w"])
    kv = linear(ctx, W, p + "ca.kv")
    k = rms_norm(kv[..., :H], eps) * f64(W[p + "ca.k_norm.w"])
    v = kv[..., H:]
    o = merge_heads(attention(split_heads(q, h), split_heads(k, h), split_heads(v, h)))
    x = x + linear(o, W, p + "ca.o")
    y = modulate(layer_norm(x, eps), sh2, sc2)
    return x + g2[:, None, :] * mlp2(y, W, p + "ffn1", p + "ffn2", gelu_tanh)


# ----------------------------------------------------------------- full forward

def final_layer(x_img, c, W, cfg):
    sh, sc = _chunks(linear(silu(f64(c)), W, "final.mod"), 2)
    return linear(modulate(norm(f64(x_img), cfg.norm_kind, cfg.norm_eps), sh, sc), W, "final.proj")


def forward(cfg, W, x, txt, t=None, cond=None, txt_index=None, grid=(1, 1, 1), rows=None):
    """v_theta for a batch.

    LATENT mode: x [B, N_img, C] latents, txt [P, N_txt, d_txt] prompt embeddings,
    t [B] times, cond [P, pooled_dim] pooled text (Flux) or None, txt_index [B]
    -> prompt row.  Returns v [B, N_img, C].

    HIDDEN mode (block stack only): x [B, N_img, H] image hidden, txt [B, N_txt, H]
    text hidden, cond [B, H] conditioning vector.  Returns (img_out, txt_out).

    ``rows`` (WAN with one block only): the velocity of the listed latent tokens,
    v[:, rows], computed with the block's sampled-row form.
    """
    x = f64(x)
    angles = rope_angles(grid_positions(grid), cfg.rope_axes, cfg.rope_theta)
    latent = cfg.io_mode == IO_LATENT
    B = x.shape[0]
    if txt_index is None:
        txt_index = np.arange(B)
    txt_index = np.asarray(txt_index, dtype=np.int64)

    if cfg.model == MODEL_MMDIT:
        if rows is not None:
            raise ValueError("sampled rows are implemented for the one-block WAN model only")
        if latent:
            c = mlp2(timestep_sinusoid(t), W, "temb.fc1", "temb.fc2", silu)
            if cfg.pooled_dim:
                c = c + mlp2(f64(cond)[txt_index], W, "pooled.fc1", "pooled.fc2", silu)
            x_img = linear(x, W, "x_in")
            x_txt = linear(txt, W, "txt_in")[txt_index]
        else:
            c = f64(cond)
            x_img, x_txt = x, f64(txt)
        for i in range(cfg.n_dual):
            x_img, x_txt = dual_block(x_img, x_txt, c, W, i, cfg, angles)
        if cfg.n_single:
            n_txt = x_txt.shape[1]
            xj = np.concatenate([x_txt, x_img], axis=1)
            for j in range(cfg.n_single):
                xj = single_block(xj, c, W, j, cfg, n_txt, angles)
            x_txt, x_img = xj[:, :n_txt], xj[:, n_txt:]
        if latent:
            return final_layer(x_img, c, W, cfg)
        return x_img, x_txt

    if cfg.model == MODEL_WAN:
        if not latent:
            raise ValueError("the WAN model runs in latent mode only")
        temb = mlp2(timestep_sinusoid(t), W, "temb.fc1", "temb.fc2", silu)
        e6 = linear(silu(temb), W, "temb.proj").reshape(B, 6, -1)
        ctx = mlp2(txt, W, "txt_in.fc1", "txt_in.fc2", gelu_tanh)[txt_index]
        xh = linear(x, W, "x_in")
        if rows is not None:
            if cfg.n_wan != 1:
                raise ValueError("sampled rows need a one-block WAN model")
            return final_layer(wan_block(xh, ctx, e6, W, 0, cfg, angles, rows=rows), temb, W, cfg)
        for i in range(cfg.n_wan):
            xh = wan_block(xh, ctx, e6, W, i, cfg, angles)
        return final_layer(xh, temb, W, cfg)
    raise ValueError(cfg.model)
