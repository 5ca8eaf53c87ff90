"""Pins of the oracle's single-stream block, WAN block, final layer and embedders (CPU only).

The paper gives no architecture (it names the backbones in Sec. 4.1 and writes the velocity
as v_theta(x_t, c, t), Eq. 1 / Eq. 2), so these functions follow the block reading that the
oracle's header states.  Each is restated here independently, token by token and head by
head in scalar Python, from that reading alone, and the oracle's vectorised numpy version must
agree with it on tiny random inputs.  To show that the comparison would catch the plausible
slips, each test also plants one such slip in a copy of the oracle function (a one-line source
mutation: text tokens rotated, the [O | GELU(U)] halves swapped, the K / V halves of the cross
projection swapped, shift and scale swapped, the time-modulation reshaped the wrong way, ...)
and requires the mutated oracle to disagree with the scalar restatement.
"""
import inspect
import math
import textwrap

import numpy as np
import pytest

from oracle import dit

from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import synth

EPS = 1e-6


# ----------------------------------------------------------------- scalar building blocks

def matvec(Wm, b, x):
    return [sum(Wm[r][j] * x[j] for j in range(len(x))) + b[r] for r in range(len(b))]


def lin(W, name, x):
    return matvec(W[name + ".w"], W[name + ".b"], x)


def silu(u):
    return u / (1.0 + math.exp(-u))


def gelu(u):
    return 0.5 * u * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u * u * u)))


def rmsn(v, eps=EPS):
    r = math.sqrt(sum(e * e for e in v) / len(v) + eps)
    return [e / r for e in v]


def lnorm(v, eps=EPS):
    mu = sum(v) / len(v)
    var = sum((e - mu) ** 2 for e in v) / len(v)
    return [(e - mu) / math.sqrt(var + eps) for e in v]


def modulate(xn, shift, scale):
    return [xn[j] * (1.0 + scale[j]) + shift[j] for j in range(len(xn))]


def token_pos(n, grid):
    """(frame, row, col) of latent token n in a row-major grid."""
    _, rr, cc = grid
    return (n // (rr * cc), (n // cc) % rr, n % cc)


def rotate(vec, pos, axes, theta):
    """Rotate the adjacent pairs of one head vector: band a of width axes[a] turns by pos[a] * theta^(-2i/width)."""
    out = list(vec)
    j = 0
    for a, width in enumerate(axes):
        for i in range(width // 2):
            ang = pos[a] * theta ** (-2.0 * i / width)
            u0, u1 = out[j], out[j + 1]
            out[j] = u0 * math.cos(ang) - u1 * math.sin(ang)
            out[j + 1] = u0 * math.sin(ang) + u1 * math.cos(ang)
            j += 2
    return out


def attend(q, keys, vals):
    """softmax over keys of q.k / sqrt(d), then the weighted sum of vals (one head, one query)."""
    d = len(q)
    s = [sum(q[i] * k[i] for i in range(d)) / math.sqrt(d) for k in keys]
    m = max(s)
    w = [math.exp(e - m) for e in s]
    tot = sum(w)
    return [sum(w[j] * vals[j][i] for j in range(len(vals))) / tot for i in range(len(vals[0]))]


def heads_of(v, h):
    d = len(v) // h
    return [v[i * d:(i + 1) * d] for i in range(h)]


def sinusoid(t):
    out = [math.cos(1000.0 * t * 10000.0 ** (-j / 128.0)) for j in range(128)]
    return out + [math.sin(1000.0 * t * 10000.0 ** (-j / 128.0)) for j in range(128)]


def to_np(rows):
    return np.array(rows, dtype=np.float64)


# ----------------------------------------------------------------- scalar restatements

def single_block_loops(x, c, W, j, cfg, n_txt, grid):
    """Single-stream block on the joint rows x [B][N][H] (text rows first)."""
    H, h, F = cfg.hidden, cfg.heads, cfg.mlp_hidden
    p = f"single.{j}."
    out = []
    for b in range(len(x)):
        mod = lin(W, p + "mod", [silu(e) for e in c[b]])
        shift, scale, gate = mod[:H], mod[H:2 * H], mod[2 * H:3 * H]
        qs, ks, vs, us = [], [], [], []
        for n, row in enumerate(x[b]):
            y = modulate(rmsn(row), shift, scale)
            z = lin(W, p + "lin1", y)
            pos = (0, 0, 0) if n < n_txt else token_pos(n - n_txt, grid)
            qh = [rmsn(v) for v in heads_of(z[:H], h)]
            kh = [rmsn(v) for v in heads_of(z[H:2 * H], h)]
            qh = [rotate([v[i] * W[p + "q_norm.w"][i] for i in range(len(v))], pos, cfg.rope_axes, cfg.rope_theta)
                  for v in qh]
            kh = [rotate([v[i] * W[p + "k_norm.w"][i] for i in range(len(v))], pos, cfg.rope_axes, cfg.rope_theta)
                  for v in kh]
            qs.append(qh)
            ks.append(kh)
            vs.append(heads_of(z[2 * H:3 * H], h))
            us.append([gelu(e) for e in z[3 * H:3 * H + F]])
        rows = []
        for n, row in enumerate(x[b]):
            o = []
            for hh in range(h):
                o += attend(qs[n][hh], [k[hh] for k in ks], [v[hh] for v in vs])
            proj = lin(W, p + "lin2", o + us[n])
            rows.append([row[i] + gate[i] * proj[i] for i in range(H)])
        out.append(rows)
    return out


def wan_block_loops(x, ctx, e6, W, i, cfg, grid):
    """WAN block on x [B][N][H] with text context ctx [B][N_t][H] and time modulation e6 [B][6][H]."""
    H, h = cfg.hidden, cfg.heads
    p = f"wan.{i}."
    out = []
    for b in range(len(x)):
        m = [[W[p + "mod"][r][col] + e6[b][r][col] for col in range(H)] for r in range(6)]
        sh1, sc1, g1, sh2, sc2, g2 = m
        qs, ks, vs = [], [], []
        for n, row in enumerate(x[b]):
            z = lin(W, p + "sa.qkv", modulate(lnorm(row), sh1, sc1))
            q = rmsn(z[:H])
            k = rmsn(z[H:2 * H])
            q = [q[e] * W[p + "sa.q_norm.w"][e] for e in range(H)]
            k = [k[e] * W[p + "sa.k_norm.w"][e] for e in range(H)]
            pos = token_pos(n, grid)
            qs.append([rotate(v, pos, cfg.rope_axes, cfg.rope_theta) for v in heads_of(q, h)])
            ks.append([rotate(v, pos, cfg.rope_axes, cfg.rope_theta) for v in heads_of(k, h)])
            vs.append(heads_of(z[2 * H:], h))
        ck, cv = [], []
        for row in ctx[b]:
            kv = lin(W, p + "ca.kv", row)
            kk = rmsn(kv[:H])
            ck.append(heads_of([kk[e] * W[p + "ca.k_norm.w"][e] for e in range(H)], h))
            cv.append(heads_of(kv[H:], h))
        rows = []
        for n, row in enumerate(x[b]):
            o = []
            for hh in range(h):
                o += attend(qs[n][hh], [k[hh] for k in ks], [v[hh] for v in vs])
            sa = lin(W, p + "sa.o", o)
            r1 = [row[e] + g1[e] * sa[e] for e in range(H)]
            yc = lnorm(r1)
            yc = [yc[e] * W[p + "ca.norm.w"][e] + W[p + "ca.norm.b"][e] for e in range(H)]
            qc = rmsn(lin(W, p + "ca.q", yc))
            qc = heads_of([qc[e] * W[p + "ca.q_norm.w"][e] for e in range(H)], h)
            oc = []
            for hh in range(h):
                oc += attend(qc[hh], [k[hh] for k in ck], [v[hh] for v in cv])
            ca = lin(W, p + "ca.o", oc)
            r2 = [r1[e] + ca[e] for e in range(H)]
            u = [gelu(e) for e in lin(W, p + "ffn1", modulate(lnorm(r2), sh2, sc2))]
            ff = lin(W, p + "ffn2", u)
            rows.append([r2[e] + g2[e] * ff[e] for e in range(H)])
        out.append(rows)
    return out


def final_layer_loops(x, c, W, cfg):
    H = cfg.hidden
    norm = rmsn if cfg.norm_kind == C.NORM_RMS else lnorm
    out = []
    for b in range(len(x)):
        mod = lin(W, "final.mod", [silu(e) for e in c[b]])
        shift, scale = mod[:H], mod[H:2 * H]
        out.append([lin(W, "final.proj", modulate(norm(row), shift, scale)) for row in x[b]])
    return out


def mmdit_latent_forward_loops(cfg, W, x, txt, t, pooled, tidx, grid):
    """Latent MMDiT: c = temb MLP + pooled MLP, x_in / txt_in embeddings with the prompt gather,
    the dual blocks (restated by test_oracle_dit's loops, reached through the oracle's vectorised
    dual block, which that file pins), the single blocks, then the final layer."""
    B = len(x)
    c = []
    for b in range(B):
        e = lin(W, "temb.fc2", [silu(u) for u in lin(W, "temb.fc1", sinusoid(t[b]))])
        if cfg.pooled_dim:
            pb = lin(W, "pooled.fc2", [silu(u) for u in lin(W, "pooled.fc1", list(pooled[tidx[b]]))])
            e = [e[i] + pb[i] for i in range(len(e))]
        c.append(e)
    x_img = [[lin(W, "x_in", list(row)) for row in x[b]] for b in range(B)]
    x_txt = [[lin(W, "txt_in", list(row)) for row in txt[tidx[b]]] for b in range(B)]
    img, tx = to_np(x_img), to_np(x_txt)
    ang = dit.rope_angles(dit.grid_positions(grid), cfg.rope_axes, cfg.rope_theta)
    for i in range(cfg.n_dual):
        img, tx = dit.dual_block(img, tx, to_np(c), W, i, cfg, ang)
    n_txt = tx.shape[1]
    joint = np.concatenate([tx, img], axis=1).tolist()
    for j in range(cfg.n_single):
        joint = single_block_loops(joint, c, W, j, cfg, n_txt, grid)
    img = [rows[n_txt:] for rows in joint]
    return to_np(final_layer_loops(img, c, W, cfg))


def wan_forward_loops(cfg, W, x, txt, t, tidx, grid):
    H = cfg.hidden
    B = len(x)
    temb, e6, ctx = [], [], []
    for b in range(B):
        e = lin(W, "temb.fc2", [silu(u) for u in lin(W, "temb.fc1", sinusoid(t[b]))])
        temb.append(e)
        pr = lin(W, "temb.proj", [silu(u) for u in e])
        e6.append([pr[r * H:(r + 1) * H] for r in range(6)])
        ctx.append([lin(W, "txt_in.fc2", [gelu(u) for u in lin(W, "txt_in.fc1", list(row))])
                    for row in txt[tidx[b]]])
    xh = [[lin(W, "x_in", list(row)) for row in x[b]] for b in range(B)]
    for i in range(cfg.n_wan):
        xh = wan_block_loops(xh, ctx, e6, W, i, cfg, grid)
    return to_np(final_layer_loops(xh, temb, W, cfg))


# ----------------------------------------------------------------- fixtures

def _weights(cfg, seed):
    rng = np.random.default_rng(seed)
    W = {}
    for name, shape, kind in synth.tensor_table(cfg):
        W[name] = rng.standard_normal(shape) * 0.3 + (1.0 if kind == "norm" else 0.0)
    return W


def _mmdit_cfg(**kw):
    base = dict(model=C.MODEL_MMDIT, io_mode=C.IO_LATENT, dtype=C.F32, n_dual=0, n_single=1, hidden=12, heads=2,
                head_dim=6, mlp_hidden=10, in_channels=3, txt_dim=5, pooled_dim=4, rope_axes=(2, 2, 2))
    base.update(kw)
    return C.ModelConfig(**base)


def _wan_cfg(**kw):
    base = dict(model=C.MODEL_WAN, io_mode=C.IO_LATENT, dtype=C.F32, n_wan=1, hidden=12, heads=2, head_dim=6,
                mlp_hidden=10, in_channels=3, txt_dim=5, norm_kind=C.NORM_LN, rope_axes=(2, 2, 2))
    base.update(kw)
    return C.ModelConfig(**base)


GRID = (2, 2, 2)     # 8 latent tokens: every axis band of the rotation takes two positions


def mutant(fn, old, new):
    """A copy of oracle function ``fn`` with one source fragment replaced (the planted slip)."""
    src = textwrap.dedent(inspect.getsource(fn))
    assert src.count(old) == 1, f"fragment not found once in {fn.__name__}: {old!r}"
    ns = dict(fn.__globals__)
    exec(compile(src.replace(old, new), f"<mutant of {fn.__name__}>", "exec"), ns)
    return ns[fn.__name__]


def _far(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) > 1e-6


# ----------------------------------------------------------------- single-stream block

def _single_case():
    cfg = _mmdit_cfg(io_mode=C.IO_HIDDEN, pooled_dim=0)
    W = _weights(cfg, 21)
    rng = np.random.default_rng(22)
    n_txt = 3
    x = rng.standard_normal((2, n_txt + 8, cfg.hidden))
    c = rng.standard_normal((2, cfg.hidden))
    ang = dit.rope_angles(dit.grid_positions(GRID), cfg.rope_axes, cfg.rope_theta)
    return cfg, W, x, c, n_txt, ang


def test_single_block_matches_scalar_loops():
    cfg, W, x, c, n_txt, ang = _single_case()
    got = dit.single_block(x, c, W, 0, cfg, n_txt, ang)
    ref = to_np(single_block_loops(x.tolist(), c.tolist(), W, 0, cfg, n_txt, GRID))
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


SINGLE_SLIPS = {
    # the text tokens rotated as if they were the first image tokens
    "text rotated": ("q[:, :, :n_txt], apply_rope", "apply_rope(q[:, :, :n_txt], img_angles[:n_txt]), apply_rope"),
    # [GELU(U) | O] into the second projection instead of [O | GELU(U)]
    "halves swapped": ("np.concatenate([o, u], axis=-1)", "np.concatenate([u, o], axis=-1)"),
    # the MLP input split off one head-block early
    "split column": ("h1[..., 3 * H:3 * H + F]", "h1[..., 3 * H - 2:3 * H + F - 2]"),
    # the gate taken from the first chunk of the modulation
    "gate chunk": ("sh, sc, g = _chunks", "g, sh, sc = _chunks"),
    # attention over the image tokens only
    "not joint": ("o = merge_heads(attention(q, k, v))",
                  "o = merge_heads(attention(q, k[:, :, n_txt:], v[:, :, n_txt:]))"),
}


@pytest.mark.parametrize("slip", list(SINGLE_SLIPS))
def test_single_block_planted_slip_is_caught(slip):
    cfg, W, x, c, n_txt, ang = _single_case()
    bad = mutant(dit.single_block, *SINGLE_SLIPS[slip])
    ref = to_np(single_block_loops(x.tolist(), c.tolist(), W, 0, cfg, n_txt, GRID))
    assert _far(bad(x, c, W, 0, cfg, n_txt, ang), ref)


# ----------------------------------------------------------------- WAN block

def _wan_case():
    cfg = _wan_cfg()
    W = _weights(cfg, 31)
    rng = np.random.default_rng(32)
    x = rng.standard_normal((2, 8, cfg.hidden))
    ctx = rng.standard_normal((2, 5, cfg.hidden))
    e6 = rng.standard_normal((2, 6, cfg.hidden))
    ang = dit.rope_angles(dit.grid_positions(GRID), cfg.rope_axes, cfg.rope_theta)
    return cfg, W, x, ctx, e6, ang


def test_wan_block_matches_scalar_loops():
    cfg, W, x, ctx, e6, ang = _wan_case()
    got = dit.wan_block(x, ctx, e6, W, 0, cfg, ang)
    ref = to_np(wan_block_loops(x.tolist(), ctx.tolist(), e6.tolist(), W, 0, cfg, GRID))
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


def test_wan_block_rows_match_full_block():
    """The oracle's sampled-row form of the block (all tokens' keys / values, the listed query
    rows only) equals those rows of the whole block."""
    cfg, W, x, ctx, e6, ang = _wan_case()
    full = dit.wan_block(x, ctx, e6, W, 0, cfg, ang)
    rows = np.array([7, 0, 3])
    np.testing.assert_allclose(dit.wan_block(x, ctx, e6, W, 0, cfg, ang, rows=rows), full[:, rows],
                               rtol=1e-13, atol=1e-13)


WAN_SLIPS = {
    # K and V halves of the cross-attention's context projection swapped
    "cross K/V swapped": ("k = rms_norm(kv[..., :H], eps) * f64(W[p + \"ca.k_norm.w\"])\n    v = kv[..., H:]",
                          "k = rms_norm(kv[..., H:], eps) * f64(W[p + \"ca.k_norm.w\"])\n    v = kv[..., :H]"),
    # the QK norm taken per head (width d) instead of over the full width H
    "per-head QK norm": ("q = rms_norm(qkv[..., :H], eps) * f64(W[p + \"sa.q_norm.w\"])",
                         "q = merge_heads(rms_norm(split_heads(qkv[..., :H], h), eps)) * f64(W[p + \"sa.q_norm.w\"])"),
    # no affine part on the LayerNorm before the cross-attention query
    "plain LN before ca.q": ("y = layer_norm(x, eps) * f64(W[p + \"ca.norm.w\"]) + f64(W[p + \"ca.norm.b\"])",
                             "y = layer_norm(x, eps)"),
    # the cross-attention residual gated like the self-attention one
    "gated cross residual": ("x = x + linear(o, W, p + \"ca.o\")", "x = x + g1[:, None, :] * linear(o, W, p + \"ca.o\")"),
    # the K RMSNorm of the text keys left out
    "no cross K norm": ("k = rms_norm(kv[..., :H], eps) * f64(W[p + \"ca.k_norm.w\"])",
                        "k = kv[..., :H] * f64(W[p + \"ca.k_norm.w\"])"),
    # shift and scale of the first modulation swapped
    "mod order": ("sh1, sc1, g1, sh2, sc2, g2 = (mod", "sc1, sh1, g1, sh2, sc2, g2 = (mod"),
    # the self-attention query rotated without its RMSNorm and weight
    "self Q unnormed": ("q = apply_rope(split_heads(q, h), angles)", "q = apply_rope(split_heads(qkv[..., :H], h), angles)"),
}


@pytest.mark.parametrize("slip", list(WAN_SLIPS))
def test_wan_block_planted_slip_is_caught(slip):
    cfg, W, x, ctx, e6, ang = _wan_case()
    bad = mutant(dit.wan_block, *WAN_SLIPS[slip])
    ref = to_np(wan_block_loops(x.tolist(), ctx.tolist(), e6.tolist(), W, 0, cfg, GRID))
    assert _far(bad(x, ctx, e6, W, 0, cfg, ang), ref)


# ----------------------------------------------------------------- final layer

@pytest.mark.parametrize("kind", [C.NORM_RMS, C.NORM_LN])
def test_final_layer_matches_scalar_loops(kind):
    cfg = _mmdit_cfg(norm_kind=kind)
    W = _weights(cfg, 41)
    rng = np.random.default_rng(42)
    x = rng.standard_normal((2, 5, cfg.hidden))
    c = rng.standard_normal((2, cfg.hidden))
    got = dit.final_layer(x, c, W, cfg)
    ref = to_np(final_layer_loops(x.tolist(), c.tolist(), W, cfg))
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    bad = mutant(dit.final_layer, "sh, sc = _chunks", "sc, sh = _chunks")
    assert _far(bad(x, c, W, cfg), ref)


# ----------------------------------------------------------------- embedders through the whole forward

def _mmdit_latent_case():
    cfg = _mmdit_cfg(n_dual=1, n_single=1)
    W = _weights(cfg, 51)
    rng = np.random.default_rng(52)
    x = rng.standard_normal((3, 8, cfg.in_channels))
    txt = rng.standard_normal((2, 3, cfg.txt_dim))
    pooled = rng.standard_normal((2, cfg.pooled_dim))
    t = np.array([0.9, 0.35, 0.6])
    tidx = np.array([1, 0, 1], dtype=np.int32)
    return cfg, W, x, txt, pooled, t, tidx


def test_mmdit_latent_forward_matches_scalar_loops():
    cfg, W, x, txt, pooled, t, tidx = _mmdit_latent_case()
    got = dit.forward(cfg, W, x, txt, t=t, cond=pooled, txt_index=tidx, grid=GRID)
    ref = mmdit_latent_forward_loops(cfg, W, x.tolist(), txt.tolist(), t.tolist(), pooled.tolist(), tidx.tolist(),
                                     GRID)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


MMDIT_EMBED_SLIPS = {
    "pooled not added": ("c = c + mlp2(f64(cond)[txt_index]", "c = 0 * c + mlp2(f64(cond)[txt_index]"),
    "pooled not gathered": ("mlp2(f64(cond)[txt_index]", "mlp2(f64(cond)[np.arange(B) % len(cond)]"),
    "text not gathered": ("x_txt = linear(txt, W, \"txt_in\")[txt_index]",
                          "x_txt = linear(txt, W, \"txt_in\")[np.arange(B) % len(txt)]"),
    "temb SiLU -> GELU": ("c = mlp2(timestep_sinusoid(t), W, \"temb.fc1\", \"temb.fc2\", silu)\n            if",
                          "c = mlp2(timestep_sinusoid(t), W, \"temb.fc1\", \"temb.fc2\", gelu_tanh)\n            if"),
}


@pytest.mark.parametrize("slip", list(MMDIT_EMBED_SLIPS))
def test_mmdit_latent_embedder_slip_is_caught(slip, monkeypatch):
    cfg, W, x, txt, pooled, t, tidx = _mmdit_latent_case()
    ref = mmdit_latent_forward_loops(cfg, W, x.tolist(), txt.tolist(), t.tolist(), pooled.tolist(), tidx.tolist(),
                                     GRID)
    bad = mutant(dit.forward, *MMDIT_EMBED_SLIPS[slip])
    assert _far(bad(cfg, W, x, txt, t=t, cond=pooled, txt_index=tidx, grid=GRID), ref)


def _wan_latent_case():
    cfg = _wan_cfg()
    W = _weights(cfg, 61)
    rng = np.random.default_rng(62)
    x = rng.standard_normal((3, 8, cfg.in_channels))
    txt = rng.standard_normal((2, 4, cfg.txt_dim))
    t = np.array([0.8, 0.25, 0.5])
    tidx = np.array([1, 1, 0], dtype=np.int32)
    return cfg, W, x, txt, t, tidx


def test_wan_latent_forward_matches_scalar_loops():
    cfg, W, x, txt, t, tidx = _wan_latent_case()
    got = dit.forward(cfg, W, x, txt, t=t, txt_index=tidx, grid=GRID)
    ref = wan_forward_loops(cfg, W, x.tolist(), txt.tolist(), t.tolist(), tidx.tolist(), GRID)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_wan_latent_forward_rows_match_full_forward():
    """The sampled-row form of the one-block WAN forward equals those rows of the whole forward."""
    cfg, W, x, txt, t, tidx = _wan_latent_case()
    full = dit.forward(cfg, W, x, txt, t=t, txt_index=tidx, grid=GRID)
    rows = np.array([1, 6, 2])
    part = dit.forward(cfg, W, x, txt, t=t, txt_index=tidx, grid=GRID, rows=rows)
    np.testing.assert_allclose(part, full[:, rows], rtol=1e-13, atol=1e-13)


WAN_EMBED_SLIPS = {
    # the time modulation reshaped as [B, H, 6] (then read as six [H] rows)
    "e6 reshape": ("e6 = linear(silu(temb), W, \"temb.proj\").reshape(B, 6, -1)",
                   "e6 = linear(silu(temb), W, \"temb.proj\").reshape(B, -1, 6).transpose(0, 2, 1)"),
    # the context MLP with SiLU instead of GELU
    "context activation": ("ctx = mlp2(txt, W, \"txt_in.fc1\", \"txt_in.fc2\", gelu_tanh)",
                           "ctx = mlp2(txt, W, \"txt_in.fc1\", \"txt_in.fc2\", silu)"),
    # the context not gathered by prompt index
    "context not gathered": ("gelu_tanh)[txt_index]", "gelu_tanh)[np.arange(B) % len(txt)]"),
    # the final layer modulated by SiLU(temb) projected through e6's weights
    "final from e6": ("return final_layer(xh, temb, W, cfg)", "return final_layer(xh, e6[:, 0], W, cfg)"),
}


@pytest.mark.parametrize("slip", list(WAN_EMBED_SLIPS))
def test_wan_latent_embedder_slip_is_caught(slip):
    cfg, W, x, txt, t, tidx = _wan_latent_case()
    ref = wan_forward_loops(cfg, W, x.tolist(), txt.tolist(), t.tolist(), tidx.tolist(), GRID)
    bad = mutant(dit.forward, *WAN_EMBED_SLIPS[slip])
    assert _far(bad(cfg, W, x, txt, t=t, txt_index=tidx, grid=GRID), ref)
