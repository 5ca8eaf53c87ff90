"""Pins of the oracle's DiT pieces (CPU only).

Library routines (torch CPU float64 functional ops, scipy) and hand-derived
values pin the elementwise ops, norms, RoPE and attention; brute-force loops on
tiny inputs pin the wiring of the dual-stream block; zero-gate special cases
pin the residual structure of every block kind.  The full random-weight
forward has no pin beyond these (parity unpinned as a whole).
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import dit

from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import synth


def t64(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


# ----------------------------------------------------------------- elementwise / norms

def test_gelu_silu_match_torch():
    x = np.linspace(-8, 8, 2001)
    np.testing.assert_allclose(dit.gelu_tanh(x), Fn.gelu(t64(x), approximate="tanh").numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(dit.silu(x), Fn.silu(t64(x)).numpy(), rtol=1e-14, atol=1e-15)
    # odd-part identity of the tanh approximation: gelu(x) - gelu(-x) = x
    np.testing.assert_allclose(dit.gelu_tanh(x) - dit.gelu_tanh(-x), x, atol=1e-14)


def test_norms_match_torch_and_modulate_invariant():
    """P9: norms equal torch's; zero shift/scale leaves unit RMS (RMS) or mean 0 / var 1 (LN)."""
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 5, 48)) * 3 + 0.5
    eps = 1e-6
    np.testing.assert_allclose(dit.rms_norm(x, eps), Fn.rms_norm(t64(x), (48,), eps=eps).numpy(), rtol=1e-13)
    np.testing.assert_allclose(dit.layer_norm(x, eps), Fn.layer_norm(t64(x), (48,), eps=eps).numpy(), rtol=1e-12, atol=1e-13)
    z = np.zeros((2, 48))
    y = dit.modulate(dit.norm(x, dit.NORM_RMS, 0.0), z, z)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1.0, rtol=1e-13)
    y = dit.modulate(dit.norm(x, dit.NORM_LN, 0.0), z, z)
    np.testing.assert_allclose(y.mean(-1), 0.0, atol=1e-13)
    np.testing.assert_allclose(y.var(-1), 1.0, rtol=1e-13)
    sh, sc = rng.standard_normal((2, 2, 48))
    xn = dit.norm(x, dit.NORM_RMS, eps)
    np.testing.assert_allclose(dit.modulate(xn, sh, sc)[1, 3], xn[1, 3] * (1 + sc[1]) + sh[1], rtol=1e-15)


def test_timestep_sinusoid_hand_values():
    e = dit.timestep_sinusoid(np.array([0.0, 0.25]))
    np.testing.assert_array_equal(e[0, :128], 1.0)
    np.testing.assert_array_equal(e[0, 128:], 0.0)
    assert e[1, 0] == pytest.approx(math.cos(250.0), abs=1e-12)     # j=0: frequency 1
    assert e[1, 128 + 64] == pytest.approx(math.sin(2.5), abs=1e-12)  # j=64: 10000^(-1/2)
    np.testing.assert_allclose(e[:, :128] ** 2 + e[:, 128:] ** 2, 1.0, rtol=1e-14)


# ----------------------------------------------------------------- RoPE

def test_grid_positions_hand():
    p = dit.grid_positions((2, 2, 3))
    assert p.tolist()[:7] == [[0, 0, 0], [0, 0, 1], [0, 0, 2], [0, 1, 0], [0, 1, 1], [0, 1, 2], [1, 0, 0]]
    assert p.tolist()[-1] == [1, 1, 2]


def test_rope_angles_hand_values():
    pos = np.array([[3, 5, 7]])
    a = dit.rope_angles(pos, (2, 4, 2), 10000.0)
    # band widths 2, 4, 2 -> pairs: (f, freq 1), (r, 1), (r, 10000^(-1/2)), (c, 1)
    np.testing.assert_allclose(a[0], [3.0, 5.0, 5.0 / 100.0, 7.0], rtol=1e-15)


def test_rope_is_complex_rotation_and_invariants():
    """P8: rotation of z = x_2i + i x_2i+1 by e^{i angle}; identity at position 0; norms kept; relative."""
    rng = np.random.default_rng(1)
    axes, d, N = (4, 6, 6), 16, 12
    pos = rng.integers(0, 9, size=(N, 3))
    ang = dit.rope_angles(pos, axes, 10000.0)
    x = rng.standard_normal((3, N, d))
    y = dit.apply_rope(x, ang)
    z = (x[..., 0::2] + 1j * x[..., 1::2]) * np.exp(1j * ang)
    np.testing.assert_allclose(y[..., 0::2], z.real, atol=1e-14)
    np.testing.assert_allclose(y[..., 1::2], z.imag, atol=1e-14)
    zero = dit.rope_angles(np.zeros((N, 3), dtype=int), axes, 10000.0)
    np.testing.assert_array_equal(dit.apply_rope(x, zero), x)
    np.testing.assert_allclose(np.hypot(y[..., 0::2], y[..., 1::2]), np.hypot(x[..., 0::2], x[..., 1::2]), rtol=1e-13)
    # <R_m q, R_n k> depends only on m - n (shift all positions by the same offset)
    q, k = rng.standard_normal((2, d))
    p1 = np.array([[1, 2, 3], [4, 0, 5]])
    p2 = p1 + np.array([[2, 7, 1]])
    a1, a2 = dit.rope_angles(p1, axes, 1e4), dit.rope_angles(p2, axes, 1e4)
    s1 = dit.apply_rope(q[None], a1[:1])[0] @ dit.apply_rope(k[None], a1[1:])[0]
    s2 = dit.apply_rope(q[None], a2[:1])[0] @ dit.apply_rope(k[None], a2[1:])[0]
    assert s1 == pytest.approx(s2, abs=1e-12)


# ----------------------------------------------------------------- attention

def _attention_loops(q, k, v):
    Nq, d = q.shape
    out = np.zeros((Nq, v.shape[1]))
    for i in range(Nq):
        w = [math.exp(sum(q[i, c] * k[j, c] for c in range(d)) / math.sqrt(d)) for j in range(k.shape[0])]
        tot = sum(w)
        for j in range(k.shape[0]):
            out[i] += w[j] / tot * v[j]
    return out


def test_attention_brute_force_and_library():
    """P7: brute force on tiny inputs; torch's SDPA (float64, math path); invariants."""
    rng = np.random.default_rng(2)
    q, k, v = rng.standard_normal((3, 2, 3, 19, 16))
    got = dit.attention(q, k, v, chunk=5)
    np.testing.assert_allclose(got[1, 2], _attention_loops(q[1, 2], k[1, 2], v[1, 2]), rtol=1e-12, atol=1e-13)
    ref = Fn.scaled_dot_product_attention(t64(q), t64(k), t64(v)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)
    perm = rng.permutation(19)
    np.testing.assert_allclose(dit.attention(q, k[..., perm, :], v[..., perm, :]), got, atol=1e-13)
    vu = np.broadcast_to(rng.standard_normal(16), v.shape)
    np.testing.assert_allclose(dit.attention(q, k, vu), vu, atol=1e-13)


# ----------------------------------------------------------------- blocks

def _tiny_cfg(**kw):
    base = dict(model=C.MODEL_MMDIT, io_mode=C.IO_HIDDEN, dtype=C.F32, n_dual=1, hidden=16, heads=2,
                head_dim=8, mlp_hidden=24, rope_axes=(2, 2, 4))
    base.update(kw)
    return C.ModelConfig(**base)


def _weights(cfg, seed=0):
    rng = np.random.default_rng(seed)
    W = {}
    for name, shape, kind in synth.tensor_table(cfg):
        W[name] = rng.standard_normal(shape) * 0.3 + (1.0 if kind == "norm" else 0.0)
    return W


def _matvec(Wm, b, x):
    return [sum(Wm[r][j] * x[j] for j in range(len(x))) + b[r] for r in range(len(b))]


def _dual_block_loops(x_img, x_txt, c, W, cfg, grid):
    """The dual-stream block written token by token and head by head with scalar math."""
    H, h, d, eps = cfg.hidden, cfg.heads, cfg.head_dim, cfg.norm_eps
    gelu = lambda u: 0.5 * u * (1 + math.tanh(math.sqrt(2 / math.pi) * (u + 0.044715 * u ** 3)))
    fr, rr, cc = grid
    out_img, out_txt = np.array(x_img, dtype=float), np.array(x_txt, dtype=float)
    for b in range(x_img.shape[0]):
        sc_ = [cj / (1 + math.exp(-cj)) for cj in c[b]]
        streams = {"txt": [list(r) for r in x_txt[b]], "img": [list(r) for r in x_img[b]]}
        mod, toks = {}, []          # toks: joint sequence entries (stream, index, q, k, v)
        for s in ("txt", "img"):
            p = f"dual.0.{s}."
            m = _matvec(W[p + "mod.w"], W[p + "mod.b"], sc_)
            mod[s] = [m[i * H:(i + 1) * H] for i in range(6)]
            for n, row in enumerate(streams[s]):
                rms = math.sqrt(sum(e * e for e in row) / H + eps)
                y = [row[j] / rms * (1 + mod[s][1][j]) + mod[s][0][j] for j in range(H)]
                qkv = _matvec(W[p + "qkv.w"], W[p + "qkv.b"], y)
                if s == "img":
                    pos = (n // (rr * cc), (n // cc) % rr, n % cc)
                else:
                    pos = (0, 0, 0)
                heads = []
                for hh in range(h):
                    qh = qkv[hh * d:(hh + 1) * d]
                    kh = qkv[H + hh * d:H + (hh + 1) * d]
                    vh = qkv[2 * H + hh * d:2 * H + (hh + 1) * d]
                    rq = math.sqrt(sum(e * e for e in qh) / d + eps)
                    rk = math.sqrt(sum(e * e for e in kh) / d + eps)
                    qh = [qh[i] / rq * W[p + "q_norm.w"][i] for i in range(d)]
                    kh = [kh[i] / rk * W[p + "k_norm.w"][i] for i in range(d)]
                    pair, start = 0, 0
                    for a, width in enumerate(cfg.rope_axes):
                        for i in range(width // 2):
                            ang = pos[a] * cfg.rope_theta ** (-2 * i / width)
                            j0 = 2 * pair
                            for vec in (qh, kh):
                                u0, u1 = vec[j0], vec[j0 + 1]
                                vec[j0] = u0 * math.cos(ang) - u1 * math.sin(ang)
                                vec[j0 + 1] = u0 * math.sin(ang) + u1 * math.cos(ang)
                            pair += 1
                    heads.append((qh, kh, vh))
                toks.append((s, n, heads))
        attn = {"txt": [None] * len(streams["txt"]), "img": [None] * len(streams["img"])}
        for (s, n, heads) in toks:
            o = []
            for hh in range(h):
                qh = heads[hh][0]
                w = [math.exp(sum(qh[i] * t[2][hh][1][i] for i in range(d)) / math.sqrt(d)) for t in toks]
                tot = sum(w)
                for i in range(d):
                    o.append(sum(w[j] * toks[j][2][hh][2][i] for j in range(len(toks))) / tot)
            attn[s][n] = o
        for s, target in (("txt", out_txt), ("img", out_img)):
            p = f"dual.0.{s}."
            for n, row in enumerate(streams[s]):
                proj = _matvec(W[p + "o.w"], W[p + "o.b"], attn[s][n])
                row = [row[j] + mod[s][2][j] * proj[j] for j in range(H)]
                rms = math.sqrt(sum(e * e for e in row) / H + eps)
                z = [row[j] / rms * (1 + mod[s][4][j]) + mod[s][3][j] for j in range(H)]
                u = [gelu(e) for e in _matvec(W[p + "mlp1.w"], W[p + "mlp1.b"], z)]
                mlp = _matvec(W[p + "mlp2.w"], W[p + "mlp2.b"], u)
                target[b, n] = [row[j] + mod[s][5][j] * mlp[j] for j in range(H)]
    return out_img, out_txt


def test_dual_block_matches_scalar_loops():
    cfg = _tiny_cfg()
    W = _weights(cfg)
    rng = np.random.default_rng(3)
    grid = (1, 2, 3)
    x_img = rng.standard_normal((2, 6, 16))
    x_txt = rng.standard_normal((2, 3, 16))
    c = rng.standard_normal((2, 16))
    img, txt = dit.forward(cfg, W, x_img, x_txt, cond=c, grid=grid)
    ref_img, ref_txt = _dual_block_loops(x_img, x_txt, c, W, cfg, grid)
    np.testing.assert_allclose(img, ref_img, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(txt, ref_txt, rtol=1e-11, atol=1e-11)


def _zero_gates(W, prefix, H, gate_chunks, n_chunks):
    W[prefix + "mod.w"] = W[prefix + "mod.w"].copy()
    W[prefix + "mod.b"] = W[prefix + "mod.b"].copy()
    for g in gate_chunks:
        W[prefix + "mod.w"][g * H:(g + 1) * H] = 0.0
        W[prefix + "mod.b"][g * H:(g + 1) * H] = 0.0


def test_zero_gates_make_blocks_identity():
    """P10: with both adaLN gates zero a dual or single block is the identity on its streams."""
    cfg = _tiny_cfg(n_dual=2, n_single=2)
    W = _weights(cfg, 4)
    H = cfg.hidden
    for i in range(2):
        for s in ("img", "txt"):
            _zero_gates(W, f"dual.{i}.{s}.", H, (2, 5), 6)
        _zero_gates(W, f"single.{i}.", H, (2,), 3)
    rng = np.random.default_rng(5)
    x_img, x_txt = rng.standard_normal((2, 2, 6, 16))[:, :, :6], rng.standard_normal((2, 3, 16))
    x_img = x_img[0]
    img, txt = dit.forward(cfg, W, x_img, x_txt, cond=rng.standard_normal((2, 16)), grid=(1, 2, 3))
    np.testing.assert_allclose(img, x_img, atol=0)
    np.testing.assert_allclose(txt, x_txt, atol=0)
    # with the gates restored the blocks act
    W2 = _weights(cfg, 4)
    img2, _ = dit.forward(cfg, W2, x_img, x_txt, cond=rng.standard_normal((2, 16)), grid=(1, 2, 3))
    assert np.abs(img2 - x_img).max() > 1e-3


def test_wan_block_identity_with_zero_gates_and_cross_output():
    cfg = C.ModelConfig(model=C.MODEL_WAN, io_mode=C.IO_LATENT, dtype=C.F32, n_wan=1, hidden=16, heads=2,
                        head_dim=8, mlp_hidden=24, in_channels=4, txt_dim=8, norm_kind=C.NORM_LN,
                        rope_axes=(2, 2, 4))
    W = _weights(cfg, 6)
    H = cfg.hidden
    W["wan.0.mod"] = W["wan.0.mod"].copy()
    W["wan.0.mod"][[2, 5]] = 0.0
    e6 = np.random.default_rng(7).standard_normal((2, 6, H))
    e6[:, [2, 5]] = 0.0
    W["wan.0.ca.o.w"] = np.zeros_like(W["wan.0.ca.o.w"])
    W["wan.0.ca.o.b"] = np.zeros_like(W["wan.0.ca.o.b"])
    rng = np.random.default_rng(8)
    x = rng.standard_normal((2, 6, H))
    ctx = rng.standard_normal((2, 5, H))
    ang = dit.rope_angles(dit.grid_positions((1, 2, 3)), cfg.rope_axes, cfg.rope_theta)
    np.testing.assert_allclose(dit.wan_block(x, ctx, e6, W, 0, cfg, ang), x, atol=0)


def test_latent_forward_prompt_broadcast():
    """P13 (oracle side): samples sharing a prompt, latent and time get identical velocities."""
    cfg = _tiny_cfg(io_mode=C.IO_LATENT, in_channels=4, txt_dim=8)
    W = _weights(cfg, 9)
    rng = np.random.default_rng(10)
    x = rng.standard_normal((1, 6, 4)).repeat(4, axis=0)
    txt = rng.standard_normal((2, 3, 8))
    v = dit.forward(cfg, W, x, txt, t=np.full(4, 0.5), txt_index=[0, 1, 0, 1], grid=(1, 2, 3))
    np.testing.assert_array_equal(v[0], v[2])
    np.testing.assert_array_equal(v[1], v[3])
    assert np.abs(v[0] - v[1]).max() > 1e-6
