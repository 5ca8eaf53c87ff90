"""GPU parity of the kernel-level entry points (ff_ops.h) against the oracle's pieces.

Shapes span several tiles and ragged tails (M, N not multiples of the GEMM
tile; token counts not multiples of the attention tile).
"""
import math

import numpy as np
import pytest
import torch

from oracle import dit as odit
from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import synth

from gpu_util import TOL, check, dev, host, normal, rel, say

pytestmark = pytest.mark.gpu

LIN = [
    # M, N, K, dtype
    (256, 256, 64, C.BF16), (300, 200, 128, C.BF16), (1000, 520, 192, C.BF16), (77, 64, 3072, C.BF16),
    (513, 9216 // 8, 3072, C.BF16), (33, 20, 16, C.F32), (130, 70, 96, C.F32), (64, 256, 64, C.F32),
]


# Shapes with at least one 256 x 256 tile per CU: these take the large-tile kernel.
# (5000, 4000): 20 x 16 tiles, whole sixteens of tile columns (the XCD-blocked tile order) with a
# partial last group of tile rows and ragged edges.
LIN_LARGE = [(4133, 4133, 192, C.BF16), (8197, 2088, 128, C.BF16), (8200, 2100, 64, C.BF16),
             (5000, 4000, 128, C.BF16)]


@pytest.mark.parametrize("M,N,K,dt", LIN + LIN_LARGE)
@pytest.mark.parametrize("epi", ["bias", "gelu", "gelu_from", "gated"])
def test_linear_parity(gpu_lib, M, N, K, dt, epi):
    say("linear", M, N, K, dt, epi)
    a = normal(1, (M, K), dt)
    w = normal(2, (N, K), dt, 0.05)
    b = normal(3, (N,), dt, 0.1)
    rps = max(1, M // 3)
    nsamp = (M + rps - 1) // rps
    gate = normal(4, (nsamp, N), C.F32)
    resid = normal(5, (M, N), dt)
    A, W, Bv = dev(a, dt), dev(w, dt), dev(b, dt)
    out = torch.empty((M, N), dtype=A.dtype, device="cuda")
    z = odit.f64(a) @ odit.f64(w).T + odit.f64(b)
    kw = {}
    if epi == "bias":
        ref = z
        code = gpu_lib.EPI_BIAS
    elif epi in ("gelu", "gelu_from"):
        g0 = 0 if epi == "gelu" else N // 3
        ref = z.copy()
        ref[:, g0:] = odit.gelu_tanh(z[:, g0:])
        code = gpu_lib.EPI_GELU
        kw["gelu_from"] = g0
    else:
        G = dev(gate, C.F32)
        R = dev(resid, dt)
        kw.update(gate=G, gate_ld=N, resid=R, rows_per_sample=rps)
        ref = resid + gate[np.arange(M) // rps] * z
        code = gpu_lib.EPI_GATED
    gpu_lib.linear(A, W, Bv, out, epi=code, **kw)
    torch.cuda.synchronize()
    check(host(out), ref, dt, 0, K, what=f"linear {M}x{N}x{K} {epi}", norm_tol=2e-6 if dt == C.F32 else 6e-3)


# 256 x 256 tiles leaving a partly filled last round on 256 CUs, K of at least 96 slabs of 64:
# (17 x 16 = 272 tiles, tail 16, split in 8), (17 x 17 = 289, tail 33, split in 7), (33 x 9 = 297
# with ragged edges, tail 41, split in 6).
LIN_SPLIT = [(4352, 4096, 6144), (4352, 4352, 12288), (8200, 2100, 6144)]


@pytest.mark.parametrize("M,N,K", LIN_SPLIT)
@pytest.mark.parametrize("epi", ["bias", "gelu", "gated"])
def test_linear_split_k_tail(gpu_lib, M, N, K, epi):
    """With a workspace the last round's tiles are split along K and their float32 partial sums added
    in a fixed order: the result matches the oracle element-wise, repeats bit for bit, and differs
    (in rounding only) from the unsplit launch, which shows the split path ran."""
    assert torch.cuda.get_device_properties(0).multi_processor_count == 256
    say("linear split-K", M, N, K, epi)
    a = normal(70, (M, K), C.BF16)
    w = normal(71, (N, K), C.BF16, 0.05)
    b = normal(72, (N,), C.BF16, 0.1)
    A, W, Bv = dev(a, C.BF16), dev(w, C.BF16), dev(b, C.BF16)
    z = odit.f64(a) @ odit.f64(w).T + odit.f64(b)
    kw, code = {}, gpu_lib.EPI_BIAS
    if epi == "gelu":
        ref, code = odit.gelu_tanh(z), gpu_lib.EPI_GELU
    elif epi == "gated":
        rps = (M + 3) // 4
        gate = normal(73, (4, N), C.F32)
        resid = normal(74, (M, N), C.BF16)
        kw = dict(gate=dev(gate, C.F32), gate_ld=N, resid=dev(resid, C.BF16), rows_per_sample=rps)
        ref, code = resid + gate[np.arange(M) // rps] * z, gpu_lib.EPI_GATED
    else:
        ref = z
    ws = torch.empty(gpu_lib.linear_workspace_size(), dtype=torch.uint8, device="cuda")
    outs = []
    for use_ws in (True, True, False):
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        gpu_lib.linear(A, W, Bv, out, epi=code, ws=ws if use_ws else None, **kw)
        outs.append(out)
    torch.cuda.synchronize()
    check(host(outs[0]), ref, C.BF16, 0, K, what=f"linear split-K {M}x{N}x{K} {epi}", norm_tol=6e-3)
    assert torch.equal(outs[0], outs[1])
    assert not torch.equal(outs[0], outs[2])
    check(host(outs[2]), ref, C.BF16, 0, K, what=f"linear unsplit {M}x{N}x{K} {epi}", norm_tol=6e-3)


def test_linear_in_place_gated_residual(gpu_lib):
    M, N, K = 256, 384, 128
    a, w = normal(6, (M, K), C.BF16), normal(7, (N, K), C.BF16, 0.05)
    x = normal(8, (M, N), C.BF16)
    g = normal(9, (2, N), C.F32)
    X = dev(x, C.BF16)
    gpu_lib.linear(dev(a, C.BF16), dev(w, C.BF16), None, X, epi=gpu_lib.EPI_GATED, gate=dev(g), gate_ld=N, resid=X,
                   rows_per_sample=128)
    torch.cuda.synchronize()
    ref = x + g[np.arange(M) // 128] * (odit.f64(a) @ odit.f64(w).T)
    check(host(X), ref, C.BF16, 0, K, what="linear in-place gated", norm_tol=6e-3)


ATT = [
    # B, heads, n_q (= n_kv), dtype, d
    (1, 1, 64, C.BF16, 128), (2, 3, 200, C.BF16, 128), (1, 2, 520, C.BF16, 128), (1, 2, 24, C.BF16, 128),
    (1, 4, 4608, C.BF16, 128), (2, 4, 24, C.F32, 16), (1, 2, 77, C.F32, 64),
    (1, 2, 128, C.BF16, 128), (2, 2, 320, C.BF16, 128),   # 2 and 5 key tiles: the ring's last loads
]


@pytest.mark.parametrize("B,h,N,dt,d", ATT)
def test_attention_parity(gpu_lib, B, h, N, dt, d):
    say("attention", B, h, N, dt, d)
    q, k, v = (normal(20 + i, (B, h, N, d), dt) for i in range(3))
    Q, K = dev(q, dt), dev(k, dt)
    V = dev(v, dt)
    Vin = V.transpose(-1, -2).contiguous() if dt == C.BF16 else V
    out = torch.empty((B, N, h * d), dtype=Q.dtype, device="cuda")
    gpu_lib.attention(Q, K, Vin, out)
    torch.cuda.synchronize()
    ref = odit.merge_heads(odit.attention(q, k, v))
    # bf16: the probabilities are rounded to bf16 before the P V product (one storage rounding)
    check(host(out), ref, dt, 1, N, what=f"attention {B}x{h}x{N} d{d}", norm_tol=1e-5 if dt == C.F32 else 1e-2)


def test_attention_cross_shape(gpu_lib):
    """Queries and keys of different lengths (n_kv with a 64-key tail)."""
    B, h, nq, nkv, d = 1, 2, 300, 136, 128
    q, k, v = normal(30, (B, h, nq, d), C.BF16), normal(31, (B, h, nkv, d), C.BF16), normal(32, (B, h, nkv, d), C.BF16)
    out = torch.empty((B, nq, h * d), dtype=torch.bfloat16, device="cuda")
    gpu_lib.attention(dev(q, C.BF16), dev(k, C.BF16), dev(v, C.BF16).transpose(-1, -2).contiguous(), out)
    torch.cuda.synchronize()
    check(host(out), odit.merge_heads(odit.attention(q, k, v)), C.BF16, 1, nkv, what="attention cross 300x136",
          norm_tol=1e-2)


@pytest.mark.parametrize("pattern", ["rising", "late-spike", "flat-high", "huge"])
def test_attention_running_max_moves(gpu_lib, pattern):
    """The softmax keeps a lagging running max and redoes a 64-key tile whose row sum passes 256.
    Scores that keep rising over the keys (the max moves by more than 8 in log2 units tile after
    tile), a spike in a late tile, many keys tied near the top (row sums large with no single
    large score) and scores in the thousands must all give the exact softmax."""
    B, h, N, d = 1, 2, 704, 128
    q, k, v = (normal(50 + i, (B, h, N, d), C.BF16) for i in range(3))
    # every query gets a component along u (|u|^2 = d); key j one of beta_j, which adds about
    # 16 beta_j to its scores in log2 units (beta_j d / sqrt(d) * log2(e))
    u = np.ones(d)
    q = q.astype(np.float64) + u
    k = k.astype(np.float64)
    beta = np.zeros(N)
    if pattern == "rising":
        beta = np.linspace(0.0, 6.0, N)             # the max moves ~9 per tile: redone tile after tile
    elif pattern == "late-spike":
        beta[600:606] = 3.0                         # ~+49 in tile 9
    elif pattern == "flat-high":
        beta[128:320] = 0.7                         # ~+11 on 192 keys: row sums past 256, no single P > 256
    else:
        q, k = q * 8.0, k * 8.0                     # scores in the thousands
    k = k + beta[None, None, :, None] * u
    q = synth.bf16_round(q.astype(np.float32))
    k = synth.bf16_round(k.astype(np.float32))
    out = torch.empty((B, N, h * d), dtype=torch.bfloat16, device="cuda")
    gpu_lib.attention(dev(q, C.BF16), dev(k, C.BF16), dev(v, C.BF16).transpose(-1, -2).contiguous(), out)
    torch.cuda.synchronize()
    got = host(out)
    assert np.all(np.isfinite(got))
    check(got, odit.merge_heads(odit.attention(q, k, v)), C.BF16, 1, N, what=f"attention max moves ({pattern})",
          norm_tol=1e-2)


NORM = [(37, 3072, C.BF16), (10, 64, C.F32), (9, 200, C.BF16), (8, 1536, C.BF16), (5, 96, C.F32)]


@pytest.mark.parametrize("rows,H,dt", NORM)
@pytest.mark.parametrize("kind", [C.NORM_RMS, C.NORM_LN])
def test_norm_modulate_parity(gpu_lib, rows, H, dt, kind):
    x = normal(40, (rows, H), dt, 2.0) + 0.3
    x = x.astype(np.float32) if dt == C.F32 else x
    rps = max(1, rows // 3)
    ns = (rows + rps - 1) // rps
    mod = normal(41, (ns, 3 * H), C.F32, 0.5)
    X = dev(x, dt)
    Y = torch.empty_like(X)
    Mo = dev(mod)
    gpu_lib.norm_modulate(X, Y, shift=Mo, scale=Mo[:, H:], mod_ld=3 * H, rows_per_sample=rps, norm_kind=kind)
    torch.cuda.synchronize()
    xin = host(X)
    b = np.arange(rows) // rps
    ref = odit.norm(xin, kind, 1e-6) * (1 + mod[b, H:2 * H]) + mod[b, :H]
    check(host(Y), ref, dt, 0, H, what=f"norm_modulate {rows}x{H} kind {kind}", norm_tol=1e-5 if dt == C.F32 else 6e-3)


@pytest.mark.parametrize("rows,rps", [(16384, 4096), (4096, 512), (1003, 1003), (40, 8)])
def test_norm_modulate_staged_path(gpu_lib, rows, rps):
    """bf16 rows of one sample per block (the LDS-staged path): 32-row blocks for many rows, 8-row
    blocks for few, a ragged single-sample tail."""
    H = 3072
    x = normal(42, (rows, H), C.BF16, 2.0) + 0.3
    ns = (rows + rps - 1) // rps
    mod = normal(43, (ns, 6 * H), C.F32, 0.5)
    X = dev(x, C.BF16)
    Y = torch.empty_like(X)
    Mo = dev(mod)
    gpu_lib.norm_modulate(X, Y, shift=Mo, scale=Mo[:, H:], mod_ld=6 * H, rows_per_sample=rps, norm_kind=C.NORM_RMS)
    torch.cuda.synchronize()
    b = np.arange(rows) // rps
    ref = odit.norm(host(X), C.NORM_RMS, 1e-6) * (1 + mod[b, H:2 * H]) + mod[b, :H]
    check(host(Y), ref, C.BF16, 0, H, what=f"norm_modulate staged {rows} rows", norm_tol=6e-3)


@pytest.mark.parametrize("dt", [C.BF16, C.F32], ids=["bf16", "f32"])
def test_qk_norm_rope_parity(gpu_lib, dt):
    B, heads, d = 2, 3, 128 if dt == C.BF16 else 16
    axes = (16, 56, 56) if dt == C.BF16 else (4, 6, 6)
    grid = (1, 10, 10)
    n_tok, n_txt = 100, 8
    n_joint = n_tok + n_txt
    H = heads * d
    qkv = normal(50, (B, n_tok, 3 * H), dt)
    # norm weights 1 + N(0, 0.02^2), held in the storage dtype on both sides
    qw, kw = normal(51, (d,), C.F32, 0.02) + 1, normal(52, (d,), C.F32, 0.02) + 1
    if dt == C.BF16:
        qw, kw = synth.bf16_round(qw), synth.bf16_round(kw)
    QKV = dev(qkv, dt)
    Qo = torch.zeros((B, heads, n_joint, d), dtype=QKV.dtype, device="cuda")
    Ko = torch.zeros_like(Qo)
    Vo = torch.zeros((B, heads, d, n_joint) if dt == C.BF16 else (B, heads, n_joint, d), dtype=QKV.dtype, device="cuda")
    rope = gpu_lib.rope_table(grid, d, axes)
    gpu_lib.qk_norm_rope(QKV, heads, d, dev(qw, dt), dev(kw, dt), Qo, Ko, Vo, n_joint, n_txt, rope=rope)
    torch.cuda.synchronize()
    ang = odit.rope_angles(odit.grid_positions(grid), axes, 10000.0)
    q = odit.split_heads(qkv[..., :H].astype(np.float64), heads)
    k = odit.split_heads(qkv[..., H:2 * H].astype(np.float64), heads)
    v = odit.split_heads(qkv[..., 2 * H:].astype(np.float64), heads)
    qr = odit.apply_rope(odit.rms_norm(q, 1e-6) * qw, ang)
    kr = odit.apply_rope(odit.rms_norm(k, 1e-6) * kw, ang)
    tol = 1e-5 if dt == C.F32 else 6e-3
    check(host(Qo)[:, :, n_txt:], qr, dt, 0, d, what="qk_norm_rope Q", norm_tol=tol)
    check(host(Ko)[:, :, n_txt:], kr, dt, 0, d, what="qk_norm_rope K", norm_tol=tol)
    vg = host(Vo)
    vg = np.swapaxes(vg, -1, -2) if dt == C.BF16 else vg
    check(vg[:, :, n_txt:], v, dt, 0, 1, what="qk_norm_rope V", norm_tol=tol)
    assert np.all(host(Qo)[:, :, :n_txt] == 0)      # other stream's rows untouched


def test_rope_table_parity(gpu_lib):
    grid, axes = (3, 5, 7), (44, 42, 42)
    t = gpu_lib.rope_table(grid, 128, axes)
    torch.cuda.synchronize()
    ang = odit.rope_angles(odit.grid_positions(grid), axes, 10000.0)
    g = t.cpu().numpy().astype(np.float64)
    assert np.max(np.abs(g[..., 0] - np.cos(ang))) <= 1e-6
    assert np.max(np.abs(g[..., 1] - np.sin(ang))) <= 1e-6


@pytest.mark.parametrize("B,N,K,dt,act", [(8, 200, 3072, C.BF16, 1), (3, 64, 256, C.F32, 0), (16, 100, 64, C.F32, 1),
                                          (11, 520, 768, C.BF16, 2), (16, 9216, 3072, C.BF16, 1),
                                          (20, 300, 1000, C.F32, 1), (1, 33, 8, C.BF16, 0)])
def test_skinny_linear_parity(gpu_lib, B, N, K, dt, act):
    x = normal(60, (B, K), C.F32)
    w, b = normal(61, (N, K), dt, 0.02), normal(62, (N,), dt, 0.02)
    out = torch.empty((B, N), dtype=torch.float32, device="cuda")
    gpu_lib.skinny_linear(dev(x), dev(w, dt), dev(b, dt), out, act_in=act)
    torch.cuda.synchronize()
    xa = odit.f64(x)
    xa = {0: xa, 1: odit.silu(xa), 2: odit.gelu_tanh(xa)}[act]
    ref = xa @ odit.f64(w).T + odit.f64(b)
    check(host(out), ref, C.F32, what=f"skinny {B}x{N}x{K} act {act}", norm_tol=1e-5)


def _classes_ref(c):
    """The row map of ff_row_classes by its definition: classes of bitwise-equal rows, numbered by
    first occurrence; members grouped by class, ascending.  B > 64: every row its own class."""
    B = c.shape[0]
    bits = np.ascontiguousarray(c).view(np.uint32)
    first, cls = [], np.empty(B, dtype=np.int64)
    for b in range(B):
        j = next((i for i, f in enumerate(first) if B <= 64 and np.array_equal(bits[f], bits[b])), None)
        if j is None:
            first.append(b)
            j = len(first) - 1
        cls[b] = j
    U = len(first)
    counts = np.bincount(cls, minlength=U)
    offs = np.concatenate([[0], np.cumsum(counts)])
    memb = np.argsort(cls, kind="stable")
    out = np.zeros(2 + 3 * B, dtype=np.int32)
    out[0] = U
    out[1:1 + U] = first
    out[1 + B:2 + B + U] = offs
    out[2 + 2 * B:] = memb
    return out, U


@pytest.mark.parametrize("pattern,B,H", [("one", 8, 3072), ("distinct", 5, 3072), ("mixed", 20, 3072),
                                         ("last-col", 6, 3072), ("signed-zero", 4, 64), ("nan", 4, 64),
                                         ("one", 1, 100), ("mixed", 64, 256), ("mixed", 65, 256)])
def test_row_classes_map(gpu_lib, pattern, B, H):
    """ff_row_classes against the definition, integer map bit for bit (U, first rows, offsets,
    members), including a pair of rows that differ only in their last column, +0 against -0
    (different bits: different classes) and NaN rows with equal bits (one class)."""
    rng = np.random.default_rng(70 + B)
    base = rng.standard_normal((4, H)).astype(np.float32)
    if pattern == "one":
        c = np.repeat(base[:1], B, axis=0)
    elif pattern == "distinct":
        c = rng.standard_normal((B, H)).astype(np.float32)
    elif pattern == "mixed":
        c = base[(np.arange(B) * 7 // 3) % 4].copy()
        if B > 20:
            c[B - 1, 0] += 1.0
    elif pattern == "last-col":
        c = np.repeat(base[:1], B, axis=0)
        c[2, -1] = np.nextafter(c[2, -1], np.float32(np.inf))
        c[4] = c[2]
    elif pattern == "signed-zero":
        c = np.zeros((B, H), dtype=np.float32)
        c[1, 7] = -0.0
        c[3, 7] = -0.0
    else:
        c = np.repeat(base[:1], B, axis=0)
        c[:, 5] = np.nan
        c[2, 6] = 1.0
    ref, U = _classes_ref(c)
    got = gpu_lib.row_classes(torch.from_numpy(c).cuda()).cpu().numpy()
    torch.cuda.synchronize()
    say("row classes", pattern, B, H, "U", U)
    # the defined entries: U, the first rows of the U classes, U + 1 offsets, B members
    assert got[0] == U
    np.testing.assert_array_equal(got[1:1 + U], ref[1:1 + U])
    np.testing.assert_array_equal(got[1 + B:2 + B + U], ref[1 + B:2 + B + U])
    np.testing.assert_array_equal(got[2 + 2 * B:], ref[2 + 2 * B:])


@pytest.mark.parametrize("B", [8, 20])
def test_skinny_linear_with_classes(gpu_lib, B):
    """The GEMV over row classes stores in every row exactly what the plain GEMV stores there."""
    K, N = 3072, 1000
    rng = np.random.default_rng(80 + B)
    base = rng.standard_normal((3, K)).astype(np.float32)
    x = base[np.arange(B) % 3 if B > 8 else np.zeros(B, dtype=np.int64)]
    X = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    w, b = normal(81, (N, K), C.BF16, 0.02), normal(82, (N,), C.BF16, 0.02)
    Wd, bd = dev(w, C.BF16), dev(b, C.BF16)
    plain = torch.empty((B, N), dtype=torch.float32, device="cuda")
    grouped = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    gpu_lib.skinny_linear(X, Wd, bd, plain, act_in=1)
    classes = gpu_lib.row_classes(X)
    gpu_lib.skinny_linear(X, Wd, bd, grouped, act_in=1, classes=classes)
    torch.cuda.synchronize()
    assert int(classes[0]) == (3 if B > 8 else 1)
    np.testing.assert_array_equal(grouped.cpu().numpy().view(np.uint32), plain.cpu().numpy().view(np.uint32))


def test_profile_filter_times_one_kernel(gpu_lib):
    """With a name filter only that kernel's launches are timed; without one, every launch is."""
    A = torch.randn(512, 256, device="cuda").to(torch.bfloat16)
    W = torch.randn(512, 256, device="cuda").to(torch.bfloat16)
    out = torch.empty(512, 512, device="cuda", dtype=torch.bfloat16)
    x = torch.randn(64, 256, device="cuda").to(torch.bfloat16)
    y = torch.empty_like(x)
    try:
        for filt, expect in (("gemm_bf16", {"gemm_bf16"}), (None, {"gemm_bf16", "norm_modulate"})):
            gpu_lib.profile_filter(filt)
            gpu_lib.profile_reset()
            gpu_lib.profile_enable(True)
            gpu_lib.linear(A, W, None, out)
            gpu_lib.norm_modulate(x, y)
            gpu_lib.linear(A, W, None, out)
            torch.cuda.synchronize()
            gpu_lib.profile_enable(False)
            prof = gpu_lib.profile_read()
            assert set(prof) == expect, (filt, sorted(prof))
            assert prof["gemm_bf16"]["launches"] == 2 and prof["gemm_bf16"]["ms"] > 0
    finally:
        gpu_lib.profile_enable(False)
        gpu_lib.profile_filter(None)
        gpu_lib.profile_reset()


@pytest.mark.parametrize("nt", [True, False])
def test_stream_probe_moves_the_bytes(gpu_lib, nt):
    """The HBM streaming probe behind the bandwidth ceiling does the work it is timed for: the copy
    reproduces the source, the write leaves its pattern, the read's per-workgroup folds XOR to the
    XOR of every 16-byte word (the bytes a ragged last pass touches included)."""
    nbytes, blocks = 16 * 65539, 37
    g = torch.Generator(device="cuda").manual_seed(5)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda", generator=g)
    dst = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    gpu_lib.stream_probe(2, src, dst, nbytes, blocks, nt)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    gpu_lib.stream_probe(1, None, dst, nbytes, blocks, nt)
    torch.cuda.synchronize()
    words = dst.view(torch.int32).view(-1, 4).cpu().numpy()
    assert (words == np.array([0x3F800000, 0, 0x3F800000, 0], dtype=np.int32)).all()
    gpu_lib.stream_probe(0, src, dst, nbytes, blocks, nt)
    torch.cuda.synchronize()
    folds = dst[:16 * blocks].view(torch.int32).view(blocks, 4).cpu().numpy()
    ref = np.bitwise_xor.reduce(src.view(torch.int32).view(-1, 4).cpu().numpy(), axis=0)
    assert (np.bitwise_xor.reduce(folds, axis=0) == ref).all()
