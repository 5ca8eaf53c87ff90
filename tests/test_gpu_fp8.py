"""FP8 (OCP E4M3) row quantisation and linear layer against the oracle.

The quantiser's codes and scales must match bit for bit (the rounding decisions are taken
in float32 on both sides); the linear layer, fed the oracle's codes and scales, must match
the exact float64 result to the bf16 output's rounding plus float32 accumulation."""
import numpy as np
import pytest
import torch

from oracle import fp8 as OF
from paper_2602_12529_amd import api
from paper_2602_12529_amd import configs as C

from gpu_util import host, normal, say

pytestmark = pytest.mark.gpu


def _rows(seed, R, Cn, code):
    x = normal(seed, (R, Cn))
    x *= np.exp(np.random.default_rng(seed + 1).uniform(-4, 4, size=(R, 1))).astype(np.float32)
    if R > 3:
        x[1] = 0.0
        x[2] = -0.0
        x[3, :] = 0.0
        x[3, 5] = -3.5e-3                  # a single entry: it maps to -448, the rest to zeros
    if R > 8:                              # rows outside the ordinary rule (see oracle.fp8)
        amin = np.float32(448.0 * 2.0 ** -126)
        x[4] = x[4] * np.float32(1e-40)    # amax far below 448 * 2^-126: a zero row
        x[5] = 0.0
        x[5, 1] = amin                     # exactly at the bound: quantised, d = 2^-126
        x[5, 2] = -amin / 4
        x[6, 7] = np.inf
        x[7, 0] = np.nan
        x[8, 3] = -np.inf
    if code == C.BF16:      # the values the device holds
        x = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    return x


@pytest.mark.parametrize("code", [C.BF16, C.F32])
@pytest.mark.parametrize("R,Cn", [(1, 8), (37, 136), (300, 3072), (5, 15360)])
def test_quantize_rows_bit_exact(gpu_lib, code, R, Cn):
    x = _rows(100 + R, R, Cn, code)
    dt = torch.bfloat16 if code == C.BF16 else torch.float32
    X = torch.from_numpy(x).to(dt).cuda()
    q, d = api.quantize_fp8(X)
    torch.cuda.synchronize()
    rq, rd = OF.quantize_rows(x)
    gq, gd = q.cpu().numpy(), d.cpu().numpy()
    bad = np.flatnonzero(gq.ravel() != rq.ravel())
    assert bad.size == 0, (bad[:8], gq.ravel()[bad[:8]], rq.ravel()[bad[:8]])
    np.testing.assert_array_equal(gd.view(np.uint32), rd.view(np.uint32))


def test_quantize_rows_strided(gpu_lib):
    """Row strides above the width on both sides: the gaps are neither read into amax nor written."""
    x = _rows(7, 40, 256, C.BF16)
    X = torch.zeros((40, 264), dtype=torch.bfloat16, device="cuda")
    X[:, 256:] = 1e4                                  # would dominate amax if read
    X[:, :256] = torch.from_numpy(x).to(torch.bfloat16).cuda()
    Q = torch.full((40, 272), 0x55, dtype=torch.uint8, device="cuda")
    d = torch.empty(40, dtype=torch.float32, device="cuda")
    api.quantize_fp8(X[:, :256], Q[:, :256], d)
    torch.cuda.synchronize()
    rq, rd = OF.quantize_rows(x)
    np.testing.assert_array_equal(Q[:, :256].cpu().numpy(), rq)
    assert torch.all(Q[:, 256:] == 0x55)
    np.testing.assert_array_equal(d.cpu().numpy(), rd)


def _codes(seed, R, K):
    """Codes and scales of a Gaussian [R, K] with per-row magnitudes, by the oracle's quantiser."""
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((R, K)) * np.exp(rng.uniform(-2, 2, size=(R, 1)))).astype(np.float32)
    return OF.quantize_rows(x)


# The matrix core's FP8 MFMA sums the 64 products of one instruction below float32 precision:
# measured errors reach ~6e-6 of sum_k |a_k w_k| (a cancelling sum of large terms), so the
# accumulation term of the bound scales with that sum, not with the result.
ACC_REL = 2.0 ** -14


def _check(out, ref, a_q, a_d, w_q, w_d, tag=""):
    o = host(out)
    err = np.abs(o - ref)
    s_abs = (np.abs(OF.decode(a_q)) @ np.abs(OF.decode(w_q)).T) * a_d.astype(np.float64)[:, None] \
        * w_d.astype(np.float64)[None, :]
    # bf16 output rounding (2^-8 relative) plus the accumulation (GELU's slope stays below 1.13)
    bound = 2.0 ** -8 * np.abs(ref) + 1.2 * ACC_REL * s_abs + 1e-30
    ratio = np.max(np.maximum(err - 2.0 ** -8 * np.abs(ref), 0) / (s_abs + 1e-30))
    say("fp8", tag, "max accumulation error / sum|a w| =", ratio)
    bad = np.argwhere(err > bound)
    assert bad.size == 0, (bad[:5], o[tuple(bad[0])], ref[tuple(bad[0])])


@pytest.mark.parametrize("M,N,K,gelu", [(1, 8, 128, False), (100, 64, 128, True), (549, 360, 384, False),
                                        (1030, 2104, 640, True), (4096, 3072, 3072, False),
                                        (3, 296, 15360, False), (520, 1032, 15360, True)])
def test_linear_fp8_parity(gpu_lib, M, N, K, gelu):
    a_q, a_d = _codes(M * 7 + 1, M, K)
    w_q, w_d = _codes(N * 11 + 2, N, K)
    bias = normal(N + 5, (N,), C.BF16, 0.5)
    bias = torch.from_numpy(bias).to(torch.bfloat16)
    ref = OF.linear_fp8(a_q, a_d, w_q, w_d, bias.float().numpy(), gelu=gelu)
    out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    api.linear_fp8(torch.from_numpy(a_q).cuda(), torch.from_numpy(a_d).cuda(), torch.from_numpy(w_q).cuda(),
                   torch.from_numpy(w_d).cuda(), bias.cuda(), out, epi=api.EPI_GELU if gelu else api.EPI_BIAS)
    torch.cuda.synchronize()
    _check(out, ref, a_q, a_d, w_q, w_d, f"{M}x{N}x{K}")


def test_linear_fp8_strided_operands_and_gelu_from(gpu_lib):
    """Row strides above K for the codes and above N for the output; GELU from a column on."""
    M, N, K = 300, 200, 256
    a_q, a_d = _codes(31, M, K)
    w_q, w_d = _codes(32, N, K)
    A = torch.zeros((M, K + 64), dtype=torch.uint8, device="cuda")
    A[:, :K] = torch.from_numpy(a_q).cuda()
    A[:, K:] = 0x7e                                      # 448: would show if read
    W = torch.zeros((N, K + 16), dtype=torch.uint8, device="cuda")
    W[:, :K] = torch.from_numpy(w_q).cuda()
    W[:, K:] = 0x7e
    out = torch.full((M, N + 8), 7.0, dtype=torch.bfloat16, device="cuda")
    api.linear_fp8(A[:, :K], torch.from_numpy(a_d).cuda(), W[:, :K], torch.from_numpy(w_d).cuda(), None,
                   out[:, :N], epi=api.EPI_GELU, gelu_from=120)
    torch.cuda.synchronize()
    lin = OF.linear_fp8(a_q, a_d, w_q, w_d)
    ref = np.concatenate([lin[:, :120], OF.gelu_tanh(lin[:, 120:])], axis=1)
    _check(out[:, :N], ref, a_q, a_d, w_q, w_d, "strided")
    assert torch.all(out[:, N:] == 7.0)


@pytest.mark.timeout(600)
def test_linear_fp8_full_size_sampled_rows(gpu_lib):
    """The MLP-up projection of the one-block Flux workload (36864 x 12288 x 3072, GELU) in FP8:
    every output is computed; the oracle recomputes 69 sampled rows (every 576th, and the edges)."""
    M, N, K = 36864, 12288, 3072
    say("fp8 full size: quantising inputs on the host")
    a_q, a_d = _codes(41, M, K)
    w_q, w_d = _codes(42, N, K)
    bias = torch.from_numpy(normal(43, (N,), C.BF16, 0.5)).to(torch.bfloat16)
    out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    api.linear_fp8(torch.from_numpy(a_q).cuda(), torch.from_numpy(a_d).cuda(), torch.from_numpy(w_q).cuda(),
                   torch.from_numpy(w_d).cuda(), bias.cuda(), out, epi=api.EPI_GELU)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, M, M // 64), [1, 255, 256, M - 257, M - 1]]))
    say("  oracle on", rows.size, "rows")
    ref = OF.linear_fp8(a_q[rows], a_d[rows], w_q, w_d, bias.float().numpy(), gelu=True)
    _check(out[torch.from_numpy(rows).cuda()], ref, a_q[rows], a_d[rows], w_q, w_d, "full size")
