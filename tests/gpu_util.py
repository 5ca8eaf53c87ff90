"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import math

import numpy as np
import torch

from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import synth

TOL = {C.F32: 1e-4, C.BF16: 2e-2}     # normwise relative error bounds on velocities and latents
LOGP_ABS = 1e-2                       # absolute bound on summed log-probs


def tdt(code):
    return torch.bfloat16 if code == C.BF16 else torch.float32


def dev(a, code=C.F32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda().to(tdt(code))


def host(t):
    return t.detach().to(torch.float64).cpu().numpy()


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


# Element-wise bound of a parity check: |got - ref| <= a |ref| + b rms(ref), with
#   a = 2 u                     the output's own rounding to bf16 (unit roundoff u = 2^-8 of an
#                               8-bit significand, round to nearest even) and one more rounding of
#                               the same element upstream (the residual stream is stored in bf16
#                               between the two halves of a block);
#   b = Z sqrt(S s^2 + K u32^2) the error carried in from upstream: S storage roundings on the path
#                               from the (identical) inputs to this output, each a relative error of
#                               at most u (standard deviation s = u / sqrt(3), the uniform case)
#                               that a random-weight layer passes on at the scale of its output's
#                               rms, plus the float32 accumulation of a K-term contraction
#                               (u32 = 2^-24 per addition, a random walk of K steps); Z = 7
#                               standard deviations is above the largest of 1e9 Gaussian draws (6.3).
# float32 paths carry no storage rounding worth modelling against their accumulation and the
# hardware transcendental approximations, so they take the per-element form of the normwise
# bound instead: b = the normwise tolerance 1e-4, a = 1e-5.
# Storage roundings per block on the path from a block's input to its output (S above): dual-stream
# block: modulated norm, normed/rotated Q K V, probabilities P, attention output, residual after
# the output projection, second modulated norm, GELU output, residual after the MLP; single-stream:
# modulated norm, Q K V | U, P, attention output, GELU output, residual; WAN: modulated norm, Q K V,
# P, attention output, residual, affine norm, cross query, cross P, cross output, residual,
# modulated norm, GELU output.  The latent embedding and the final layer's modulated norm add one
# each.
STAGES_DUAL, STAGES_SINGLE, STAGES_WAN, STAGES_EMBED, STAGES_FINAL = 8, 6, 12, 1, 1


def model_stages(m):
    s = m.n_dual * STAGES_DUAL + m.n_single * STAGES_SINGLE + m.n_wan * STAGES_WAN
    return s + (STAGES_EMBED + STAGES_FINAL if m.io_mode == C.IO_LATENT else 0)


U_BF16 = 2.0 ** -8
U_F32 = 2.0 ** -24
Z_MAX = 7.0
ELEM_F32 = (1e-5, 1e-4)


def elem_coeffs(code, stages=0, k=1):
    if code == C.F32:
        return ELEM_F32
    s = U_BF16 / math.sqrt(3.0)
    return 2.0 * U_BF16, Z_MAX * math.sqrt(stages * s * s + k * U_F32 * U_F32)


def check(got, ref, code, stages=0, k=1, what="", norm_tol=None):
    """Asserts the element-wise bound above and the normwise bound (TOL, or ``norm_tol``);
    prints the normwise error, the largest absolute difference, the largest difference over
    rms(ref) and the largest ratio to the element-wise bound, so every parity case reports them."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = np.abs(got - ref)
    r = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    a, b = elem_coeffs(code, stages, k)
    bound = a * np.abs(ref) + b * r
    nrm = rel(got, ref)
    worst = float(np.max(d / np.maximum(bound, 1e-300))) if d.size else 0.0
    maxabs = float(d.max()) if d.size else 0.0
    say(f"PARITY {what} rel={nrm:.3e} maxabs={maxabs:.3e} max/rms={maxabs / max(r, 1e-300):.3e} "
        f"worst/bound={worst:.3f} (a={a:.2e} b={b:.2e})")
    assert nrm <= (TOL[code] if norm_tol is None else norm_tol), (what, nrm)
    assert worst <= 1.0, (what, worst, maxabs)
    return nrm, maxabs, worst


def normal(seed, shape, code=C.F32, scale=1.0):
    return synth.normal(seed, shape, code, scale)


def say(*a):
    print(*a, flush=True)
