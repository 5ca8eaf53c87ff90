"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
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


def normal(seed, shape, code=C.F32, scale=1.0):
    return synth.normal(seed, shape, code, scale)


def say(*a):
    print(*a, flush=True)
