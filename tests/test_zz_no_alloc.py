"""The allocation-free SDE step (ff_sde_step_noalloc) against ff_sde_step with a workspace.

Both run the same kernels in the same order, so the next latent and the log-probability must be
bit-identical; each is also checked against the oracle (Eq. 1 and the Gaussian transition density,
Sec. 3.1) to the usual bounds.  Two calls in a row on the library's shared scratch, the second
smaller, show that nothing left by the first call leaks into the second.
"""
import math

import numpy as np
import pytest
import torch

from oracle import sde as osde
from paper_2602_12529_amd import configs as C

from gpu_util import LOGP_ABS, check, dev, host, normal, say

pytestmark = pytest.mark.gpu

# (B, D) of consecutive calls: a large batch first, then a smaller one with a ragged D.
CALLS = [(8, 64 * 4096 + 8), (3, 1000)]


@pytest.mark.parametrize("dt", [C.F32, C.BF16], ids=["f32", "bf16"])
def test_noalloc_matches_workspace_entry_two_calls(gpu_lib, dt):
    t, tn = 0.6, 0.5
    sigma = 0.7 * math.sqrt(t / (1 - t))
    for i, (B, D) in enumerate(CALLS):
        say("noalloc call", i, "B", B, "D", D, "dtype", dt)
        x, v, e = (normal(700 + 10 * i + j, (B, D), dt) for j in range(3))
        X, V, E = dev(x, dt), dev(v, dt), dev(e, dt)
        Xr, Xn = torch.empty_like(X), torch.empty_like(X)
        lr = torch.empty(B, dtype=torch.float64, device="cuda")
        ln = torch.full((B,), float("nan"), dtype=torch.float64, device="cuda")
        gpu_lib.sde_step(X, V, E, Xr, t, tn, sigma, logp=lr)
        gpu_lib.sde_step_noalloc(X, V, E, Xn, t, tn, sigma, logp=ln)
        torch.cuda.synchronize()
        assert torch.equal(Xn, Xr)
        assert torch.equal(ln, lr)
        got = host(Xn)
        check(got, osde.sde_step(x, v, e, t, tn, sigma), dt, 0, 3, what=f"noalloc sde step {B}x{D}")
        assert np.max(np.abs(host(ln) - osde.step_log_prob(x, v, got, t, tn, sigma))) <= LOGP_ABS


def test_noalloc_ode_step_and_errors(gpu_lib):
    """An ODE step (sigma = 0, no log-probability) equals ff_sde_step's; a log-probability asked of
    an ODE step is refused before any launch."""
    B, D = 4, 999
    x, v = normal(720, (B, D), C.BF16), normal(721, (B, D), C.BF16)
    X, V = dev(x, C.BF16), dev(v, C.BF16)
    Xr, Xn = torch.empty_like(X), torch.empty_like(X)
    gpu_lib.sde_step(X, V, X, Xr, 0.7, 0.6, 0.0)
    gpu_lib.sde_step_noalloc(X, V, X, Xn, 0.7, 0.6, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(Xn, Xr)
    with pytest.raises(gpu_lib.FFError):
        gpu_lib.sde_step_noalloc(X, V, X, Xn, 0.7, 0.6, 0.0, logp=torch.empty(B, dtype=torch.float64, device="cuda"))
