"""Plain, slow, float64 CPU oracle of the Flow-GRPO SDE rollout of a flow-matching DiT.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import or call anything here.  The product path (the HIP
library and its Python binding) never imports this package, and this package
imports nothing from the product: the two share no code.  The only common
ground is the seeded input generator, which holds none of the method's
arithmetic; every function here receives plain numpy arrays.

Modules:
  sde        -- time grid, sigma schedules (Table 1), the SDE / ODE step (Eq. 1)
                and the Gaussian transition log-probability (Sec. 3.1)
  advantage  -- group-normalised advantages, weighted-sum and GDPO-style
                multi-reward aggregation (Sec. 2.3)
  dit        -- the DiT velocity field v_theta(x_t, c, t): norms, modulation,
                RoPE, plain-softmax attention, dual-stream, single-stream and
                WAN blocks, embedders, final layer
  rollout    -- the K-step rollout loop with mixed ODE/SDE steps (Sec. 3.1,
                MixGRPO), per-step log-probs and final advantages
  losses     -- the objectives that consume the rollout: forward noising and
                the AWM (Eq. 3) and DiffusionNFT (Eq. 2) losses, the clipped
                GRPO ratio surrogate on stored trajectories
  noise      -- counter-based Gaussian noise for the SDE step (Philox4x32-10
                with Box-Muller)
  fp8        -- OCP E4M3 row quantisation and the scaled FP8 linear layer (a
                throughput variant of the DiT's linear layers, not the paper's)
"""
from . import advantage, dit, fp8, losses, noise, rollout, sde  # noqa: F401
