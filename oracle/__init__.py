"""CPU oracle for the Fast3Dcache cached flow-DiT sampler (arXiv 2511.22533).

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, deliberately
unoptimised restatement of what the paper's method computes. It exists so the
HIP library can be checked against it; nothing in the product path may import,
call or link it. Only the test suite, the smoke check and the benchmark's CPU
baseline leg use it.

It shares no code with the HIP library. It takes its inputs (weights, noise,
condition tokens, quota schedules) as plain arrays produced by the seeded
generators, and never reads anything produced by the GPU path.

Modules
-------
ssc       Spatiotemporal Stability Criterion: velocity magnitude, acceleration
          (Eq. 2), min-max normalisation (Eq. 7), cache-ability score (Eq. 6),
          and the selection of the c_t lowest-scoring tokens (Algorithm 1, SSC).
schedule  Timestep grid with the shift of Eq. (S1), the anchor / CFG-off step
          arithmetic, the three-phase quota rule of Algorithm 1 and the
          predictive scheduler of Eqs. (3)-(5).
dit       The flow transformer evaluated on a token subset (Sec. 3.2, Sec. 4.2
          index-based selection), in float64.
sampler   One denoising step of Algorithm 1 (select, forward on the active
          subset, merge with the cached velocities, Euler update, cache
          rotation) and the full trajectory loop.
flops     The per-block FLOPs model of the supplement (FLOPs Calculation).

Precision: the paper fixes none. The transformer runs in float64. The sampler
state (latent grid and the two velocity caches) is float32, and every float32
operation that feeds the token selection (scores) or the latent update is done
one rounded float32 operation at a time, in the order written, so that the
integer outcome (which tokens are cached) is decided in the same precision as
on the device.

Parity status: the absolute velocities of the random-initialised transformer
are "parity unpinned" (no trained weights and no printed activations exist);
every other function is pinned by the tests under tests/ (closed forms,
brute force on tiny inputs, invariants, the paper's worked example).
"""
from . import ssc, schedule, dit, sampler, flops  # noqa: F401
