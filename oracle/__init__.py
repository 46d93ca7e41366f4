"""CPU oracle for the cached Picard sliding-window sampler — TEST INFRASTRUCTURE ONLY.

A plain, slow, serial float64 implementation of what the device path computes, written
from the paper (Sec. 2.1 Eq. (1)-(2); Sec. 2.2 Eq. (3)-(7)). Only ``tests/``, the smoke
entry point and the CPU-baseline leg of the benchmark may import it; the product path
(the HIP library and its Python binding) never does, and shares no code with it.

Modules:
  schedule     scaled-linear alpha_bar, trailing timesteps, DDIM and generalized-step
               (eta) coefficients
  eps_models   linear network, patch-MLP network (bf16 operand rounding emulated)
  sampler      per-step cached Picard sweep, uncached Picard, serial DDIM and DDPM
               references, the revisit statistic
  scalar_sim   scalar recurrence for the linear network (pins the sampler's decisions)
  parareal     cached and uncached Parareal sampler (not imported here; import it directly)

Pins (tests/test_oracle_*.py, run with -m "not gpu") tie every function to something
other than itself: closed forms, textbook DDIM and DDPM, the scalar recurrence, library
routines on tiny inputs, and brute force; tests/test_oracle_mutations.py checks that
plausible mistakes planted in a copy of this package fail them. No function here is
"parity unpinned".
"""
from . import schedule, eps_models, sampler, scalar_sim  # noqa: F401
