"""Named synthetic workloads (shapes, step counts, window, tolerances).

Each workload stands in for a setting of the paper: the SD-v1.5 latent shape
4x64x64 (Sec. 3.2), DDIM sampling with a sliding window of P timesteps (Sec. 2.1,
Sec. 3.3) and a cache tolerance delta (Sec. 2.2, Eq. (5)). The paper's UNet is replaced
by a synthetic network: a linear map eps = c_j * x, or a 2x2-patch MLP with a
sinusoidal time embedding. Pure data: no arithmetic of the method lives here.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    latent: tuple          # (C, H, W); batch is 1
    T: int                 # DDIM sampling steps
    window: int            # Picard window P
    delta: float           # cache tolerance (strict '<' hit test)
    tol: float             # Picard convergence tolerance tau (mean square)
    model: str             # "linear" or "patch_mlp"
    hidden: int = 0        # patch-MLP hidden width H
    temb_dim: int = 128
    patch: int = 2
    blocks: int = 0        # Parareal blocks (0: the Picard sampler's workload)

    @property
    def D(self) -> int:
        c, h, w = self.latent
        return c * h * w

    @property
    def tokens(self) -> int:
        c, h, w = self.latent
        return (h // self.patch) * (w // self.patch)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# Tiny closed-form case: linear eps, T=10, window 4.
TINY_LINEAR = Workload("tiny_linear_1x4x8x8_T10_P4", (4, 8, 8), 10, 4, 0.05, 1e-3, "linear")
# Small patch-MLP case: 4x32x32, T=50, window 16, H=512 over 256 tokens.
SMALL_MLP = Workload("mlp_4x32x32_T50_P16_H512", (4, 32, 32), 50, 16, 0.05, 1e-3,
                     "patch_mlp", hidden=512)
# Headline case: SD latent shape 4x64x64, T=100, window 32, H=1024 over 1024 tokens.
SD_MLP = Workload("mlp_4x64x64_T100_P32_H1024", (4, 64, 64), 100, 32, 0.05, 1e-3,
                  "patch_mlp", hidden=1024)
# Long-window stress case: T=1000 (full schedule), window 128.
LONG_MLP = Workload("mlp_4x64x64_T1000_P128_H1024", (4, 64, 64), 1000, 128, 0.05, 1e-3,
                    "patch_mlp", hidden=1024)

# Parareal-style variant: 4x96x96 latent, T=100 in 10 blocks of 10 fine steps, H=2048 over
# 2304 tokens, fine and coarse outputs cached at delta=0.05.
PARAREAL_MLP = Workload("parareal_4x96x96_T100_B10_H2048", (4, 96, 96), 100, 1, 0.05, 1e-3,
                        "patch_mlp", hidden=2048, blocks=10)

HEADLINE_DELTAS = (0.0, 0.02, 0.05, 0.1)

ALL = {w.name: w for w in (TINY_LINEAR, SMALL_MLP, SD_MLP, LONG_MLP, PARAREAL_MLP)}
