"""Workload shapes for the selective-upsampling step.

Each workload is a seeded, synthetic stand-in for the activations of one
FLUX- or Qwen-Image-Edit-shaped block at a resolution transition.  The shapes
follow the paper's experimental setting (Section 4.1: FLUX.1-dev at 1024^2 and
2048^2 output, Qwen-Image-Edit editing with reference-image tokens); the
values are random (no trained weights or benchmark prompts are used).

This module holds sizes only: no arithmetic of the method.
"""
from __future__ import annotations

import dataclasses
import math


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str          # "f32" or "bf16": storage and GEMM operand type
    D: int              # hidden size
    H: int              # heads
    d: int              # head dim (D == H * d)
    L: int              # text tokens
    R: int              # always-kept reference tokens (editing workloads)
    H_lr: int           # low-res latent grid
    W_lr: int
    rho: float          # keep ratio
    alpha: float        # fusion weight between spatial and temporal score
    weight_std: float | None  # None: 1/sqrt(fan_in)
    D_f: int | None = None    # temporal-feature channels (None: D)
    seed: int = 0
    n_double: int = 1
    n_single: int = 0
    steps: int = 1
    mlp_ratio: int = 4
    eps_minmax: float = 1e-8

    @property
    def H_hr(self) -> int:
        return 2 * self.H_lr

    @property
    def W_hr(self) -> int:
        return 2 * self.W_lr

    @property
    def N(self) -> int:
        """High-res image tokens that are scored."""
        return self.H_hr * self.W_hr

    @property
    def N_lr(self) -> int:
        return self.H_lr * self.W_lr

    @property
    def Df(self) -> int:
        return self.D if self.D_f is None else self.D_f

    @property
    def k(self) -> int:
        return keep_count(self.rho, self.N)

    @property
    def LR(self) -> int:
        return self.L + self.R

    @property
    def S(self) -> int:
        return self.L + self.R + self.k

    def with_rho(self, rho: float) -> "Workload":
        return dataclasses.replace(self, rho=rho, name=f"{self.name}@rho{rho:g}")

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def keep_count(rho: float, n: int) -> int:
    """Number of high-res tokens kept: round-half-up of rho*n, computed in fp64."""
    return int(math.floor(rho * n + 0.5))


def mixed_keep_count(rho: float, n_lr: int) -> int:
    """Low-res tokens expanded in the mixed-resolution sequence: floor(rho M')
    (Section 3.2, Stage 2), computed in fp64."""
    return int(math.floor(rho * n_lr))


# Tiny fp32 block: hidden 256, 4x64 heads, 32 text tokens, 16x16 -> 32x32.
TINY_F32 = Workload("tiny_f32_d256", "f32", D=256, H=4, d=64, L=32, R=0,
                    H_lr=16, W_lr=16, rho=0.25, alpha=0.5, weight_std=None, seed=0)

# FLUX-shaped double-stream block at 1024^2 output (64x64 high-res latent).
FLUX_1024 = Workload("flux_1024_double", "bf16", D=3072, H=24, d=128, L=512, R=0,
                     H_lr=32, W_lr=32, rho=0.3, alpha=0.5, weight_std=0.02, seed=1)

# FLUX-shaped block at 2048^2 output (128x128 high-res latent), keep-ratio sweep.
FLUX_2048 = Workload("flux_2048_double", "bf16", D=3072, H=24, d=128, L=512, R=0,
                     H_lr=64, W_lr=64, rho=0.3, alpha=0.5, weight_std=0.02, seed=2)
FLUX_2048_RHOS = (0.1, 0.3, 0.5, 1.0)

# Qwen-Image-Edit-shaped editing block: 256 text + 4096 reference tokens.
QWEN_EDIT = Workload("qwen_edit_double", "bf16", D=3072, H=24, d=128, L=256, R=4096,
                     H_lr=32, W_lr=32, rho=0.2, alpha=0.5, weight_std=0.02, seed=3)

# Full FLUX-shaped stack (19 double + 38 single blocks), 4 denoising steps.
FLUX_STACK = Workload("flux_1024_stack", "bf16", D=3072, H=24, d=128, L=512, R=0,
                      H_lr=32, W_lr=32, rho=0.3, alpha=0.5, weight_std=0.02, seed=4,
                      n_double=19, n_single=38, steps=4)

# Small cases used only by tests: several tiles plus a ragged tail.
TINY_BF16 = Workload("tiny_bf16_d256", "bf16", D=256, H=2, d=128, L=40, R=0,
                     H_lr=12, W_lr=10, rho=0.3, alpha=0.5, weight_std=None, seed=10)
TINY_BF16_REF = Workload("tiny_bf16_ref", "bf16", D=384, H=3, d=128, L=24, R=60,
                         H_lr=9, W_lr=11, rho=0.2, alpha=0.5, weight_std=None, seed=11)
TINY_F32_RAGGED = Workload("tiny_f32_ragged", "f32", D=192, H=3, d=64, L=17, R=0,
                           H_lr=7, W_lr=9, rho=0.37, alpha=0.3, weight_std=None, seed=12)

ALL = {w.name: w for w in (TINY_F32, FLUX_1024, FLUX_2048, QWEN_EDIT, FLUX_STACK,
                           TINY_BF16, TINY_BF16_REF, TINY_F32_RAGGED)}
