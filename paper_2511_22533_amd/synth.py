"""Seeded synthetic workloads for the cached sparse-structure flow-DiT step.

This module only *draws* inputs: model shapes, seeded weights, initial noise
grids, image-condition tokens and the per-step cache-quota schedules that stand
in for the calibrated scheduler. It holds none of the method's arithmetic
(scoring, selection, the transformer, the Euler update, the timestep shift or
the predictive scheduler live elsewhere, twice: once in the oracle and once in
the HIP library). Both sides receive the arrays produced here.

Shapes follow the TRELLIS sparse-structure stage the paper accelerates
(Sec. 3.2: a latent grid S in R^{B x C x D x H x W} evolved by a flow
transformer conditioned on DINOv2 image tokens). Trained weights and real image
features are not available, so every tensor is drawn from a fixed seed:

* weights and biases: N(0, 0.02), seed 0, drawn in ``weight_specs`` order;
  rounded to bfloat16 (round-to-nearest-even) for the bf16 workloads;
* initial noise x_T: N(0, 1), seed 1000 + b;
* condition tokens: N(0, 1), seed 2000 + b (rounded to bf16 for bf16 models);
* quota schedule parameters: seed 3000 (shared) and 3100 + b (per sample).

Token order inside a grid is row-major over (z, y, x): n = (z*G + y)*G + x.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Tuple

import numpy as np

IN_CH = 8          # latent channels of the sparse-structure grid
T_FREQ = 256       # sinusoidal timestep features (128 cos + 128 sin)
OUT_CH = 8


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    grid: int
    width: int
    depth: int
    heads: int
    cond_tokens: int
    cond_width: int
    dtype: str                  # "f32" or "bf16"
    mlp_ratio: int = 4
    in_ch: int = IN_CH

    @property
    def tokens(self) -> int:
        return self.grid ** 3

    @property
    def head_dim(self) -> int:
        return self.width // self.heads

    @property
    def mlp_width(self) -> int:
        return self.width * self.mlp_ratio


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    steps: int
    shift: float                # timestep shift factor eta (1.0 = uniform)
    schedule: str               # quota recipe name, see ``quota_schedule``
    description: str
    guidance: float = 0.0       # guidance weight w of guided steps (0: no guided steps)
    guidance_interval: tuple = (0.5, 1.0)   # steps whose start time lies here are guided


TINY = ModelConfig(grid=8, width=128, depth=2, heads=4, cond_tokens=64, cond_width=128, dtype="f32")
TRELLIS16 = ModelConfig(grid=16, width=1024, depth=24, heads=16, cond_tokens=1374, cond_width=1024, dtype="bf16")
TRELLIS32 = ModelConfig(grid=32, width=1024, depth=12, heads=16, cond_tokens=1374, cond_width=1024, dtype="bf16")

WORKLOADS: Dict[str, Workload] = {
    "tiny_f32": Workload("tiny_f32", TINY, 1, 10, 1.0, "linear_half",
                         "8^3 grid, width 128, 2 blocks, 4x32 heads, 64x128 cond, fp32, "
                         "10 uniform steps, quota 0 up to step 3 then linear to 50% at step 10"),
    "trellis16_full": Workload("trellis16_full", TRELLIS16, 1, 25, 3.0, "none",
                               "16^3 grid, width 1024, 24 blocks, 16x64 heads, 1374x1024 cond, bf16, "
                               "25 shifted steps, no caching"),
    "trellis16_cached": Workload("trellis16_cached", TRELLIS16, 1, 25, 3.0, "logistic80",
                                 "as trellis16_full with 5 full steps then a seeded logistic quota "
                                 "reaching 80% cached tokens at step 25"),
    "trellis16_cached_b4": Workload("trellis16_cached_b4", TRELLIS16, 4, 25, 3.0, "logistic_ragged",
                                    "trellis16_cached at batch 4 with per-sample final quota in [0.40, 0.85]"),
    "trellis32_cached": Workload("trellis32_cached", TRELLIS32, 1, 25, 3.0, "fixed70",
                                 "32^3 grid, width 1024, 12 blocks, 1374x1024 cond, bf16, "
                                 "5 full steps then a fixed 70% quota"),
    "trellis16_cached_cfg": Workload("trellis16_cached_cfg", TRELLIS16, 1, 25, 3.0, "logistic80",
                                     "trellis16_cached with classifier-free guidance (w = 3, zero "
                                     "unconditional input) on the steps starting at t in [0.5, 1] "
                                     "(steps 1-19 under the eta = 3 shift)", guidance=3.0),
}


def weight_specs(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Canonical parameter list (name, shape); linear weights are [out][in]."""
    d, dc, dm, n = cfg.width, cfg.cond_width, cfg.mlp_width, cfg.tokens
    specs: List[Tuple[str, Tuple[int, ...]]] = [
        ("in_w", (d, cfg.in_ch)), ("in_b", (d,)), ("pos", (n, d)),
        ("t1_w", (d, T_FREQ)), ("t1_b", (d,)), ("t2_w", (d, d)), ("t2_b", (d,)),
    ]
    for l in range(cfg.depth):
        p = f"blk{l}."
        specs += [
            (p + "mod_w", (6 * d, d)), (p + "mod_b", (6 * d,)),
            (p + "qkv_w", (3 * d, d)), (p + "qkv_b", (3 * d,)),
            (p + "o_w", (d, d)), (p + "o_b", (d,)),
            (p + "q_w", (d, d)), (p + "q_b", (d,)),
            (p + "kv_w", (2 * d, dc)), (p + "kv_b", (2 * d,)),
            (p + "co_w", (d, d)), (p + "co_b", (d,)),
            (p + "fc1_w", (dm, d)), (p + "fc1_b", (dm,)),
            (p + "fc2_w", (d, dm)), (p + "fc2_b", (d,)),
        ]
    specs += [("out_w", (OUT_CH, d)), ("out_b", (OUT_CH,))]
    return specs


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    rounded = (bits + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    out = rounded.view(np.float32).copy()
    nan = np.isnan(a)
    if nan.any():
        out[nan] = np.float32(np.nan)
    return out


def make_weights(cfg: ModelConfig, seed: int = 0, scale: float = 0.02) -> Dict[str, np.ndarray]:
    """Seeded N(0, scale) float32 weights; bf16-representable for bf16 models."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out: Dict[str, np.ndarray] = {}
    s = np.float32(scale)
    for name, shape in weight_specs(cfg):
        w = rng.standard_normal(shape, dtype=np.float32) * s
        out[name] = round_bf16(w) if cfg.dtype == "bf16" else w
    return out


def make_noise(cfg: ModelConfig, batch: int, seed_base: int = 1000) -> np.ndarray:
    """x_T ~ N(0, 1), float32 [B][N][C] (token-major)."""
    x = np.empty((batch, cfg.tokens, cfg.in_ch), np.float32)
    for b in range(batch):
        rng = np.random.Generator(np.random.PCG64(seed_base + b))
        x[b] = rng.standard_normal((cfg.tokens, cfg.in_ch), dtype=np.float32)
    return x


def make_cond(cfg: ModelConfig, batch: int, seed_base: int = 2000) -> np.ndarray:
    """Stand-in for DINOv2 image tokens: N(0, 1), float32 [B][Nc][dc]."""
    c = np.empty((batch, cfg.cond_tokens, cfg.cond_width), np.float32)
    for b in range(batch):
        rng = np.random.Generator(np.random.PCG64(seed_base + b))
        c[b] = rng.standard_normal((cfg.cond_tokens, cfg.cond_width), dtype=np.float32)
    return round_bf16(c) if cfg.dtype == "bf16" else c


def make_uncond(cfg: ModelConfig, batch: int) -> np.ndarray:
    """Unconditional input of guided steps: all-zero condition tokens, float32 [B][Nc][dc]."""
    return np.zeros((batch, cfg.cond_tokens, cfg.cond_width), np.float32)


def quota_schedule(w: Workload, seed: int = 3000) -> np.ndarray:
    """Cached-token counts c[k-1][b] for steps k = 1..T (int64, each in [0, N]).

    These schedules stand in for the calibrated predictive scheduler, whose
    anchor measurement needs the trained occupancy decoder. Recipes:

    * ``none``: every step full.
    * ``linear_half``: 0 for k <= 3, then floor(N/2 * (k-3)/(T-3)).
    * ``logistic80``: 0 for k <= 5; for k >= 6, u_k = 1/(1+exp(-s(k-k0))),
      c = floor(N * 0.8 * (u_k-u_5)/(u_T-u_5)); s ~ U[0.3,0.8], k0 ~ U[10,18].
    * ``logistic_ragged``: as logistic80 with the 0.8 replaced by a per-sample
      Q_b ~ U[0.40, 0.85] (seed 3100 + b).
    * ``fixed70``: 0 for k <= 5, then floor(0.7 N).
    """
    n, T, B = w.model.tokens, w.steps, w.batch
    c = np.zeros((T, B), np.int64)
    if w.schedule == "none":
        return c
    if w.schedule == "linear_half":
        for k in range(4, T + 1):
            c[k - 1, :] = (n // 2) * (k - 3) // (T - 3)
        return c
    if w.schedule == "fixed70":
        c[5:, :] = int(math.floor(0.7 * n))
        return c
    if w.schedule in ("logistic80", "logistic_ragged"):
        rng = np.random.Generator(np.random.PCG64(seed))
        s = float(rng.uniform(0.3, 0.8))
        k0 = float(rng.uniform(10.0, 18.0))
        u = lambda k: 1.0 / (1.0 + math.exp(-s * (k - k0)))
        targets = [0.8] * B
        if w.schedule == "logistic_ragged":
            targets = [float(np.random.Generator(np.random.PCG64(seed + 100 + b)).uniform(0.40, 0.85))
                       for b in range(B)]
        for k in range(6, T + 1):
            frac = (u(k) - u(5)) / (u(T) - u(5))
            for b in range(B):
                c[k - 1, b] = min(n, max(0, int(math.floor(n * targets[b] * frac))))
        return c
    raise ValueError(f"unknown schedule {w.schedule!r}")
