"""Shared helpers for the GPU parity tests (not collected as tests)."""
from __future__ import annotations

import sys
from typing import Optional

import numpy as np

from oracle import dit, sampler, ssc
from paper_2511_22533_amd import synth


def say(*a):
    """Name the case before each GPU step (flushed, so it survives a crash)."""
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def max_rel(got: np.ndarray, want: np.ndarray) -> float:
    """max_i |g_i - o_i| / max_i |o_i| (elementwise relative error is ill-posed near 0)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    den = np.max(np.abs(want))
    return float(np.max(np.abs(got - want)) / (den if den > 0 else 1.0))


def rel_l2(got: np.ndarray, want: np.ndarray) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    return float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))


def bf16_round(a: np.ndarray) -> np.ndarray:
    return synth.round_bf16(np.asarray(a, np.float32))


def torch_dtype(cfg_dtype: str):
    import torch
    return torch.bfloat16 if cfg_dtype == "bf16" else torch.float32


def to_dev(a: np.ndarray, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def depth_variant(cfg: synth.ModelConfig, depth: int) -> synth.ModelConfig:
    return synth.ModelConfig(grid=cfg.grid, width=cfg.width, depth=depth, heads=cfg.heads,
                             cond_tokens=cfg.cond_tokens, cond_width=cfg.cond_width, dtype=cfg.dtype,
                             mlp_ratio=cfg.mlp_ratio)


class Pair:
    """One model on both sides: the HIP library (through the C ABI) and the oracle."""

    def __init__(self, cfg: synth.ModelConfig, batch: int, seed: int = 0, scale: float = 0.02,
                 uncond: Optional[np.ndarray] = None):
        """uncond: the unconditional input of guided steps ([B][Nc][dc]); the
        state is then created for guided steps."""
        import torch
        from paper_2511_22533_amd import f3c
        self.cfg, self.B = cfg, batch
        self.W = synth.make_weights(cfg, seed=seed, scale=scale)
        self.cond = synth.make_cond(cfg, batch)
        self.x_T = synth.make_noise(cfg, batch)
        self.model = f3c.Model(cfg).load(self.W)
        self.state = f3c.State(self.model, batch, guided=uncond is not None)
        self.cond_dev = to_dev(self.cond)
        self.state.set_cond(self.cond_dev)
        self.uncond = uncond
        if uncond is not None:
            self.uncond_dev = to_dev(uncond)
            self.state.set_uncond(self.uncond_dev)
        self.oracle = dit.Model(cfg, self.W)
        torch.cuda.synchronize()

    def velocity(self):
        return sampler.model_velocity(self.oracle, self.cond)

    def velocity_uncond(self):
        return sampler.model_velocity(self.oracle, self.uncond)


def oracle_selection(v_cache: np.ndarray, v_prev: np.ndarray, n_cache, omega=0.7):
    out = []
    for b in range(v_cache.shape[0]):
        if n_cache[b] == 0:
            out.append((None, np.arange(v_cache.shape[1])))
        else:
            s = ssc.cache_score(v_cache[b], v_prev[b], omega)
            out.append((s, ssc.select(s, int(n_cache[b]))[1]))
    return out
