"""One denoising step of the cached sampler, and the trajectory loop (Algorithm 1).

Step k with times (t, t') = (t_k, t_{k+1}) and per-sample cached counts c_b:
  1. score the tokens from the two stored velocity caches (SSC) when c_b > 0;
  2. cache the c_b lowest-scoring tokens, keep the rest active (ascending);
  3. run the flow transformer on the active tokens only;
  4. merge: v = v_cache with the active rows replaced by the fresh velocities;
  5. Euler: x <- x - (t - t') * v   (rectified flow, Sec. 3.1);
  6. rotate: v_prev <- v_cache, v_cache <- v.
Both caches start at zero. A step with c_b = 0 for every sample is the full step.

Readings: the batch is handled per sample (each sample has its own index set);
an empty active set (c_b = N) skips the transformer for that sample; the step
size is (t - t') computed in float64 and rounded once to float32; the Euler
product and difference are two rounded float32 operations.

Guided steps (classifier-free guidance inside the CFG interval, Sec. 3.2 and
the supplement's sampling configuration): the transformer runs twice on the
same active set, once with the condition and once with the unconditional
input, and the fresh velocity is (1 + w) v_cond - w v_uncond (Ho and
Salimans' form), each pass's output rounded to float32 first. The caches hold
the guided velocity, so the scores, the selection and the Euler update are
those of the unguided step applied to it.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Optional, Sequence

import numpy as np

from . import ssc

F32 = np.float32


@dataclasses.dataclass
class State:
    x: np.ndarray        # float32 [B][N][C] latent grid, token-major
    v_cache: np.ndarray  # float32 [B][N][C] velocity used at the previous step
    v_prev: np.ndarray   # float32 [B][N][C] velocity used two steps back

    @classmethod
    def start(cls, x_T: np.ndarray) -> "State":
        x = np.array(x_T, dtype=F32, copy=True)
        return cls(x, np.zeros_like(x), np.zeros_like(x))

    def copy(self) -> "State":
        return State(self.x.copy(), self.v_cache.copy(), self.v_prev.copy())


@dataclasses.dataclass
class StepRecord:
    active: List[np.ndarray]       # per sample, ascending token indices
    scores: List[Optional[np.ndarray]]
    v_active: List[np.ndarray]     # per sample, float32 [n_b][C] (guided when the step is)
    v_cond: List[np.ndarray] = dataclasses.field(default_factory=list)    # guided steps: each pass's
    v_uncond: List[np.ndarray] = dataclasses.field(default_factory=list)  # float32 output


# velocity(b, x_active [n][C] float32, idx [n] int64, t) -> [n][C]
VelocityFn = Callable[[int, np.ndarray, np.ndarray, float], np.ndarray]


def model_velocity(model, cond: np.ndarray) -> VelocityFn:
    """Adapt a dit.Model and per-sample condition tokens [B][Nc][dc] to a VelocityFn."""
    def fn(b, x_active, idx, t):
        return model.forward(x_active, idx, t, cond[b])
    return fn


def guide(v_cond: np.ndarray, v_uncond: np.ndarray, w: float) -> np.ndarray:
    """Classifier-free guidance: (1 + w) * v_cond - w * v_uncond in float32.

    The weights are rounded to float32 once, 1 + w computed in float64 first;
    each product and the difference are rounded float32 operations (no fused
    multiply-add)."""
    a, ws = F32(1.0 + float(w)), F32(float(w))
    return (a * np.asarray(v_cond, F32)) - (ws * np.asarray(v_uncond, F32))


def step(state: State, velocity: VelocityFn, t: float, t_next: float,
         n_cache: Sequence[int], omega: float = 0.7, uncond: Optional[VelocityFn] = None,
         w: float = 0.0) -> StepRecord:
    """Advance ``state`` in place by one step of Algorithm 1; returns what was selected.

    With ``uncond`` the step is guided: both passes see the same active set."""
    B, N, C = state.x.shape
    dt = F32(float(t) - float(t_next))
    rec = StepRecord([], [], [])
    for b in range(B):
        c = int(n_cache[b])
        if c > 0:
            score = ssc.cache_score(state.v_cache[b], state.v_prev[b], omega)
            _, active = ssc.select(score, c)
        else:
            score, active = None, np.arange(N, dtype=np.int64)
        v = state.v_cache[b].copy()
        if active.size:
            v_act = np.asarray(velocity(b, state.x[b][active], active, t), dtype=np.float64).astype(F32)
            if uncond is not None:
                v_un = np.asarray(uncond(b, state.x[b][active], active, t), dtype=np.float64).astype(F32)
                rec.v_cond.append(v_act)
                rec.v_uncond.append(v_un)
                v_act = guide(v_act, v_un, w)
            v[active] = v_act
        else:
            v_act = np.zeros((0, C), F32)
        state.x[b] = state.x[b] - dt * v
        state.v_prev[b] = state.v_cache[b]
        state.v_cache[b] = v
        rec.active.append(active)
        rec.scores.append(score)
        rec.v_active.append(v_act)
    return rec


def sample(x_T: np.ndarray, velocity: VelocityFn, times: Sequence[float],
           quotas: np.ndarray, omega: float = 0.7, records: list | None = None,
           uncond: Optional[VelocityFn] = None, w: float = 0.0,
           guided: Optional[Sequence[bool]] = None) -> State:
    """Run the loop k = 1..T with times[k-1] -> times[k] and quotas[k-1][b].

    With ``uncond``, step k is guided when ``guided[k-1]`` holds (every step
    when ``guided`` is None)."""
    st = State.start(x_T)
    for k in range(len(times) - 1):
        g = uncond is not None and (guided is None or bool(guided[k]))
        rec = step(st, velocity, times[k], times[k + 1], quotas[k], omega, uncond if g else None, w)
        if records is not None:
            records.append(rec)
    return st
