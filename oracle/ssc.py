"""Spatiotemporal Stability Criterion (Sec. 4.2, Eqs. 2, 6, 7; Algorithm 1 SSC).

Float32 throughout, one rounded operation at a time, because the result is an
integer decision (which tokens are cached) and must be taken in the same
precision as on the device.

Readings where the paper is silent:
* the two velocity fields fed to the criterion are the two stored caches
  (v_cache, v_prev_cache) that Algorithm 1 passes to SSC;
* min/max of Eq. (7) run over all tokens of one sample (cached ones included);
  NaN entries are ignored by min/max;
* when max == min the normalised term is 0 for every token;
* the squared norm is accumulated channel by channel from 0, in channel order;
* w_a = float32(omega), w_v = float32(1) - float32(omega);
* ties in the score are broken by the smaller token index; NaN scores order
  after every number (such tokens are never cached before a finite one).
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


def velocity_magnitude(v: np.ndarray) -> np.ndarray:
    """V_i = ||v_i||_2 for v float32 [N][C]: sequential float32 sum of squares, then sqrt."""
    v = np.asarray(v, dtype=F32)
    s = np.zeros(v.shape[0], dtype=F32)
    for ch in range(v.shape[1]):
        sq = v[:, ch] * v[:, ch]          # rounded float32 product
        s = s + sq                        # rounded float32 sum
    return np.sqrt(s)                     # correctly rounded float32 sqrt


def acceleration(v_cur: np.ndarray, v_prev: np.ndarray) -> np.ndarray:
    """A_i = ||v_i(t) - v_i(t-1)||_2 (Eq. 2): the difference is rounded first."""
    d = np.asarray(v_cur, dtype=F32) - np.asarray(v_prev, dtype=F32)
    return velocity_magnitude(d)


def minmax_normalise(a: np.ndarray) -> np.ndarray:
    """Eq. (7): (a_i - min_j a_j) / (max_j a_j - min_j a_j), 0 where max == min."""
    a = np.asarray(a, dtype=F32)
    lo = np.fmin.reduce(a)                # NaN-ignoring
    hi = np.fmax.reduce(a)
    if not (hi > lo):
        return np.zeros_like(a)
    return (a - lo) / (hi - lo)           # two rounded float32 operations


def cache_score(v_cache: np.ndarray, v_prev: np.ndarray, omega: float) -> np.ndarray:
    """Eq. (6): C_i = omega * norm(A_i) + (1 - omega) * norm(V_i), float32 [N]."""
    w_a = F32(omega)
    w_v = F32(1.0) - w_a
    n_a = minmax_normalise(acceleration(v_cache, v_prev))
    n_v = minmax_normalise(velocity_magnitude(v_cache))
    return (w_a * n_a) + (w_v * n_v)


def select(score: np.ndarray, n_cache: int):
    """Algorithm 1, SSC: the n_cache tokens with the lowest score are cached.

    The order is ascending (score, token index) with NaN last, i.e. the first
    n_cache entries of a stable ascending sort. Returns (cached, active), both
    ascending int64 token indices; active = all indices minus cached.
    """
    n = int(score.shape[0])
    if not 0 <= n_cache <= n:
        raise ValueError("n_cache out of range")
    order = np.argsort(np.asarray(score, dtype=F32), kind="stable")  # NaN sorts last
    cached = np.sort(order[:n_cache])
    mask = np.ones(n, dtype=bool)
    mask[cached] = False
    active = np.nonzero(mask)[0]
    return cached.astype(np.int64), active.astype(np.int64)
