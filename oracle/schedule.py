"""Timestep grid, phase rule and predictive scheduler (Algorithm 1; Eqs. 3-5, S1).

Readings where the paper is silent or loose:
* ratios (rho_a, rho_CFG-OFF) are exact decimals; ceilings are exact;
* the "t" of the predictive curve (Eq. 4) is the step index k (the curve is
  anchored at the step index ceil(T * rho_a));
* Eq. (5) yields a real bound on the cached count; the integer quota is the
  largest integer not above it, clamped to [0, N];
* Phase 3 with f_corr = 0 never forces a full step, f_corr = 1 always does;
* Error Accumulation Elimination (tau): "consecutive caches" counts the
  immediately preceding steps that ran with a non-empty cached set (a full
  step resets it). Two readings of the threshold are kept: the cycle reading
  of the prose (a full refresh every tau steps: tau - 1 cached steps, then a
  forced full one, so tau = 1 never caches) and the literal reading of
  Algorithm 1 (force a full step once tau cached steps have passed, so tau = 1
  alternates). tau = 0 disables the constraint. It applies in every phase.
"""
from __future__ import annotations

import math
from fractions import Fraction


def _exact(x) -> Fraction:
    return x if isinstance(x, Fraction) else Fraction(str(x))


def shift_time(t_uniform: float, eta: float) -> float:
    """Eq. (S1): t = eta * t_l / (1 + (eta - 1) * t_l)."""
    return eta * t_uniform / (1.0 + (eta - 1.0) * t_uniform)


def unshift_time(t: float, eta: float) -> float:
    """Inverse of Eq. (S1): the uniform t_l that maps to t."""
    return t / (eta - (eta - 1.0) * t)


def time_grid(steps: int, eta: float = 1.0):
    """t_1 = 1 > t_2 > ... > t_{T+1} = 0: uniform grid, shifted by Eq. (S1)."""
    return [shift_time(1.0 - k / steps, eta) for k in range(steps + 1)]


def ceil_ratio(steps: int, rho) -> int:
    """ceil(T * rho) with rho an exact decimal."""
    return math.ceil(steps * _exact(rho))


def anchor_step(steps: int, rho_a=0.2) -> int:
    """Last step of Phase 1, ceil(T * rho_a) (Sec. 4.2, PCSC)."""
    return ceil_ratio(steps, rho_a)


def guidance_off_step(steps: int, eta: float, cutoff: float = 0.5) -> int:
    """Step index at which the shifted time first falls below the guidance cutoff.

    Supplement, impact of sampling parameters: solve Eq. (S1) for the uniform
    time t_l at the cutoff, then the turning point is ceil(T * (1 - t_l)).
    """
    t_l = _exact(cutoff) / (_exact(eta) - (_exact(eta) - 1) * _exact(cutoff))
    return math.ceil(steps * (1 - t_l))


def pcsc_predicted_change(k: int, sigma: float, mu: float, k_anchor: int) -> float:
    """Eq. (4): predicted dynamic voxels, sigma * exp(mu * (k - k_anchor))."""
    return sigma * math.exp(mu * (k - k_anchor))


def pcsc_quota(k: int, n_tokens: int, sigma: float, mu: float, k_anchor: int, gamma_up: float) -> int:
    """Eq. (5): c_t = D^3 - Delta_s_hat / gamma_up as an integer upper bound, clamped to [0, N]."""
    bound = n_tokens - pcsc_predicted_change(k, sigma, mu, k_anchor) / gamma_up
    return int(min(n_tokens, max(0, math.floor(bound))))


def phase_quota(k: int, steps: int, n_tokens: int, n_cache_phase2: int,
                rho_a=0.2, rho_cfg_off=0.75, xi=0.7, f_corr: int = 3) -> int:
    """Algorithm 1, step 1: cache budget c_t for step k (1-based).

    Phase 1 (k <= ceil(T rho_a)): 0. Phase 2 (k < ceil(T rho_CFG-OFF)): the
    scheduler's value. Phase 3: 0 on correction steps ((k_refine + 1) mod f_corr
    == 0), else floor(D^3 * xi).
    """
    if k <= ceil_ratio(steps, rho_a):
        return 0
    k_off = ceil_ratio(steps, rho_cfg_off)
    if k < k_off:
        return int(n_cache_phase2)
    k_refine = k - k_off
    if f_corr > 0 and (k_refine + 1) % f_corr == 0:
        return 0
    return int(math.floor(n_tokens * _exact(xi)))


TAU_CYCLE = 0
TAU_LITERAL = 1


def tau_forces_full(consecutive: int, tau: int, reading: int = TAU_CYCLE) -> bool:
    """Algorithm 1, SSC: whether the cached set is emptied after `consecutive`
    cached steps in a row (see the module readings)."""
    if tau <= 0:
        return False
    limit = tau - 1 if reading == TAU_CYCLE else tau
    return consecutive >= limit


def plan(steps: int, n_tokens: int, sigma: float, mu: float = -0.07, gamma_up: float = 1.0,
         rho_a=0.2, rho_cfg_off=0.75, xi=0.7, f_corr: int = 3, tau: int = 0,
         reading: int = TAU_CYCLE):
    """Cached count c_k for k = 1..T, pre-calculated before the loop.

    Step 1 of Algorithm 1 with the Phase 2 budget N_cache(t) from the predictive
    curve (Eqs. 4-5, sigma measured at the anchor step ceil(T rho_a)), then the
    Error Accumulation Elimination of the SSC function over the run of cached
    steps.
    """
    k_anchor = anchor_step(steps, rho_a)
    out, run = [], 0
    for k in range(1, steps + 1):
        c = phase_quota(k, steps, n_tokens, pcsc_quota(k, n_tokens, sigma, mu, k_anchor, gamma_up),
                        rho_a, rho_cfg_off, xi, f_corr)
        if c > 0 and tau_forces_full(run, tau, reading):
            c = 0
        run = run + 1 if c > 0 else 0
        out.append(c)
    return out


def cfg_active(t: float, lo: float = 0.5, hi: float = 1.0) -> bool:
    """Classifier-free guidance applies at a step whose start time t lies in
    the guidance interval [lo, hi] (the supplement's sampling configuration:
    [0.5, 1] by default; [0, 1] is continuous guidance)."""
    return lo <= float(t) <= hi


def guided_steps(times, lo: float = 0.5, hi: float = 1.0) -> list:
    """Per step k = 1..T (times t_1..t_{T+1}): whether step k is guided."""
    return [cfg_active(t, lo, hi) for t in list(times)[:-1]]

