"""Pins for the oracle's schedules: Eq. (S1) shift, Algorithm 1 phases, Eqs. (3)-(5), FLOPs model."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import dit, flops, schedule
from paper_2511_22533_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_worked_example_eta2_turning_point():
    g = _golden("eta_shift_turning_point.json")
    t_l = schedule.unshift_time(g["cutoff"], g["eta"])
    assert math.isclose(t_l, g["t_uniform_num"] / g["t_uniform_den"], rel_tol=1e-15)
    assert schedule.guidance_off_step(g["steps"], g["eta"], g["cutoff"]) == g["turning_step"]


def test_eta3_turning_point_matches_default_cfg_off_ratio():
    hp = _golden("default_hyperparameters.json")
    assert schedule.guidance_off_step(25, 3.0, 0.5) == schedule.ceil_ratio(25, hp["rho_cfg_off"]) == 19


def test_shift_properties():
    for eta in (1.0, 2.0, 3.0, 5.5):
        assert schedule.shift_time(0.0, eta) == 0.0
        assert schedule.shift_time(1.0, eta) == 1.0
        for t in np.linspace(0.01, 0.99, 23):
            assert math.isclose(schedule.unshift_time(schedule.shift_time(t, eta), eta), t, rel_tol=1e-12)
            if eta > 1:
                assert schedule.shift_time(t, eta) > t          # biases steps toward high t
    for t in np.linspace(0, 1, 11):
        assert schedule.shift_time(t, 1.0) == t
    assert schedule.shift_time(0.5, 3.0) == 0.75


def test_time_grid_endpoints_and_monotone():
    for T, eta in ((10, 1.0), (25, 3.0)):
        g = schedule.time_grid(T, eta)
        assert len(g) == T + 1 and g[0] == 1.0 and g[-1] == 0.0
        assert all(a > b for a, b in zip(g, g[1:]))
    g = schedule.time_grid(10, 1.0)
    assert all(math.isclose(g[k], 1 - k / 10) for k in range(11))


def test_phase_table_at_defaults():
    hp = _golden("default_hyperparameters.json")
    T, N = 25, 4096
    ka = schedule.anchor_step(T, hp["rho_a"])
    assert ka == 5
    got = [schedule.phase_quota(k, T, N, 1234, hp["rho_a"], hp["rho_cfg_off"], hp["xi"], hp["f_corr"])
           for k in range(1, T + 1)]
    fixed = int(N * 7 // 10)
    want = [0] * 5 + [1234] * 13 + [fixed, fixed, 0, fixed, fixed, 0, fixed]
    assert got == want


def test_phase3_correction_extremes():
    T, N = 25, 100
    q = lambda k, f: schedule.phase_quota(k, T, N, 7, 0.2, 0.75, 0.7, f)
    assert [q(k, 1) for k in range(19, 26)] == [0] * 7        # f_corr = 1: full sampling
    assert [q(k, 0) for k in range(19, 26)] == [70] * 7       # f_corr = 0: never corrected
    assert [q(k, 2) for k in range(19, 26)] == [70, 0, 70, 0, 70, 0, 70]


def test_pcsc_curve_is_log_linear_and_anchored():
    sigma, mu, ka = 5000.0, -0.07, 5
    assert schedule.pcsc_predicted_change(ka, sigma, mu, ka) == sigma
    vals = [schedule.pcsc_predicted_change(k, sigma, mu, ka) for k in range(5, 26)]
    slopes = np.diff(np.log(vals))
    assert np.allclose(slopes, mu, atol=1e-12)
    assert math.isclose(vals[-1] / sigma, math.exp(-0.07 * 20))


def test_pcsc_quota_bound_and_clamp():
    N = 4096
    # predicted change 6400 voxels, gamma 64 -> 100 active -> 3996 cached
    assert schedule.pcsc_quota(5, N, 6400.0, -0.07, 5, 64.0) == N - 100
    # fractional bound rounds down (the quota is an upper bound)
    q = schedule.pcsc_quota(6, N, 6400.0, -0.07, 5, 64.0)
    assert q == math.floor(N - 6400.0 * math.exp(-0.07) / 64.0)
    assert schedule.pcsc_quota(5, N, 1e9, -0.07, 5, 64.0) == 0
    assert schedule.pcsc_quota(5, N, 0.0, -0.07, 5, 64.0) == N
    qs = [schedule.pcsc_quota(k, N, 2e5, -0.07, 5, 64.0) for k in range(5, 26)]
    assert all(a <= b for a, b in zip(qs, qs[1:]))       # mu < 0: quota never shrinks


@pytest.mark.parametrize("case", _golden("flops_simplified.json")["cases"])
def test_flops_itemised_terms_sum_to_printed_totals(case):
    B, N, D, H, Nc = case["B"], case["N"], case["D"], case["H"], case["Nc"]
    t = flops.block_terms(B, N, D, H, Nc, D)
    sa = t["sa_qkv"] + t["sa_qk"] + t["sa_softmax"] + t["sa_av"] + t["sa_out"]
    ca = t["ca_q"] + t["ca_kv"] + t["ca_qk"] + t["ca_softmax"] + t["ca_av"] + t["ca_out"]
    mlp = t["fc1"] + t["act"] + t["fc2"]
    assert math.isclose(sa, 8 * B * N * D * D + 4 * B * N * N * D + 5 * B * H * N * N)
    assert math.isclose(ca, 4 * B * N * D * D + 4 * B * Nc * D * D + 4 * B * N * Nc * D + 5 * B * H * N * Nc)
    assert math.isclose(mlp, 16 * B * N * D * D + 20 * B * N * D)


def test_flops_contraction_terms_match_executed_matmuls(monkeypatch):
    cfg = synth.ModelConfig(grid=3, width=16, depth=2, heads=4, cond_tokens=5, cond_width=12, dtype="f32")
    W = synth.make_weights(cfg, seed=1)
    model = dit.Model(cfg, W)
    counted = []
    real = dit._matmul

    def counting(a, b):
        m = 1 if a.ndim == 1 else a.shape[0]
        counted.append(2 * m * a.shape[-1] * b.shape[-1])
        return real(a, b)

    monkeypatch.setattr(dit, "_matmul", counting)
    rng = np.random.default_rng(0)
    n = 11
    idx = np.sort(rng.choice(cfg.tokens, n, replace=False))
    model.forward(rng.standard_normal((n, 8)), idx, 0.4, rng.standard_normal((5, 12)))
    d = cfg.width
    outside_blocks = 2 * 256 * d + 2 * d * d + 2 * n * 8 * d + 2 * n * d * 8   # temb MLP, embed, output
    t = flops.block_terms(1, n, d, cfg.heads, cfg.cond_tokens, cfg.cond_width)
    contraction = sum(t[k] for k in ("sa_qkv", "sa_qk", "sa_av", "sa_out", "ca_q", "ca_kv", "ca_qk",
                                     "ca_av", "ca_out", "fc1", "fc2"))
    mod_matmul = 2 * d * 6 * d
    assert sum(counted) == outside_blocks + cfg.depth * (contraction + mod_matmul)


def test_flops_at_trellis_shape():
    # 24 blocks, width 1024, 16 heads, 1374 x 1024 condition tokens, 4096 tokens
    f = flops.forward_flops(synth.TRELLIS16, 4096)
    assert math.isclose(f / 1e12, 5.2744894464, rel_tol=1e-12)


# ---------------------------------------------------------------- full plan

def _cached(pattern_plan):
    return [1 if c > 0 else 0 for c in pattern_plan]


def test_plan_defaults_tau3_worked_by_hand():
    # T = 25 with the default hyperparameters (rho_a 0.2, rho_CFG-OFF 0.75,
    # xi 0.7, f_corr 3, tau 3, cycle reading): Phase 1 is k = 1..5, Phase 2
    # k = 6..18, Phase 3 k = 19..25 with correction steps at k = 21 and 24.
    # Worked by hand from Algorithm 1: two cached steps, then a refresh.
    p = schedule.plan(25, 4096, sigma=100.0, tau=3)
    want = [0] * 5 + [1, 1, 0, 1, 1, 0, 1, 1, 0, 1, 1, 0, 1] + [1, 0, 0, 1, 1, 0, 1]
    assert _cached(p) == want
    # Phase 3 cached steps use floor(4096 * 0.7) = 2867
    assert p[18] == p[21] == p[22] == p[24] == 2867


def test_plan_tau_extremes():
    kw = dict(steps=25, n_tokens=4096, sigma=50.0)
    assert schedule.plan(tau=1, **kw) == [0] * 25                      # cycle reading: never caches
    lit = _cached(schedule.plan(tau=1, reading=schedule.TAU_LITERAL, **kw))
    assert all(not (a and b) for a, b in zip(lit, lit[1:]))            # literal: never two cached in a row
    assert sum(lit) > 0
    base = schedule.plan(tau=0, **kw)
    assert schedule.plan(tau=26, **kw) == base                         # a limit beyond T changes nothing
    assert schedule.plan(tau=26, reading=schedule.TAU_LITERAL, **kw) == base


def test_plan_literal_is_cycle_shifted_by_one():
    # literal tau reads as the cycle reading with tau + 1 (both count the same run)
    for tau in (1, 2, 3, 5, 8):
        for f_corr in (0, 3):
            kw = dict(steps=50, n_tokens=32768, sigma=900.0, mu=-0.05, gamma_up=4.0, f_corr=f_corr)
            assert (schedule.plan(tau=tau, reading=schedule.TAU_LITERAL, **kw)
                    == schedule.plan(tau=tau + 1, **kw))


def test_plan_without_tau_is_phase_rule_with_pcsc():
    T, N, sigma, mu, g = 25, 4096, 300.0, -0.07, 2.0
    p = schedule.plan(T, N, sigma, mu=mu, gamma_up=g)
    ka = schedule.anchor_step(T)
    for k in range(1, T + 1):
        if k <= ka or k == 21 or k == 24:
            assert p[k - 1] == 0
        elif k < 19:
            # Eq. (5) closed form at the step index
            assert p[k - 1] == math.floor(N - sigma * math.exp(mu * (k - ka)) / g)
        else:
            assert p[k - 1] == 2867


def test_plan_runs_never_exceed_the_limit():
    import itertools
    for tau, reading in itertools.product((2, 3, 4, 7), (schedule.TAU_CYCLE, schedule.TAU_LITERAL)):
        c = _cached(schedule.plan(40, 512, sigma=20.0, f_corr=0, tau=tau, reading=reading))
        limit = tau - 1 if reading == schedule.TAU_CYCLE else tau
        run = longest = 0
        for v in c:
            run = run + 1 if v else 0
            longest = max(longest, run)
        assert longest == limit          # Phase 2/3 are long enough to reach the limit
