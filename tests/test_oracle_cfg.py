"""Pins for the oracle's guided (classifier-free guidance) step and the
guidance interval.

* guidance arithmetic: hand-worked float32 values, w = 0 returns the
  conditional velocity bit for bit, equal passes return it up to rounding;
* two straight-line fields toward different end points: the guided field is
  the straight line toward (1 + w) y0_c - w y0_u, so Euler and caching stay
  exact and any quota schedule lands there (a wrong weight or sign lands
  elsewhere);
* both passes of a guided step see the same active set and the same inputs;
* the guidance interval t in [0.5, 1] ends at the supplement's turning steps
  (eta = 1, 2, 3 at 25 steps: 13, 17, 19), and [0, 1] guides every step.
"""
import numpy as np

from oracle import sampler, schedule

F32 = np.float32


def test_guide_hand_worked():
    # (1 + 2) * 1.5 - 2 * 0.25 = 4.5 - 0.5 = 4
    assert sampler.guide(np.array([1.5], F32), np.array([0.25], F32), 2.0)[0] == F32(4.0)
    # w = 0.5: 1.5 * 2 - 0.5 * 3 = 1.5; negative values
    g = sampler.guide(np.array([2.0, -1.0], F32), np.array([3.0, 1.0], F32), 0.5)
    assert g.tolist() == [1.5, -2.0]
    assert g.dtype == F32


def test_guide_weight_zero_and_equal_passes():
    rng = np.random.default_rng(0)
    vc = rng.standard_normal((100, 8)).astype(F32)
    vu = rng.standard_normal((100, 8)).astype(F32)
    assert np.array_equal(sampler.guide(vc, vu, 0.0).view(np.uint32), vc.view(np.uint32))
    for w in (0.5, 3.0, 7.5):
        g = sampler.guide(vc, vc, w)
        # (1 + w) v - w v = v exactly in real arithmetic; three roundings apart in float32
        bound = (2.0 * w + 1.0) * np.abs(vc).astype(np.float64) * 2.0 ** -23 + 1e-30
        assert np.all(np.abs(g.astype(np.float64) - vc) <= bound)


def test_guide_rounds_each_operation():
    # the product (1 + w) v_c is rounded before the difference: choose values
    # where a fused multiply-add would give a different float32
    rng = np.random.default_rng(5)
    vc = (1.0 + rng.random(4000)).astype(F32)
    vu = (1.0 + rng.random(4000)).astype(F32)
    w = 0.3
    a, ws = F32(1.3), F32(0.3)
    two_step = (a * vc) - (ws * vu)
    fused = (a.astype(np.float64) * vc - (ws * vu).astype(np.float64)).astype(F32)
    assert not np.array_equal(two_step, fused)
    assert np.array_equal(sampler.guide(vc, vu, w), two_step)


def _straight_field(y0):
    def v(b, x_act, idx, t):
        return (x_act.astype(np.float64) - y0[b][idx]) / t
    return v


def test_guided_straight_lines_reach_the_guided_end_point():
    rng = np.random.default_rng(1)
    B, N, T = 2, 64, 12
    y0c = rng.standard_normal((B, N, 8))
    y0u = rng.standard_normal((B, N, 8))
    for w in (0.5, 3.0):
        y_star = (1.0 + w) * y0c - w * y0u
        y1 = rng.standard_normal((B, N, 8))
        times = schedule.time_grid(T, 3.0)
        quotas = np.zeros((T, B), np.int64)
        quotas[2:, 0] = rng.integers(0, N + 1, size=T - 2)
        quotas[2:, 1] = N // 4
        st = sampler.sample(y1.astype(F32), _straight_field(y0c), times, quotas,
                            uncond=_straight_field(y0u), w=w)
        scale = np.max(np.abs(y_star))
        assert np.max(np.abs(st.x - y_star)) < 2e-5 * scale * (1 + 2 * w)
        # the conditional end point alone is not reached
        assert np.max(np.abs(st.x - y0c)) > 0.1


def test_both_passes_share_the_active_set():
    rng = np.random.default_rng(2)
    B, N = 2, 32
    calls = []

    def field(tag, y0):
        def v(b, x_act, idx, t):
            calls.append((tag, b, idx.copy(), x_act.copy()))
            return (x_act.astype(np.float64) - y0[b][idx]) / t + rng.standard_normal(x_act.shape) * 0.01
        return v

    y0 = rng.standard_normal((B, N, 8))
    st = sampler.State.start(rng.standard_normal((B, N, 8)).astype(F32))
    sampler.step(st, field("c", y0), 1.0, 0.9, [0, 0], uncond=field("u", -y0), w=2.0)
    sampler.step(st, field("c", y0), 0.9, 0.8, [0, 0], uncond=field("u", -y0), w=2.0)
    calls.clear()
    rec = sampler.step(st, field("c", y0), 0.8, 0.7, [10, 25], uncond=field("u", -y0), w=2.0)
    assert [c[0] for c in calls] == ["c", "u", "c", "u"]
    for b in range(B):
        c, u = calls[2 * b], calls[2 * b + 1]
        assert c[1] == u[1] == b
        assert np.array_equal(c[2], u[2]) and np.array_equal(c[2], rec.active[b])
        assert np.array_equal(c[3], u[3])
        assert len(rec.active[b]) == N - [10, 25][b]
        assert np.array_equal(rec.v_active[b], sampler.guide(rec.v_cond[b], rec.v_uncond[b], 2.0))


def test_unguided_steps_of_a_guided_run_use_the_conditional_pass_only():
    rng = np.random.default_rng(3)
    B, N, T = 1, 16, 6
    y0c = rng.standard_normal((B, N, 8))
    times = schedule.time_grid(T, 1.0)
    x_T = rng.standard_normal((B, N, 8)).astype(F32)
    quotas = np.zeros((T, B), np.int64)
    recs = []
    sampler.sample(x_T, _straight_field(y0c), times, quotas, records=recs,
                   uncond=_straight_field(-y0c), w=1.0, guided=[True, True, True, False, False, False])
    assert [len(r.v_uncond) for r in recs] == [1, 1, 1, 0, 0, 0]


def test_guidance_interval_ends_at_the_turning_steps():
    for eta, last in ((1.0, 13), (2.0, 17), (3.0, 19)):
        g = schedule.guided_steps(schedule.time_grid(25, eta))
        k_last = max(k + 1 for k, on in enumerate(g) if on)
        assert k_last == last == schedule.guidance_off_step(25, eta, 0.5)
        assert all(g[:k_last]) and not any(g[k_last:])
    assert all(schedule.guided_steps(schedule.time_grid(25, 3.0), lo=0.0))
    assert schedule.cfg_active(0.5) and schedule.cfg_active(1.0) and not schedule.cfg_active(0.4999)
