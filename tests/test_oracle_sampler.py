"""Pins for the oracle's sampler step (Algorithm 1, state update; Sec. 3.1).

* a straight-line velocity field makes Euler exact *and* caching exact, so any
  quota schedule and any selection must land on the path's end point;
* quota 0 equals the definition x - (t - t') * G(x) with every token active;
* cached rows carry the cached velocity bit for bit, so their acceleration
  at the next step is exactly 0 (caching is sticky);
* quota N skips the transformer and extrapolates with the cached velocity.
"""
import numpy as np

from oracle import dit, sampler, schedule, ssc
from paper_2511_22533_amd import synth

F32 = np.float32


def _straight_field(y0):
    def v(b, x_act, idx, t):
        return (x_act.astype(np.float64) - y0[b][idx]) / t
    return v


def test_straight_line_field_any_quota_reaches_endpoint():
    rng = np.random.default_rng(0)
    B, N = 2, 64
    y0 = rng.standard_normal((B, N, 8))
    y1 = rng.standard_normal((B, N, 8))
    for eta in (1.0, 3.0):
        times = schedule.time_grid(12, eta)
        # start exactly on the path at t_1 = 1: y_1 = (1 - 1) y0 + 1 * y1
        x_T = y1.astype(F32)
        y0_eff = y0
        quotas = np.zeros((12, B), np.int64)
        quotas[1:, 0] = rng.integers(0, N + 1, size=11)
        quotas[1:, 1] = N // 2
        st = sampler.sample(x_T, _straight_field(y0_eff), times, quotas)
        # the oracle's float32 state drifts only by rounding
        assert np.max(np.abs(st.x - y0)) < 1e-4
        # every cached velocity is a copy of one computed earlier on the same path
        v_exact = (y1 - y0)
        assert np.max(np.abs(st.v_cache - v_exact)) < 1e-3


def test_quota_zero_is_the_full_step_definition():
    cfg = synth.ModelConfig(grid=3, width=16, depth=2, heads=4, cond_tokens=5, cond_width=8, dtype="f32")
    W = synth.make_weights(cfg, seed=3, scale=0.2)
    model = dit.Model(cfg, W)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((1, cfg.tokens, 8)).astype(F32)
    cond = rng.standard_normal((1, cfg.cond_tokens, cfg.cond_width)).astype(F32)
    st = sampler.State.start(x)
    st.v_cache[:] = rng.standard_normal(st.v_cache.shape).astype(F32)
    st.v_prev[:] = rng.standard_normal(st.v_prev.shape).astype(F32)
    t, tn = 0.7, 0.55
    v_full = model.forward(x[0], np.arange(cfg.tokens), t, cond[0]).astype(F32)
    want_x = x[0] - F32(t - tn) * v_full
    old_cache = st.v_cache.copy()
    rec = sampler.step(st, sampler.model_velocity(model, cond), t, tn, [0])
    assert np.array_equal(st.x[0], want_x)
    assert np.array_equal(st.v_cache[0], v_full)
    assert np.array_equal(st.v_prev, old_cache)
    assert rec.scores[0] is None and np.array_equal(rec.active[0], np.arange(cfg.tokens))


def test_cached_rows_bit_identical_and_sticky():
    cfg = synth.ModelConfig(grid=4, width=16, depth=1, heads=2, cond_tokens=5, cond_width=8, dtype="f32")
    W = synth.make_weights(cfg, seed=4, scale=0.2)
    model = dit.Model(cfg, W)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((1, cfg.tokens, 8)).astype(F32)
    cond = rng.standard_normal((1, cfg.cond_tokens, cfg.cond_width)).astype(F32)
    vel = sampler.model_velocity(model, cond)
    st = sampler.State.start(x)
    sampler.step(st, vel, 1.0, 0.9, [0])
    sampler.step(st, vel, 0.9, 0.8, [0])
    before = st.v_cache.copy()
    rec = sampler.step(st, vel, 0.8, 0.7, [40])
    active = rec.active[0]
    cached = np.setdiff1d(np.arange(cfg.tokens), active)
    assert len(cached) == 40 and len(active) == cfg.tokens - 40
    assert np.array_equal(st.v_cache[0][cached].view(np.uint32), before[0][cached].view(np.uint32))
    assert np.array_equal(st.v_prev, before)
    acc = ssc.acceleration(st.v_cache[0], st.v_prev[0])
    assert np.all(acc[cached] == 0)
    assert np.all(acc[active] > 0)


def test_quota_n_skips_forward():
    calls = []

    def vel(b, x_act, idx, t):
        calls.append(len(idx))
        return np.zeros((len(idx), 8))

    rng = np.random.default_rng(3)
    x = rng.standard_normal((1, 27, 8)).astype(F32)
    st = sampler.State.start(x)
    st.v_cache[:] = rng.standard_normal(st.v_cache.shape).astype(F32)
    vc = st.v_cache.copy()
    sampler.step(st, vel, 0.5, 0.25, [27])
    assert calls == []
    assert np.array_equal(st.x, x - F32(0.25) * vc)
    assert np.array_equal(st.v_cache, vc)


def test_euler_step_size_rounded_once():
    # dt is t - t' in float64 rounded once to float32
    x = np.ones((1, 1, 8), F32)
    st = sampler.State.start(x)

    def vel(b, x_act, idx, t):
        return np.ones((len(idx), 8))

    t, tn = 0.98630136986301364, 0.9726027397260274
    sampler.step(st, vel, t, tn, [0])
    assert np.all(st.x == F32(1.0) - F32(t - tn))
