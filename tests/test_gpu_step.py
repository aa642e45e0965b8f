"""GPU parity of whole cached steps and trajectories, through the C ABI.

Per step (teacher-forced on the GPU's own pre-step state):
* the selection equals the oracle's selection on the downloaded caches, bit
  for bit (indices and position map);
* the fresh velocities equal the oracle transformer on the same active set
  within 1e-4 (f32 build) / 2e-2 (bf16) max-rel, per sample;
* cached rows carry the stored velocity bit for bit, the Euler update and the
  cache rotation are bit-exact given the merged velocity;
Trajectories: final latents within 3e-2 relative L2 of the free-running oracle.
Also: quota 0 equals the full step bit for bit, checkpoint export/import
resumes bit-identically, and repeated runs are bit-identical.
"""
import numpy as np
import pytest

from helpers import Pair, depth_variant, max_rel, oracle_selection, rel_l2, say, to_dev
from oracle import dit, sampler, schedule
from paper_2511_22533_amd import synth

pytestmark = pytest.mark.gpu

F32 = np.float32


def _gpu_step(torch, pair, x_dev, t, tn, n_cache, w=None):
    before = pair.state.tensors()
    torch.cuda.synchronize()
    vc = before["v_cache"].cpu().numpy()
    vp = before["v_prev"].cpu().numpy()
    x_before = x_dev.cpu().numpy()
    if w is not None:
        pair.state.guided_step(x_dev, t, tn, n_cache if any(n_cache) else None, w)
    elif any(n_cache):
        pair.state.cached_step(x_dev, t, tn, n_cache)
    else:
        pair.state.full_step(x_dev, t, tn)
    torch.cuda.synchronize()
    after = pair.state.tensors()
    if any(n_cache):
        idx, pos = after["idx_active"].cpu().numpy(), after["pos"].cpu().numpy()
    else:   # a step without selection leaves no index views
        assert after["idx_active"] is None and after["pos"] is None
        idx = pos = None
    return dict(vc=vc, vp=vp, x0=x_before, x1=x_dev.cpu().numpy(), idx=idx,
                pos=pos, vact=after["v_act"].cpu().numpy(), off=after["act_off"],
                vnew=after["v_cache"].cpu().numpy(), vold=after["v_prev"].cpu().numpy())


def _check_step(pair, r, t, tn, n_cache, vel_tol, omega=0.7):
    B, N = pair.B, pair.cfg.tokens
    ref = oracle_selection(r["vc"], r["vp"], n_cache, omega)
    dt = F32(t - tn)
    worst = 0.0
    for b in range(B):
        active = ref[b][1]
        lo, hi = r["off"][b], r["off"][b + 1]
        assert hi - lo == N - n_cache[b]
        if any(n_cache):
            assert np.array_equal(r["idx"][lo:hi], active), f"selection sample {b}"
            want_pos = np.full(N, -1)
            want_pos[active] = lo + np.arange(hi - lo)
            assert np.array_equal(r["pos"][b], want_pos)
        # merged velocity: cached rows bit-identical, active rows from v_act
        cached = np.setdiff1d(np.arange(N), active)
        assert np.array_equal(r["vnew"][b][cached].view(np.uint32), r["vc"][b][cached].view(np.uint32))
        assert np.array_equal(r["vnew"][b][active].view(np.uint32), r["vact"][lo:hi].view(np.uint32))
        assert np.array_equal(r["vold"][b].view(np.uint32), r["vc"][b].view(np.uint32))
        # Euler, bit-exact given the merged velocity
        assert np.array_equal(r["x1"][b].view(np.uint32), (r["x0"][b] - dt * r["vnew"][b]).view(np.uint32))
        # fresh velocities vs the oracle transformer on the same tokens
        if hi > lo:
            want = pair.oracle.forward(r["x0"][b][active], active, t, pair.cond[b])
            err = max_rel(r["vact"][lo:hi], want)
            worst = max(worst, err)
            assert err < vel_tol, f"sample {b}: velocity max-rel {err}"
    return worst


def _check_guided_step(pair, r, t, tn, n_cache, w, vel_tol, omega=0.7):
    """A guided step: selection bit-exact on the guided caches; each pass's
    velocities against the oracle transformer with its own condition; the
    guided merge bit-exact given the two passes; cached rows, rotation and
    Euler bit-exact."""
    B, N = pair.B, pair.cfg.tokens
    ref = oracle_selection(r["vc"], r["vp"], n_cache, omega)
    dt = F32(t - tn)
    rows = r["off"][-1]
    assert r["vact"].shape[0] == 2 * rows
    v_c, v_u = r["vact"][:rows], r["vact"][rows:]
    guided = sampler.guide(v_c, v_u, w)
    worst = 0.0
    for b in range(B):
        active = ref[b][1]
        lo, hi = r["off"][b], r["off"][b + 1]
        assert hi - lo == N - n_cache[b]
        if any(n_cache):
            assert np.array_equal(r["idx"][lo:hi], active), f"selection sample {b}"
        cached = np.setdiff1d(np.arange(N), active)
        assert np.array_equal(r["vnew"][b][cached].view(np.uint32), r["vc"][b][cached].view(np.uint32))
        assert np.array_equal(r["vnew"][b][active].view(np.uint32), guided[lo:hi].view(np.uint32)), f"guide {b}"
        assert np.array_equal(r["vold"][b].view(np.uint32), r["vc"][b].view(np.uint32))
        assert np.array_equal(r["x1"][b].view(np.uint32), (r["x0"][b] - dt * r["vnew"][b]).view(np.uint32))
        if hi > lo:
            for got, c in ((v_c[lo:hi], pair.cond[b]), (v_u[lo:hi], pair.uncond[b])):
                want = pair.oracle.forward(r["x0"][b][active], active, t, c)
                err = max_rel(got, want)
                worst = max(worst, err)
                assert err < vel_tol, f"sample {b}: velocity max-rel {err}"
    return worst


@pytest.fixture(scope="module")
def torch():
    import torch as t
    from paper_2511_22533_amd import f3c
    f3c.lib()
    return t


def test_tiny_f32_trajectory(torch):
    w = synth.WORKLOADS["tiny_f32"]
    pair = Pair(w.model, w.batch)
    times = schedule.time_grid(w.steps, w.shift)
    quotas = synth.quota_schedule(w)
    x = to_dev(pair.x_T)
    for k in range(w.steps):
        say("tiny_f32 step", k + 1, quotas[k].tolist())
        r = _gpu_step(torch, pair, x, times[k], times[k + 1], quotas[k].tolist())
        _check_step(pair, r, times[k], times[k + 1], quotas[k].tolist(), 1e-4)
    final = x.cpu().numpy()
    ref = sampler.sample(pair.x_T, pair.velocity(), times, quotas)
    assert rel_l2(final, ref.x) < 3e-2
    assert rel_l2(final, ref.x) < 1e-4


def test_tiny_f32_amplified_sublayers(torch):
    # larger weights: attention, cross-attention and MLP all move h by O(1)
    cfg = synth.TINY
    pair = Pair(cfg, 2, seed=5, scale=0.08)
    x = to_dev(pair.x_T)
    times = schedule.time_grid(7, 1.0)
    # the last two steps: one sample's active set empty, then every sample's (no transformer rows at all)
    for k, q in enumerate([[0, 0], [0, 0], [100, 300], [256, 0], [511, 1], [512, 200], [512, 512]]):
        say("tiny amplified step", k + 1, q)
        r = _gpu_step(torch, pair, x, times[k], times[k + 1], q)
        _check_step(pair, r, times[k], times[k + 1], q, 1e-4)


def test_quota_zero_equals_full_step_and_determinism(torch):
    cfg = synth.TINY
    a = Pair(cfg, 2, seed=1)
    b = Pair(cfg, 2, seed=1)
    xa, xb = to_dev(a.x_T), to_dev(b.x_T)
    say("quota zero vs full")
    a.state.full_step(xa, 1.0, 0.9)
    b.state.cached_step(xb, 1.0, 0.9, [0, 0])
    a.state.full_step(xa, 0.9, 0.8)
    b.state.cached_step(xb, 0.9, 0.8, [0, 0])
    a.state.cached_step(xa, 0.8, 0.7, [100, 200])
    b.state.cached_step(xb, 0.8, 0.7, [100, 200])
    torch.cuda.synchronize()
    assert torch.equal(xa, xb)
    assert np.array_equal(a.state.export(), b.state.export())


def test_checkpoint_resume_bit_identical(torch):
    cfg = synth.TINY
    pair = Pair(cfg, 1, seed=3)
    times = schedule.time_grid(8, 1.0)
    q = [[0], [0], [0], [100], [200], [300], [400], [500]]
    x = to_dev(pair.x_T)
    say("checkpoint")
    for k in range(4):
        pair.state.cached_step(x, times[k], times[k + 1], q[k])
    snap_x = x.clone()
    snap = pair.state.export()
    for k in range(4, 8):
        pair.state.cached_step(x, times[k], times[k + 1], q[k])
    torch.cuda.synchronize()
    first = x.clone()
    pair.state.import_(snap)
    x.copy_(snap_x)
    for k in range(4, 8):
        pair.state.cached_step(x, times[k], times[k + 1], q[k])
    torch.cuda.synchronize()
    assert torch.equal(first, x)


def test_two_states_on_two_streams_match_sequential(torch):
    """Every per-step buffer lives in the state and the model holds only
    weights, so two states of one model stepping on two streams at once
    (launches interleaved, nothing orders one stream against the other) give
    bit for bit what they give stepping on one stream."""
    from paper_2511_22533_amd import f3c
    cfg = depth_variant(synth.TRELLIS16, 2)
    model = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    states = [f3c.State(model, 1) for _ in range(2)]
    conds = [to_dev(synth.make_cond(cfg, 1, seed_base=2000 + 10 * i)) for i in range(2)]
    x_T = [synth.make_noise(cfg, 1, seed_base=1000 + 10 * i) for i in range(2)]
    times = schedule.time_grid(6, 3.0)
    quotas = [[0], [0], [1024], [2048], [3000], [3276]]

    def run(streams):
        xs = [to_dev(x) for x in x_T]
        torch.cuda.synchronize()
        for st, cond, s in zip(states, conds, streams):
            st.reset(s)
            st.set_cond(cond, s)
        for k, q in enumerate(quotas):
            for st, x, s in zip(states, xs, streams):
                st.cached_step(x, times[k], times[k + 1], q, s)
        torch.cuda.synchronize()
        return [x.cpu() for x in xs]

    say("two states, one stream")
    one = torch.cuda.current_stream().cuda_stream
    seq = run([one, one])
    say("two states, two streams")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    par = run([s1.cuda_stream, s2.cuda_stream])
    assert all(torch.equal(a, b) for a, b in zip(seq, par))
    assert not torch.equal(seq[0], seq[1])


def test_graph_capture_of_a_trajectory_replays_exactly(torch):
    """A whole trajectory (state reset, condition K/V, modulation plan, cached
    steps) captured in one HIP graph: the library records only kernels on the caller's stream
    (the reset zeroes the caches with a kernel, not a memset node), so every
    replay, with eager work and synchronisations in between, gives the eager
    trajectory bit for bit."""
    from paper_2511_22533_amd import f3c
    cfg = depth_variant(synth.TRELLIS16, 2)
    model = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    state = f3c.State(model, 1)
    cond = to_dev(synth.make_cond(cfg, 1))
    x_T = to_dev(synth.make_noise(cfg, 1))
    times = schedule.time_grid(6, 3.0)
    quotas = [[0], [0], [1024], [2048], [3000], [3276]]

    def trajectory(x):
        state.reset()
        state.set_cond(cond)
        state.plan_times(times[:-1])
        for k, q in enumerate(quotas):
            state.cached_step(x, times[k], times[k + 1], q)

    x = x_T.clone()
    say("eager trajectory")
    trajectory(x)
    torch.cuda.synchronize()
    eager = x.clone()
    xg = x_T.clone()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    say("capture")
    with torch.cuda.graph(graph):
        trajectory(xg)
    torch.cuda.synchronize()
    for rep in range(3):
        xg.copy_(x_T)
        junk = torch.arange(1 << 20, device="cuda", dtype=torch.float32).mul_(0.5).sum()
        torch.cuda.synchronize()
        say("replay", rep)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(xg, eager), f"replay {rep}"
        assert float(junk) > 0
    # the eager path still works after capture, and still agrees
    x2 = x_T.clone()
    trajectory(x2)
    torch.cuda.synchronize()
    assert torch.equal(x2, eager)


_PLAN_CFGS = [synth.TINY, synth.ModelConfig(grid=4, width=1024, depth=3, heads=16, cond_tokens=8, cond_width=64,
                                            dtype="bf16")]


@pytest.mark.parametrize("cfg", _PLAN_CFGS, ids=["tiny_f32", "w1024_bf16"])
def test_modulation_plan_equals_per_step_modulation_bitwise(torch, cfg):
    """The planned modulation of 11 times (one pass of 8 times, one of 3)
    equals the per-time modulation entry bit for bit, and the oracle's
    modulation within the per-step tolerance."""
    from paper_2511_22533_amd import f3c
    W = synth.make_weights(cfg, seed=2, scale=0.05)
    m = f3c.Model(cfg).load(W)
    st = f3c.State(m, 1)
    times = [float(t) for t in schedule.time_grid(10, 3.0)[:-1]] + [0.5, 0.0]
    say("plan", cfg.dtype, len(times), "times")
    st.plan_times(times)
    torch.cuda.synchronize()
    R = cfg.depth * 6 * cfg.width
    plan = st.plan_buf[: len(times) * R * 4].view(torch.float32).reshape(len(times), R).cpu().numpy()
    om = dit.Model(cfg, W)
    tol = 1e-4 if cfg.dtype == "f32" else 5e-3
    for i, t in enumerate(times):
        want = m.modulation(t).cpu().numpy().ravel()
        assert np.array_equal(plan[i].view(np.uint32), want.view(np.uint32)), f"time {i} ({t})"
    assert max_rel(plan[3], om.modulation(times[3]).ravel()) < tol


def test_planned_trajectory_is_bit_identical(torch):
    """A trajectory whose step times are planned (all of them, some of them,
    then the plan cleared) gives the unplanned trajectory bit for bit; a step
    at a planned time launches no modulation kernels."""
    from paper_2511_22533_amd import f3c
    cfg = depth_variant(synth.TRELLIS16, 2)
    model = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    state = f3c.State(model, 1)
    cond = to_dev(synth.make_cond(cfg, 1))
    x_T = to_dev(synth.make_noise(cfg, 1))
    times = [float(t) for t in schedule.time_grid(6, 3.0)]
    quotas = [[0], [0], [1024], [2048], [3000], [3276]]

    def trajectory():
        x = x_T.clone()
        state.reset()
        state.set_cond(cond)
        state.profile(["mod"])
        state.profile_reset()
        for k, q in enumerate(quotas):
            if any(q):
                state.cached_step(x, times[k], times[k + 1], q)
            else:
                state.full_step(x, times[k], times[k + 1])
        torch.cuda.synchronize()
        n_mod = state.profile_read()["mod"]["launches"]
        state.profile(False)
        return x, n_mod

    say("unplanned trajectory")
    ref, n = trajectory()
    assert n == 6
    for plan, mod_calls in ((times[:-1], 0), (times[1:4:2], 4), ([], 6)):
        say("planned", len(plan), "times")
        state.plan_times(plan)
        x, n = trajectory()
        assert n == mod_calls
        assert torch.equal(x, ref), f"plan of {len(plan)} times"


def test_planned_guided_trajectory_is_bit_identical(torch):
    """Guided steps read the planned modulation for both passes: a guided
    trajectory with its times planned equals the unplanned one bit for bit."""
    from paper_2511_22533_amd import f3c
    cfg = depth_variant(synth.TRELLIS16, 2)
    model = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    state = f3c.State(model, 2, guided=True)
    cond = to_dev(synth.make_cond(cfg, 2))
    uncond = to_dev(synth.make_uncond(cfg, 2))
    x_T = to_dev(synth.make_noise(cfg, 2))
    times = [float(t) for t in schedule.time_grid(4, 3.0)]
    quotas = [None, [1000, 3000], [2048, 0], [3276, 3276]]

    def trajectory():
        x = x_T.clone()
        state.reset()
        state.set_cond(cond)
        state.set_uncond(uncond)
        for k, q in enumerate(quotas):
            state.guided_step(x, times[k], times[k + 1], q, 3.0)
        torch.cuda.synchronize()
        return x

    say("guided, unplanned")
    ref = trajectory()
    state.plan_times(times[:-1])
    say("guided, planned")
    assert torch.equal(trajectory(), ref)


def test_modulation_plan_validation(torch):
    """Bad plans are refused before anything is enqueued and keep the previous
    plan; the binding reuses its buffer."""
    import ctypes
    from paper_2511_22533_amd import f3c
    cfg = synth.TINY
    m = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    st = f3c.State(m, 1)
    st.set_cond(to_dev(synth.make_cond(cfg, 1)))
    st.plan_times([0.9, 0.8])
    buf = st.plan_buf
    L = f3c.lib()
    need = ctypes.c_size_t()
    assert L.f3c_plan_bytes(m.h, 2, ctypes.byref(need)) == f3c.F3C_OK
    R = cfg.depth * 6 * cfg.width

    def a256(v):
        return (v + 255) // 256 * 256
    assert need.value == a256(2 * R * 4) + a256(2 * 2 * cfg.width * 4)
    assert L.f3c_plan_bytes(m.h, -1, ctypes.byref(need)) == f3c.F3C_EINVAL
    assert L.f3c_plan_bytes(m.h, 1025, ctypes.byref(need)) == f3c.F3C_EINVAL
    ptr, nb = buf.data_ptr(), buf.numel()
    t2 = (ctypes.c_double * 2)(0.7, float("nan"))
    ok = (ctypes.c_double * 2)(0.7, 0.6)
    assert L.f3c_state_plan_times(st.h, t2, 2, ptr, nb, None) == f3c.F3C_EINVAL
    assert b"not finite" in L.f3c_last_error()
    assert L.f3c_state_plan_times(st.h, ok, 2, ptr + 16, nb - 16, None) == f3c.F3C_EINVAL
    assert L.f3c_state_plan_times(st.h, ok, 2, ptr, 1024, None) == f3c.F3C_ENOMEM
    assert L.f3c_state_plan_times(st.h, None, 2, ptr, nb, None) == f3c.F3C_EINVAL
    assert L.f3c_state_plan_times(st.h, ok, 2000, ptr, nb, None) == f3c.F3C_EINVAL
    # the plan of 0.9 and 0.8 is still in place
    x = to_dev(synth.make_noise(cfg, 1))
    st.profile(["mod"])
    st.profile_reset()
    st.full_step(x, 0.9, 0.8)
    st.full_step(x, 0.8, 0.75)
    st.full_step(x, 0.75, 0.7)
    torch.cuda.synchronize()
    assert st.profile_read()["mod"]["launches"] == 1
    st.profile(False)
    st.plan_times([0.5])
    assert st.plan_buf is buf


def test_trellis16_cached_step_full_depth(torch):
    """Full-size model (24 blocks, width 1024, 4096 tokens), cached step at 80% quota."""
    cfg = synth.TRELLIS16
    pair = Pair(cfg, 1)
    rng = np.random.default_rng(7)
    x = to_dev(pair.x_T)
    vc = (0.5 * rng.standard_normal((1, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    t = schedule.time_grid(25, 3.0)
    say("trellis16 cached step k=25")
    r = _gpu_step(torch, pair, x, t[24], t[25], [3276])
    err = _check_step(pair, r, t[24], t[25], [3276], 2e-2)
    say("trellis16 cached max-rel", err)


def test_trellis16_full_step_two_blocks(torch):
    cfg = depth_variant(synth.TRELLIS16, 2)
    pair = Pair(cfg, 1)
    x = to_dev(pair.x_T)
    say("trellis16 depth-2 full step")
    r = _gpu_step(torch, pair, x, 1.0, 0.98630136986301364, [0])
    _check_step(pair, r, 1.0, 0.98630136986301364, [0], 2e-2)


def test_trellis16_batch4_ragged_cached_step(torch):
    cfg = depth_variant(synth.TRELLIS16, 2)
    pair = Pair(cfg, 4)
    rng = np.random.default_rng(8)
    x = to_dev(pair.x_T)
    vc = (0.5 * rng.standard_normal((4, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    q = synth.quota_schedule(synth.WORKLOADS["trellis16_cached_b4"])[-1].tolist()
    say("trellis16 b4 ragged", q)
    r = _gpu_step(torch, pair, x, 0.3, 0.25, q)
    _check_step(pair, r, 0.3, 0.25, q, 2e-2)


def test_trellis32_cached_step_one_block(torch):
    cfg = depth_variant(synth.TRELLIS32, 1)
    pair = Pair(cfg, 1)
    rng = np.random.default_rng(9)
    x = to_dev(pair.x_T)
    vc = (0.5 * rng.standard_normal((1, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    say("trellis32 cached 70%")
    r = _gpu_step(torch, pair, x, 0.5, 0.45, [22937])
    _check_step(pair, r, 0.5, 0.45, [22937], 2e-2)


def test_trellis16_trajectory_one_block(torch):
    """25 shifted steps with the seeded logistic quota: final latent within 3e-2 rel L2."""
    w = synth.WORKLOADS["trellis16_cached"]
    cfg = depth_variant(w.model, 1)
    pair = Pair(cfg, 1)
    times = schedule.time_grid(w.steps, w.shift)
    quotas = synth.quota_schedule(w)
    x = to_dev(pair.x_T)
    for k in range(w.steps):
        say("trellis16 trajectory step", k + 1)
        pair.state.cached_step(x, times[k], times[k + 1], quotas[k].tolist())
    torch.cuda.synchronize()
    ref = sampler.sample(pair.x_T, pair.velocity(), times, quotas)
    err = rel_l2(x.cpu().numpy(), ref.x)
    say("trajectory rel L2", err)
    assert err < 3e-2


def test_profiler_times_kernels_and_leaves_results_unchanged(torch):
    """With every class profiled, launches go through the event-stamping
    extended launch: the step's results stay bit-identical, every class that
    launched has a positive time, and the class times fit inside the step's
    wall time. The condition is long enough (4096 tokens, 64 key tiles) and the
    active set small enough (112 tokens) that cross-attention splits its key
    range over workgroups, so a class of two kernels is timed too."""
    from paper_2511_22533_amd import f3c
    from paper_2511_22533_amd.f3c import PROF_CLASSES
    cfg = synth.ModelConfig(grid=8, width=256, depth=2, heads=4, cond_tokens=4096, cond_width=64, dtype="bf16")
    model = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    state = f3c.State(model, 1)
    cond = to_dev(synth.make_cond(cfg, 1))
    x_T = synth.make_noise(cfg, 1)
    outs = []
    for profiled in (False, True):
        say(f"profiled={profiled}")
        state.reset()
        state.set_cond(cond)
        x = to_dev(x_T)
        state.full_step(x, 1.0, 0.9)
        state.full_step(x, 0.9, 0.8)
        state.profile(True if profiled else None)
        state.profile_reset()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        state.cached_step(x, 0.8, 0.7, [400])
        e1.record()
        torch.cuda.synchronize()
        prof = state.profile_read()
        state.profile(None)
        outs.append(x.cpu().numpy())
        if profiled:
            want = {"select": 1, "embed": 1, "mod": 1, "ln": 3 * cfg.depth, "gemm_qkv": cfg.depth,
                    "attn_self": cfg.depth, "gemm_o": cfg.depth, "gemm_q": cfg.depth, "attn_cross": cfg.depth,
                    "gemm_co": cfg.depth, "gemm_fc1": cfg.depth, "gemm_fc2": cfg.depth, "final": 1, "euler": 1}
            for c in PROF_CLASSES:
                assert prof[c]["launches"] == want.get(c, 0), c
                if want.get(c):
                    assert prof[c]["ms"] > 0, c
            total = sum(prof[c]["ms"] for c in PROF_CLASSES)
            assert total <= e0.elapsed_time(e1) * 1.02 + 0.01
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


def _uncond(cfg, batch, seed=2500):
    """An unconditional input distinct from the condition: seeded N(0, 1) tokens, or zeros (seed None)."""
    if seed is None:
        return np.zeros((batch, cfg.cond_tokens, cfg.cond_width), F32)
    return synth.make_cond(cfg, batch, seed_base=seed)


def test_guided_tiny_f32_trajectory(torch):
    """Guided steps inside the guidance interval, then plain steps, against the
    oracle step by step and over the trajectory."""
    w_ = synth.WORKLOADS["tiny_f32"]
    pair = Pair(w_.model, 2, uncond=_uncond(w_.model, 2))
    times = schedule.time_grid(w_.steps, w_.shift)
    quotas = np.concatenate([synth.quota_schedule(w_)] * 2, axis=1)
    quotas[:, 1] = quotas[:, 1] // 2
    guided = schedule.guided_steps(times)
    assert guided[0] and not guided[-1]
    w = 3.0
    x = to_dev(pair.x_T)
    for k in range(w_.steps):
        q = quotas[k].tolist()
        say("guided tiny step", k + 1, q, guided[k])
        if guided[k]:
            r = _gpu_step(torch, pair, x, times[k], times[k + 1], q, w)
            _check_guided_step(pair, r, times[k], times[k + 1], q, w, 1e-4)
        else:
            r = _gpu_step(torch, pair, x, times[k], times[k + 1], q)
            _check_step(pair, r, times[k], times[k + 1], q, 1e-4)
    ref = sampler.sample(pair.x_T, pair.velocity(), times, quotas, uncond=pair.velocity_uncond(), w=w,
                         guided=guided)
    assert rel_l2(x.cpu().numpy(), ref.x) < 1e-4


def test_guided_passes_are_independent(torch):
    """With the unconditional input equal to the condition, the two passes get
    identical rows and identical keys/values, so their outputs must be equal
    bit for bit (any mixing of the two halves' segments or keys/values breaks
    it), and the step stays within tolerance of the oracle."""
    cfg = depth_variant(synth.TRELLIS16, 2)
    base = Pair(cfg, 2)
    pair = Pair(cfg, 2, uncond=base.cond.copy())
    rng = np.random.default_rng(11)
    vc = (0.5 * rng.standard_normal((2, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    x = to_dev(pair.x_T)
    q = [1500, 3000]
    say("guided equal passes", q)
    r = _gpu_step(torch, pair, x, 0.8, 0.75, q, 2.0)
    rows = r["off"][-1]
    assert np.array_equal(r["vact"][:rows].view(np.uint32), r["vact"][rows:].view(np.uint32))
    _check_guided_step(pair, r, 0.8, 0.75, q, 2.0, 2e-2)


def test_guided_trellis16_full_depth(torch):
    """Full-size model, a guided Phase 2 step (50% cached) with a zero unconditional input."""
    cfg = synth.TRELLIS16
    pair = Pair(cfg, 1, uncond=_uncond(cfg, 1, seed=None))
    rng = np.random.default_rng(12)
    vc = (0.5 * rng.standard_normal((1, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    x = to_dev(pair.x_T)
    t = schedule.time_grid(25, 3.0)
    say("trellis16 guided step k=12")
    r = _gpu_step(torch, pair, x, t[11], t[12], [2048], 7.5)
    err = _check_guided_step(pair, r, t[11], t[12], [2048], 7.5, 2e-2)
    say("trellis16 guided max-rel", err)


def test_guided_batch4_ragged_and_full(torch):
    cfg = depth_variant(synth.TRELLIS16, 1)
    pair = Pair(cfg, 4, uncond=_uncond(cfg, 4))
    x = to_dev(pair.x_T)
    say("guided b4 full")
    r = _gpu_step(torch, pair, x, 1.0, 0.98, [0, 0, 0, 0], 1.5)
    _check_guided_step(pair, r, 1.0, 0.98, [0, 0, 0, 0], 1.5, 2e-2)
    say("guided b4 ragged")
    q = [4096, 100, 2500, 3900]                # an empty active set, and ragged ones
    r = _gpu_step(torch, pair, x, 0.98, 0.95, q, 1.5)
    _check_guided_step(pair, r, 0.98, 0.95, q, 1.5, 2e-2)


def test_guided_step_preconditions(torch):
    from paper_2511_22533_amd import f3c
    cfg = synth.TINY
    plain = Pair(cfg, 1)
    x = to_dev(plain.x_T)
    with pytest.raises(f3c.F3CError) as e:
        plain.state.guided_step(x, 1.0, 0.9, None, 2.0)
    assert e.value.code == f3c.F3C_ESTATE
    with pytest.raises(f3c.F3CError) as e:
        plain.state.set_uncond(plain.cond_dev)
    assert e.value.code == f3c.F3C_ESTATE
    g = f3c.State(plain.model, 1, guided=True)
    g.set_cond(plain.cond_dev)
    with pytest.raises(f3c.F3CError) as e:             # unconditional input not set
        g.guided_step(x, 1.0, 0.9, None, 2.0)
    assert e.value.code == f3c.F3C_ESTATE
    g.set_uncond(plain.cond_dev)
    with pytest.raises(f3c.F3CError) as e:
        g.guided_step(x, 1.0, 0.9, None, float("nan"))
    assert e.value.code == f3c.F3C_EINVAL
    # a guided state runs plain steps too, bit-identical to a plain state's
    x2 = to_dev(plain.x_T)
    plain.state.cached_step(x, 1.0, 0.9, [0])
    g.cached_step(x2, 1.0, 0.9, [0])
    torch.cuda.synchronize()
    assert torch.equal(x, x2)



@pytest.mark.parametrize("case", ["tiny_f32", "trellis16_bf16", "trellis16_bf16_guided", "trellis16_bf16_amplified"])
def test_per_block_residual_changes(torch, case):
    """The change each block makes to the residual stream (its gated
    self-attention, cross-attention and MLP outputs) against the oracle's, on
    the GPU's own active set, plus the embedding. With random-init gates
    (about 0.03) a wrong sublayer moves the final velocity too little for the
    velocity tolerance; the per-block change exposes it. At N(0, 0.02)
    weights the gated self-attention term is about a fifth of the ungated
    cross-attention's (RMS 0.005 against 0.028 at the full width); the
    amplified case (N(0, 0.05)) brings all three terms to the same order
    (0.9, 0.7 and 1.7 for self-attention, cross-attention and MLP)."""
    from paper_2511_22533_amd import f3c
    guided = case.endswith("guided")
    cfg = synth.TINY if case == "tiny_f32" else depth_variant(synth.TRELLIS16, 2)
    B = 2 if case == "tiny_f32" else 1
    scale = 0.05 if case.endswith("amplified") else 0.02
    pair = Pair(cfg, B, scale=scale, uncond=synth.make_cond(cfg, B, seed_base=2500) if guided else None)
    rng = np.random.default_rng(13)
    vc = (0.5 * rng.standard_normal((B, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    q = [100, 300] if case == "tiny_f32" else [2048]
    rows = sum(cfg.tokens - c for c in q) * (2 if guided else 1)
    L, d = cfg.depth, cfg.width
    buf = torch.zeros(((L + 1) * rows * d,), dtype=torch.float32, device="cuda")
    pair.state.trace_blocks(buf)
    x = to_dev(pair.x_T)
    say("per-block parity", case, q)
    r = _gpu_step(torch, pair, x, 0.7, 0.65, q, 2.0 if guided else None)
    pair.state.trace_blocks(None)
    tr_gpu = buf.cpu().numpy().reshape(L + 1, rows, d).astype(np.float64)
    tol_e, tol_dh = (1e-5, 1e-4) if cfg.dtype == "f32" else (1e-5, 1.5e-2)
    n_act = rows // (2 if guided else 1)
    worst = 0.0
    for p_idx, cond in enumerate([pair.cond] + ([pair.uncond] if guided else [])):
        for b in range(B):
            lo, hi = r["off"][b] + p_idx * n_act, r["off"][b + 1] + p_idx * n_act
            active = r["idx"][r["off"][b]:r["off"][b + 1]] if any(q) else np.arange(cfg.tokens)
            tr = {}
            pair.oracle.forward(r["x0"][b][active], active, 0.7, cond[b], trace=tr)
            assert max_rel(tr_gpu[0][lo:hi], tr["embed"]) < tol_e
            prev_gpu, prev_ref = tr_gpu[0][lo:hi], tr["embed"]
            for l in range(L):
                dh_gpu = tr_gpu[l + 1][lo:hi] - prev_gpu
                dh_ref = tr[l]["h"] - prev_ref
                err = max_rel(dh_gpu, dh_ref)
                worst = max(worst, err)
                assert err < tol_dh, f"pass {p_idx} sample {b} block {l}: {err}"
                prev_gpu, prev_ref = tr_gpu[l + 1][lo:hi], tr[l]["h"]
    say("per-block worst max-rel", worst)
