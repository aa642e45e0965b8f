"""Full-depth parity of the measured workloads against the oracle's stored
trajectories, and per-sublayer parity of the transformer, through the C ABI.

The stored trajectories (tests/golden/<workload>.s<b>.npz) are written by
tests/golden/make_trajectories.py, which runs Algorithm 1 with the CPU oracle
only (float64 transformer, float32 sampler state) on the seeded workloads:
the 24-block 16^3 model with the logistic quota (its first steps are full
steps, so step 1 is also the first step of the uncached 16^3 trajectory), the
same model at batch 4 with ragged quotas, and the 12-block 32^3 model with the
70% quota. Three checks per workload:

* free-running: the library's own 25-step trajectory from x_T ends within
  relative L2 3e-2 of the oracle's final latent (per sample);
* teacher-forced selection: every cached step takes the oracle's active sets
  (f3c_debug_force_active), so selection drift is removed; the fresh
  velocities of the stored steps agree within max-rel 2e-2 and the final
  latent within relative L2 3e-2;
* one step from the oracle's own state (f3c_state_import of its caches, its
  latent): the selection is bit-exact (the same score inputs) and the fresh
  velocities agree within max-rel 2e-2.

Per-sublayer parity: the pre-gate outputs of self-attention, cross-attention
and the MLP of every block (f3c_state_trace_sublayers) against the oracle's
sublayers evaluated on the library's own input to each sublayer, so that an
error in one sublayer cannot hide behind another.
"""
import os

import numpy as np
import pytest

from helpers import Pair, depth_variant, max_rel, rel_l2, say, to_dev
from oracle import schedule
from paper_2511_22533_amd import synth

pytestmark = pytest.mark.gpu

F32 = np.float32
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
VEL_TOL = 2e-2       # per-step velocity, max-rel, bf16
LATENT_TOL = 3e-2    # final latent, relative L2


@pytest.fixture(scope="module")
def torch():
    import torch as t
    from paper_2511_22533_amd import f3c
    f3c.lib()
    return t


def _golden(workload):
    """The stored trajectories of the workload's samples, None for a sample
    whose file has not been written (the samples of a batch are independent
    trajectories, each written on its own); skips when none exists."""
    w = synth.WORKLOADS[workload]
    out = []
    for b in range(w.batch):
        path = os.path.join(GOLDEN, f"{workload}.s{b}.npz")
        if os.path.exists(path):
            with np.load(path) as z:
                out.append({k: z[k] for k in z.files})
        else:
            out.append(None)
    if all(g is None for g in out):
        pytest.skip(f"no stored trajectory of {workload} (tests/golden/make_trajectories.py)")
    return out


def _active(g, k, N):
    """Sample's active token indices of step k (1-based), ascending."""
    return np.nonzero(np.unpackbits(g["active"][k - 1], bitorder="little")[:N])[0]


class Run:
    """One workload on the library: model, state and the seeded inputs."""

    def __init__(self, workload):
        from paper_2511_22533_amd import f3c
        self.w = w = synth.WORKLOADS[workload]
        self.cfg = cfg = w.model
        self.gold = _golden(workload)
        self.model = f3c.Model(cfg).load(synth.make_weights(cfg))
        self.state = f3c.State(self.model, w.batch)
        self.cond_dev = to_dev(synth.make_cond(cfg, w.batch))
        self.x_T = synth.make_noise(cfg, w.batch)
        self.quotas = synth.quota_schedule(w)
        self.times = schedule.time_grid(w.steps, w.shift)
        self.have = [b for b, g in enumerate(self.gold) if g is not None]   # samples with a stored trajectory
        for b in self.have:
            assert np.array_equal(self.gold[b]["times"], np.array(self.times)), "stored times differ"
            assert np.array_equal(self.gold[b]["quotas"], self.quotas[:, b])

    def start(self, torch):
        self.state.reset()
        self.state.set_cond(self.cond_dev)
        return to_dev(self.x_T)

    def step(self, x, k, forced=None):
        q = self.quotas[k - 1].tolist()
        if forced is not None:
            self.state.force_active(forced)
        if any(q):
            self.state.cached_step(x, float(self.times[k - 1]), float(self.times[k]), q)
        else:
            self.state.full_step(x, float(self.times[k - 1]), float(self.times[k]))

    def forced_sets(self, torch, k):
        """The oracle's active sets of step k for the stored samples; a sample
        without a stored trajectory gets its first N - c_b tokens (the samples
        are independent, and that one is not compared)."""
        N = self.cfg.tokens
        sets = [_active(g, k, N) if g is not None else np.arange(N - int(self.quotas[k - 1][b]))
                for b, g in enumerate(self.gold)]
        return torch.from_numpy(np.concatenate(sets).astype(np.int32)).cuda()

    def v_act_per_sample(self, torch):
        t = self.state.tensors()
        v = t["v_act"].cpu().numpy()
        off = t["act_off"]
        return [v[off[b]:off[b + 1]] for b in range(self.w.batch)]


_runs = {}


def _run(workload):
    if workload not in _runs:
        _runs.clear()                      # one workload's model on the device at a time
        _runs[workload] = Run(workload)
    return _runs[workload]


WORKLOADS = ["trellis16_cached", "trellis16_cached_b4", "trellis32_cached"]


@pytest.mark.parametrize("workload", WORKLOADS)
def test_free_running_trajectory_final_latent(torch, workload):
    r = _run(workload)
    N = r.cfg.tokens
    x = r.start(torch)
    same = 0
    for k in range(1, r.w.steps + 1):
        say(workload, "free-running step", k, r.quotas[k - 1].tolist())
        r.step(x, k)
        torch.cuda.synchronize()
        if any(r.quotas[k - 1]):
            t = r.state.tensors()
            idx, off = t["idx_active"].cpu().numpy(), t["act_off"]
            same += int(all(np.array_equal(idx[off[b]:off[b + 1]], _active(r.gold[b], k, N)) for b in r.have))
    final = x.cpu().numpy()
    errs = [rel_l2(final[b], r.gold[b]["x_final"]) for b in r.have]
    cached_steps = int(np.sum(r.quotas.sum(axis=1) > 0))
    say(workload, "final latent rel-L2 per sample", errs, f"identical selections {same}/{cached_steps}")
    assert max(errs) < LATENT_TOL, errs


@pytest.mark.parametrize("workload", WORKLOADS)
def test_teacher_forced_trajectory_velocities(torch, workload):
    r = _run(workload)
    x = r.start(torch)
    worst = {}
    for k in range(1, r.w.steps + 1):
        forced = r.forced_sets(torch, k) if any(r.quotas[k - 1]) else None
        say(workload, "teacher-forced step", k, r.quotas[k - 1].tolist())
        r.step(x, k, forced)
        torch.cuda.synchronize()
        key = f"v_act_k{k}"
        if key in r.gold[r.have[0]]:
            got = r.v_act_per_sample(torch)
            errs = [max_rel(got[b], r.gold[b][key]) for b in r.have]
            worst[k] = max(errs)
            assert max(errs) < VEL_TOL, (k, errs)
    final = x.cpu().numpy()
    errs = [rel_l2(final[b], r.gold[b]["x_final"]) for b in r.have]
    say(workload, "teacher-forced velocity max-rel per stored step", worst, "final rel-L2", errs)
    assert max(errs) < LATENT_TOL, errs


@pytest.mark.parametrize("workload", WORKLOADS)
def test_step_from_oracle_state(torch, workload):
    r = _run(workload)
    k = 15
    B, N = r.w.batch, r.cfg.tokens
    # samples without a stored trajectory start from zero caches and x_T (not compared)
    vc = np.stack([g[f"v_cache_before_k{k}"] if g is not None else np.zeros((N, 8), F32) for g in r.gold])
    vp = np.stack([g[f"v_prev_before_k{k}"] if g is not None else np.zeros((N, 8), F32) for g in r.gold])
    x = to_dev(np.stack([g[f"x_before_k{k}"] if g is not None else r.x_T[b] for b, g in enumerate(r.gold)]))
    r.start(torch)
    r.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    say(workload, "step", k, "from the oracle's state")
    r.step(x, k)
    torch.cuda.synchronize()
    t = r.state.tensors()
    idx, off = t["idx_active"].cpu().numpy(), t["act_off"]
    got = r.v_act_per_sample(torch)
    for b in r.have:
        assert np.array_equal(idx[off[b]:off[b + 1]], _active(r.gold[b], k, N)), f"selection sample {b}"
        err = max_rel(got[b], r.gold[b][f"v_act_k{k}"])
        assert err < VEL_TOL, (b, err)


def test_trellis16_full_step_full_depth(torch):
    """The first step of the uncached 24-block 16^3 trajectory (every token
    active) equals the oracle's: it is step 1 of the stored cached trajectory,
    which starts with full steps from the same weights, noise and condition."""
    r = _run("trellis16_cached")
    x = r.start(torch)
    say("trellis16 full step at full depth")
    r.state.full_step(x, float(r.times[0]), float(r.times[1]))
    torch.cuda.synchronize()
    err = max_rel(r.v_act_per_sample(torch)[0], r.gold[0]["v_act_k1"])
    say("full step velocity max-rel", err)
    assert err < VEL_TOL, err


@pytest.mark.parametrize("case", ["tiny_f32", "trellis16_bf16", "trellis16_bf16_amplified", "trellis16_bf16_full"])
def test_sublayer_outputs_match_oracle(torch, case):
    """Each sublayer's output before its gate against the oracle sublayer on
    the library's own input to that sublayer: the residual stream entering the
    block (f3c_state_trace_blocks) for self-attention, plus the gated
    self-attention output for cross-attention, plus the cross-attention output
    for the MLP."""
    cfg = synth.TINY if case == "tiny_f32" else depth_variant(synth.TRELLIS16, 2)
    B = 2 if case == "tiny_f32" else 1
    scale = 0.05 if case.endswith("amplified") else 0.02
    pair = Pair(cfg, B, scale=scale)
    rng = np.random.default_rng(17)
    vc = (0.5 * rng.standard_normal((B, cfg.tokens, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    pair.state.import_(np.concatenate([vc.ravel(), vp.ravel()]))
    q = [100, 300] if case == "tiny_f32" else ([0] if case.endswith("full") else [2048])
    rows = sum(cfg.tokens - c for c in q)
    L, d = cfg.depth, cfg.width
    hbuf = torch.zeros(((L + 1) * rows * d,), dtype=torch.float32, device="cuda")
    sbuf = torch.zeros((3 * L * rows * d,), dtype=torch.float32, device="cuda")
    pair.state.trace_blocks(hbuf)
    pair.state.trace_sublayers(sbuf)
    x = to_dev(pair.x_T)
    x0 = pair.x_T.copy()
    t, tn = 0.7, 0.65
    say("sublayer parity", case, q)
    if any(q):
        pair.state.cached_step(x, t, tn, q)
    else:
        pair.state.full_step(x, t, tn)
    torch.cuda.synchronize()
    pair.state.trace_blocks(None)
    pair.state.trace_sublayers(None)
    tens = pair.state.tensors()
    off = tens["act_off"]
    idx = tens["idx_active"].cpu().numpy() if any(q) else np.arange(cfg.tokens)
    H = hbuf.cpu().numpy().reshape(L + 1, rows, d).astype(np.float64)
    S = sbuf.cpu().numpy().reshape(L, 3, rows, d).astype(np.float64)
    tol = 1e-4 if cfg.dtype == "f32" else VEL_TOL
    mod = pair.oracle.modulation(t)
    worst = {"sa": 0.0, "ca": 0.0, "mlp": 0.0}
    for b in range(B):
        lo, hi = off[b], off[b + 1]
        active = idx[lo:hi] if any(q) else np.arange(cfg.tokens)
        assert max_rel(H[0][lo:hi], pair.oracle.embed(x0[b][active], active)) < 1e-5
        for l in range(L):
            ck, cv = pair.oracle.cond_kv(pair.cond[b], l)
            h0 = H[l][lo:hi]
            sa, ca, mlp = S[l, 0][lo:hi], S[l, 1][lo:hi], S[l, 2][lo:hi]
            h1 = h0 + mod[l][2] * sa
            h2 = h1 + ca
            for name, got, want in (("sa", sa, pair.oracle.self_attention_sublayer(l, h0, mod[l])),
                                    ("ca", ca, pair.oracle.cross_attention_sublayer(l, h1, ck, cv)),
                                    ("mlp", mlp, pair.oracle.mlp_sublayer(l, h2, mod[l]))):
                err = max_rel(got, want)
                worst[name] = max(worst[name], err)
                assert err < tol, f"sample {b} block {l} {name}: max-rel {err}"
            # the residual update of the block is the sum of the traced terms
            assert max_rel(H[l + 1][lo:hi] - h0, mod[l][2] * sa + ca + mod[l][5] * mlp) < 1e-3
    say("sublayer worst max-rel", case, worst)


def test_forced_selection(torch):
    """f3c_debug_force_active: forcing the library's own selection reproduces
    the step bit for bit; forcing another active set runs the transformer on
    exactly that set (positions, merge and Euler as for a selected set); the
    hook is consumed by one step; a step with nothing cached ignores it."""
    from paper_2511_22533_amd import f3c
    cfg = synth.TINY
    B, N = 2, cfg.tokens
    pair = Pair(cfg, B, seed=4)
    rng = np.random.default_rng(23)
    vc = (0.5 * rng.standard_normal((B, N, 8))).astype(F32)
    vp = (vc + 0.05 * rng.standard_normal(vc.shape)).astype(F32)
    snap = np.concatenate([vc.ravel(), vp.ravel()])
    q = [100, 300]
    t, tn = 0.6, 0.55
    say("forced selection: own set")
    pair.state.import_(snap)
    x = to_dev(pair.x_T)
    pair.state.cached_step(x, t, tn, q)
    torch.cuda.synchronize()
    own = pair.state.tensors()["idx_active"].clone()
    x_own, st_own = x.clone(), pair.state.export()
    pair.state.import_(snap)
    x = to_dev(pair.x_T)
    pair.state.force_active(own)
    pair.state.cached_step(x, t, tn, q)
    torch.cuda.synchronize()
    assert torch.equal(x, x_own) and np.array_equal(pair.state.export(), st_own)

    say("forced selection: a random set")
    sets = [np.sort(rng.choice(N, N - c, replace=False)) for c in q]
    forced = torch.from_numpy(np.concatenate(sets).astype(np.int32)).cuda()
    pair.state.import_(snap)
    x = to_dev(pair.x_T)
    pair.state.force_active(forced)
    pair.state.cached_step(x, t, tn, q)
    torch.cuda.synchronize()
    tens = pair.state.tensors()
    off = tens["act_off"]
    assert np.array_equal(tens["idx_active"].cpu().numpy(), np.concatenate(sets))
    pos = tens["pos"].cpu().numpy()
    v_act = tens["v_act"].cpu().numpy()
    v_new = tens["v_cache"].cpu().numpy()
    dt = F32(t - tn)
    for b in range(B):
        want_pos = np.full(N, -1)
        want_pos[sets[b]] = off[b] + np.arange(len(sets[b]))
        assert np.array_equal(pos[b], want_pos)
        want = pair.oracle.forward(pair.x_T[b][sets[b]], sets[b], t, pair.cond[b])
        assert max_rel(v_act[off[b]:off[b + 1]], want) < 1e-4
        merged = vc[b].copy()
        merged[sets[b]] = v_act[off[b]:off[b + 1]]
        assert np.array_equal(v_new[b].view(np.uint32), merged.view(np.uint32))
        assert np.array_equal(x.cpu().numpy()[b].view(np.uint32), (pair.x_T[b] - dt * merged).view(np.uint32))

    say("forced selection: consumed by one step")
    x2 = x.clone()
    pair.state.cached_step(x2, tn, 0.5, q)      # selects on its own again
    torch.cuda.synchronize()
    after = pair.state.tensors()["idx_active"].cpu().numpy()
    from helpers import oracle_selection
    ref = oracle_selection(v_new, vc, q)
    assert np.array_equal(after, np.concatenate([ref[b][1] for b in range(B)]))

    say("forced selection: a full step ignores it")
    pair.state.force_active(forced)
    pair.state.full_step(x2, 0.5, 0.45)
    torch.cuda.synchronize()
    assert pair.state.tensors()["idx_active"] is None
    pair.state.force_active(None)
    with pytest.raises(f3c.F3CError):
        f3c.check(f3c.lib().f3c_debug_force_active(None, None))
