"""Throughput of the cached sparse-structure flow-DiT sampler on one MI355X.

Workload (default, ``trellis32_cached``): the 12-block, width-1024
TRELLIS-shaped sparse-structure transformer on a 32^3 latent grid (32768
tokens, 8 channels), 16 heads of 64, cross-attention to 1374 condition tokens
of width 1024, bf16, batch 1, 25 shifted Euler steps: 5 full steps, then a
fixed 70% cache quota (9831 active tokens per cached step). Weights, noise and
condition tokens are seeded synthetic data (no trained weights or image
features exist here). The 24-block 16^3 workload with the logistic quota
(``trellis16_cached``) is measured after it over one whole trajectory and
reported in the ``secondary`` field.

A "step" is one denoising step of that schedule: stability scoring and top-k
selection, gather + embedding, timestep modulation, the blocks on the active
tokens, output projection and the merge/Euler/cache update. K timed steps walk
through the schedule from a trajectory start and wrap around; every trajectory
start re-zeroes the caches, reloads x_T, recomputes the condition keys/values
and plans the timestep modulation of all the trajectory's step times (one pass
over the modulation weights per 8 times) inside the timed region.

Prints one JSON line. ``value`` is denoising steps per second; the line also
carries active tokens/s, the whole-step MFMA fraction (FLOPs model of the
supplement over wall time), the roofline entry of the dominant kernel (HIP
events on the launch stream around each of its launches in the timed region)
and the CPU oracle baseline (a bounded sample timed on this host).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 matrix/vector
PEAK_HBM_GBS = 8000.0
# Sustained dense bf16 matrix-core rate measured by `f3c_drive --peaks` (independent
# v_mfma_f32_32x32x16_bf16 on register operands, four waves per SIMD; about 83% of the
# published peak, a clock near 2.0 GHz under a full MFMA load). Reported beside the
# published peak, which stays the roofline's reference.
MEASURED_BF16_TFLOPS = 2080.6
DENSE_CLASSES = ["gemm_qkv", "attn_self", "gemm_o", "gemm_q", "attn_cross", "gemm_co", "gemm_fc1", "gemm_fc2"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default="trellis32_cached")
    ap.add_argument("--secondary", default="trellis16_cached",
                    help="workload timed over one whole trajectory after the main one ('' = none)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-depth", type=int, default=None,
                    help="oracle blocks timed (default: as many as keep the sample near 15 s; 0 = full depth)")
    ap.add_argument("--copy-ref-mb", type=int, default=0,
                    help="first run one plain device-to-device copy of this many MiB (a known-size reference "
                         "for hardware byte counters)")
    ap.add_argument("--log-steps", action="store_true",
                    help="after the timed region, run one more trajectory and print one JSON line per step to "
                         "stderr (k, t, quotas, active tokens, model FLOPs, wall time, per-class kernel times); "
                         "every class is profiled there, so its wall times include the event stamps")
    ap.add_argument("--hbm-sweep", action="store_true",
                    help="instead of the sampler: time the memory-bound kernels in isolation over a size sweep "
                         "and report algorithmic bytes / kernel time against HBM peak")
    return ap.parse_args()


def counter_traffic(cls: str, workload: str, timed_ks):
    """HBM-side bytes per launch of a kernel class over the timed launches, from
    the committed FETCH_SIZE / WRITE_SIZE counter summary of the workload's
    trajectory (profiles/<workload>_traffic.md), or (None, reason).

    The summary holds one line per step k of the trajectory and class:
    "traffic <cls> k=<k>: <bytes> bytes over <calls> calls; sources <files>
    sha256 <hex>". The figure is the byte total of the timed steps' launches
    over their count (the same launches as the roofline's achieved rate), and
    is used only while the SHA-256 of the kernel's source files equals the one
    recorded with the counters."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"{workload}_traffic.md")
    if not os.path.exists(path):
        return None, f"no counter summary for {workload}"
    pat = re.compile(r"traffic (\w+) k=(\d+): (\d+) bytes over (\d+) calls; sources (\S+) sha256 ([0-9a-f]{64})")
    per_k = {}
    sources = None
    for line in open(path):
        m = pat.search(line)
        if not m or m.group(1) != cls:
            continue
        per_k[int(m.group(2))] = (int(m.group(3)), int(m.group(4)))
        sources = (m.group(5), m.group(6))
    if not per_k:
        return None, f"no counter line for {cls}"
    h = hashlib.sha256()
    for name in sources[0].split("+"):
        with open(os.path.join(ROOT, "paper_2511_22533_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != sources[1]:
        return None, "kernel sources changed since the counters were taken"
    if any(k not in per_k for k in timed_ks):
        return None, "counter summary does not cover every timed step"
    total = sum(per_k[k][0] for k in timed_ks)
    calls = sum(per_k[k][1] for k in timed_ks)
    return (round(total / calls) if calls else None,
            "rocprofv3 FETCH_SIZE + WRITE_SIZE per dispatch, scaled by a 256 MiB copy reference, over the timed "
            "steps' launches")


def _event_time_ms(torch, fn, reps):
    """Average duration of fn() over reps launches, HIP events on the current stream."""
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def _graph_time_ms(torch, fn, reps):
    """Average kernel time of fn() with no host gaps: reps calls captured in
    one HIP graph (the operator entries only enqueue kernels on the current
    stream), replayed once to warm up, then timed over one replay."""
    fn()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(reps):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    graph.replay()
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def hbm_sweep():
    """Isolated memory-bound kernels of the step through their C-ABI operator
    entries. Algorithmic bytes per launch (what the kernel must move at least):
      score+select  B*N*(64 + 4) + sum(n)*4   (two velocity caches in, pos + idx out)
      embed         sum(n)*(32 + 2d + 4d)     (x row, bf16 position row, f32 h row)
      merge+Euler   B*N*(32*4 + 4)            (x in/out, v in, v_new out, pos)
      LN+mod        rows*d*(4 + 2)            (f32 h in, bf16 out)
      modulation    the bf16 weights of the two timestep layers and all blocks' 6d outputs
      pack_occ      B*V*(4 + 1/8)             (f32 logit per voxel in, one bit out)
      dyn_voxels    B*V/4                     (two packed grids in, Eq. 1)
    Times are per launch with no host gaps (the launches of each size are
    captured in one graph). A selection call is two kernels: the scoring pass
    streams the caches over the whole chip (its share: B*N*64 bytes), then one
    workgroup per sample selects from its keys held in LDS, so below about
    256 samples that second kernel's time is latency."""
    import torch
    from paper_2511_22533_amd import f3c, synth
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda").manual_seed(0)
    rows_out = []

    def add(kernel, shape, nbytes, ms):
        gbs = nbytes / (ms * 1e-3) / 1e9
        rows_out.append({"kernel": kernel, "shape": shape, "bytes": int(nbytes), "us": round(ms * 1e3, 2),
                         "GB/s": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)})
        print(f"[sweep] {kernel:12s} {shape:28s} {ms * 1e3:9.2f} us {gbs:8.1f} GB/s", file=sys.stderr, flush=True)

    for B, N in [(1, 4096), (4, 4096), (1, 32768), (16, 32768), (64, 32768)]:
        vc = torch.randn((B, N, 8), device="cuda", generator=g)
        vp = torch.randn((B, N, 8), device="cuda", generator=g)
        n_cache = [int(0.8 * N)] * B
        tot = sum(N - c for c in n_cache)
        idx = torch.empty((tot,), dtype=torch.int32, device="cuda")
        pos = torch.empty((B, N), dtype=torch.int32, device="cuda")
        ms = _graph_time_ms(torch, lambda: f3c.op_select(vc, vp, 0.7, n_cache, idx, pos), 20)
        add("select", f"B={B} N={N}", B * N * 68 + tot * 4, ms)
        del vc, vp, idx, pos

    cfg = synth.ModelConfig(grid=32, width=1024, depth=1, heads=16, cond_tokens=8, cond_width=64, dtype="bf16")
    model = f3c.Model(cfg).load(synth.make_weights(cfg, seed=0))
    N, d = cfg.grid ** 3, cfg.width
    for B in (1, 4, 16):
        x = torch.randn((B, N, 8), device="cuda", generator=g)
        for frac in (0.3, 1.0):
            n = int(frac * N)
            idx = torch.sort(torch.randperm(N, device="cuda", generator=g)[:n])[0].to(torch.int32).repeat(B)
            off = [b * n for b in range(B + 1)]
            h = torch.empty((B * n, d), dtype=torch.float32, device="cuda")
            ms = _graph_time_ms(torch, lambda: f3c.op_embed(model, x, off, h, idx_active=idx), 10)
            add("embed", f"B={B} N={N} n={n}", B * n * (32 + 6 * d), ms)
            del h
        del x

    for B, N in [(1, 4096), (16, 32768), (16, 1 << 20)]:
        x = torch.randn((B, N, 8), device="cuda", generator=g)
        vc = torch.randn((B, N, 8), device="cuda", generator=g)
        vn = torch.empty_like(vc)
        n = N // 5
        va = torch.randn((B * n, 8), device="cuda", generator=g)
        pos = torch.full((B, N), -1, dtype=torch.int32, device="cuda")
        pos[:, :n] = torch.arange(B * n, device="cuda", dtype=torch.int32).view(B, n)
        off = [b * n for b in range(B + 1)]
        ms = _graph_time_ms(torch, lambda: f3c.op_euler(x, vc, va, pos, off, 0.5, 0.45, vn), 20)
        add("euler", f"B={B} N={N}", B * N * 132, ms)
        del x, vc, vn, va, pos

    for rows in (820, 4096, 32768, 262144):
        h = torch.randn((rows, 1024), device="cuda", generator=g)
        out = torch.empty((rows, 1024), dtype=torch.bfloat16, device="cuda")
        sh = torch.randn((1024,), device="cuda", generator=g)
        sc = torch.randn((1024,), device="cuda", generator=g)
        ms = _graph_time_ms(torch, lambda: f3c.op_ln_mod(f3c.F3C_BF16, h, out, sh, sc), 20)
        add("ln_mod", f"rows={rows} d=1024", rows * 1024 * 6, ms)
        del h, out

    for B, V in [(1, 64 ** 3), (16, 64 ** 3), (1, 256 ** 3), (8, 256 ** 3)]:
        logits = torch.randn((B, V), device="cuda", generator=g)
        bits = torch.empty((2, B, (V + 31) // 32), dtype=torch.int32, device="cuda")
        ms = _graph_time_ms(torch, lambda: f3c.op_pack_occupancy(logits, bits[0]), 20)
        add("pack_occ", f"B={B} V={V}", B * V * 4 + B * V // 8, ms)
        counts = torch.empty((B,), dtype=torch.int64, device="cuda")
        ms = _graph_time_ms(torch, lambda: f3c.op_dynamic_voxels(bits[0], bits[1], counts), 20)
        add("dyn_voxels", f"B={B} V={V}", B * V // 4, ms)
        del logits, bits

    mcfg = synth.TRELLIS16
    mm = f3c.Model(mcfg).load(synth.make_weights(mcfg, seed=0))
    d, L = mcfg.width, mcfg.depth
    mod = torch.empty((L * 6 * d,), dtype=torch.float32, device="cuda")
    scratch = torch.empty((2 * d,), dtype=torch.float32, device="cuda")
    ms = _graph_time_ms(torch, lambda: f3c.check(f3c.lib().f3c_op_modulation(
        mm.h, 0.5, mod.data_ptr(), scratch.data_ptr(), f3c._stream(None))), 20)
    wbytes = 2 * (256 * d + d * d + L * 6 * d * d) + 4 * L * 6 * d
    add("modulation", f"L={L} d={d}", wbytes, ms)
    print(json.dumps({"mode": "hbm_sweep", "peak_GB/s": PEAK_HBM_GBS, "rows": rows_out}), flush=True)


def _cpu_model() -> str:
    """The host CPU's model name from /proc/cpuinfo (empty if unavailable)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


CPU_SAMPLE_S = 15.0   # target seconds of oracle work in the CPU baseline sample


def cpu_baseline(w, W, cond, x_T, quotas, times, depth=None, guided=None):
    """Time the CPU oracle on a bounded sample of the workload and scale it to
    steps/s over the schedule.

    The sample is one cached step at the schedule's largest quota, at `depth`
    blocks (default: one block for the 12-block 32^3 model, eight for the
    24-block 16^3 model), then one full step at the same depth if the FLOPs
    model predicts it fits the CPU_SAMPLE_S budget from the cached step's rate;
    otherwise the full step's time is that prediction (labelled as such). Step
    times are scaled by the block count and interpolated over the schedule's
    active counts with the FLOPs model. A guided step counts as two passes."""
    from oracle import dit, flops, sampler
    from paper_2511_22533_amd import synth
    cfg = w.model
    if depth is None:
        depth = 1 if cfg.tokens > 4096 else min(8, cfg.depth)
    depth = depth or cfg.depth
    sub = synth.ModelConfig(grid=cfg.grid, width=cfg.width, depth=depth, heads=cfg.heads,
                            cond_tokens=cfg.cond_tokens, cond_width=cfg.cond_width, dtype=cfg.dtype,
                            mlp_ratio=cfg.mlp_ratio)
    model = dit.Model(sub, W)
    vel = sampler.model_velocity(model, cond)
    st = sampler.State.start(x_T)
    rng = np.random.default_rng(0)
    st.v_cache[:] = rng.standard_normal(st.v_cache.shape).astype(np.float32)
    st.v_prev[:] = rng.standard_normal(st.v_prev.shape).astype(np.float32)
    k_max = int(np.argmax(quotas.sum(axis=1)))
    q_max = [int(c) for c in quotas[k_max]]
    N = cfg.tokens
    t0 = time.perf_counter()
    sampler.step(st, vel, times[k_max], times[k_max + 1], q_max)
    t_cached = time.perf_counter() - t0
    f_full = sum(flops.forward_flops(sub, N, 1) for _ in range(w.batch))
    f_cached = sum(flops.forward_flops(sub, N - c, 1) for c in q_max)
    predicted_full = t_cached * f_full / f_cached if f_cached > 0 else t_cached
    if predicted_full <= CPU_SAMPLE_S:
        t0 = time.perf_counter()
        sampler.step(st, vel, times[0], times[1], [0] * w.batch)
        t_full = time.perf_counter() - t0
        full_how = f"one full step ({N} tokens per sample, {t_full:.2f} s)"
    else:
        t_full = predicted_full
        full_how = (f"the full step ({N} tokens per sample) not run: its time, {t_full:.1f} s, is the cached "
                    f"step's rate times the FLOPs model's full/cached ratio")
    scale = cfg.depth / depth
    total = 0.0
    tokens = 0
    for k, q in enumerate(quotas):
        f = sum(flops.forward_flops(sub, N - int(c), 1) for c in q)
        frac = (f - f_cached) / (f_full - f_cached) if f_full > f_cached else 1.0
        passes = 2 if guided is not None and guided[k] else 1
        total += passes * scale * (t_cached + (t_full - t_cached) * frac)
        tokens += sum(N - int(c) for c in q)
    steps = len(quotas)
    threads = len(os.sched_getaffinity(0))
    return {
        "value": steps / total,
        "unit": "steps/s",
        "cores": threads,
        "cpu_model": _cpu_model(),
        "kind": "oracle",
        "sample": (f"float64 NumPy oracle, {depth} of {cfg.depth} blocks: one cached step at the schedule's "
                   f"largest quota ({sum(N - c for c in q_max)} active tokens, {t_cached:.2f} s) and {full_how}; "
                   f"scaled by {scale:g} to all blocks and interpolated over the {steps}-step schedule with the "
                   f"FLOPs model"
                   + (f", guided steps counted as two passes ({sum(guided)} of {steps})" if guided is not None else "")),
        "active_tokens_per_s": tokens / total,
        "seconds_measured": t_cached + (t_full if predicted_full <= CPU_SAMPLE_S else 0.0),
    }


class Runner:
    """One workload on the library: model, state, seeded inputs and the step loop."""

    def __init__(self, name: str):
        import torch
        from paper_2511_22533_amd import f3c, synth
        self.torch, self.f3c = torch, f3c
        w = self.w = synth.WORKLOADS[name]
        cfg = self.cfg = w.model
        self.W = synth.make_weights(cfg)
        self.cond = synth.make_cond(cfg, w.batch)
        self.x_T = synth.make_noise(cfg, w.batch)
        self.quotas = synth.quota_schedule(w)
        self.times = f3c.time_grid(w.steps, w.shift)
        self.model = f3c.Model(cfg).load(self.W)
        self.guided = [w.guidance > 0 and f3c.guidance_active(float(t), *w.guidance_interval)
                       for t in self.times[:-1]]
        self.state = f3c.State(self.model, w.batch, guided=any(self.guided))
        self.x = torch.empty((w.batch, cfg.tokens, cfg.in_ch), dtype=torch.float32, device="cuda")
        self.x_T_dev = torch.from_numpy(self.x_T).cuda()
        self.cond_dev = torch.from_numpy(self.cond).cuda()
        self.uncond_dev = (torch.from_numpy(synth.make_uncond(cfg, w.batch)).cuda() if any(self.guided)
                           else None)
        self.T = w.steps

    def step(self, i: int) -> int:
        """Step i of the endless schedule (a trajectory start every T steps); returns its active tokens."""
        w, cfg, st, x, times = self.w, self.cfg, self.state, self.x, self.times
        k = i % self.T
        if k == 0:
            st.reset()
            x.copy_(self.x_T_dev)
            st.set_cond(self.cond_dev)
            if self.uncond_dev is not None:
                st.set_uncond(self.uncond_dev)
            st.plan_times(times[:-1])
        q = self.quotas[k].tolist()
        if self.guided[k]:
            st.guided_step(x, float(times[k]), float(times[k + 1]), q if any(q) else None, w.guidance)
        elif any(q):
            st.cached_step(x, float(times[k]), float(times[k + 1]), q)
        else:
            st.full_step(x, float(times[k]), float(times[k + 1]))
        return sum(cfg.tokens - c for c in q)

    def step_flops(self, i: int) -> float:
        k = i % self.T
        return (2 if self.guided[k] else 1) * sum(self.f3c.forward_flops(self.cfg, self.cfg.tokens - int(c), 1)
                                                  for c in self.quotas[k])

    def trajectory_ms(self, reps: int = 1) -> float:
        """Wall time of whole trajectories (host clock around synchronised runs), ms per trajectory."""
        torch = self.torch
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(reps * self.T):
            self.step(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / reps


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "f3c runs on one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.hbm_sweep:
        hbm_sweep()
        return

    import torch
    from paper_2511_22533_amd import f3c
    from paper_2511_22533_amd.f3c import PROF_CLASSES

    torch.cuda.set_device(0)
    if args.copy_ref_mb:
        src = torch.ones(args.copy_ref_mb << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] reference copy of {args.copy_ref_mb} MiB done", file=sys.stderr, flush=True)
        del src, dst
    run = Runner(args.workload)
    w, cfg, state, x, times, quotas, guided, T = (run.w, run.cfg, run.state, run.x, run.times, run.quotas,
                                                  run.guided, run.T)
    print(f"[bench] workload {w.name}: {w.description}", file=sys.stderr, flush=True)

    # warmup (untimed)
    for i in range(args.warmup):
        run.step(i)
    torch.cuda.synchronize()
    print(f"[bench] warmup {args.warmup} steps done", file=sys.stderr, flush=True)

    # calibration pass (untimed): which dense kernel class takes the most time
    state.profile(True)
    state.profile_reset()
    for i in range(T):
        run.step(i)
    torch.cuda.synchronize()
    calib = state.profile_read()
    state.profile(False)
    state.profile_reset()
    dominant = max(DENSE_CLASSES, key=lambda c: calib[c]["ms"])
    print(f"[bench] per-class ms over one trajectory: "
          + ", ".join(f"{c}={calib[c]['ms']:.2f}" for c in PROF_CLASSES if calib[c]["launches"]),
          file=sys.stderr, flush=True)

    # timed region: K steps from a trajectory start, events only around the dominant class
    state.profile([dominant])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    active = 0
    flop_total = 0.0
    for i in range(args.steps):
        active += run.step(i)
        flop_total += run.step_flops(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = state.profile_read()[dominant]
    state.profile(False)
    print(f"[bench] timed {args.steps} steps in {elapsed * 1e3:.1f} ms", file=sys.stderr, flush=True)

    # Whole trajectories (untimed for `value`): samples per second.
    traj_ms = run.trajectory_ms(1)

    # Full and cached steps timed apart (untimed for `value`): repeated full
    # steps from a trajectory start, and repeated cached steps at the
    # schedule's largest quota (its smallest active set).
    state.reset()
    x.copy_(run.x_T_dev)
    state.set_cond(run.cond_dev)
    full_ms = _event_time_ms(torch, lambda: state.full_step(x, float(times[0]), float(times[1])), 10)
    guided_full_ms = _event_time_ms(torch, lambda: state.guided_step(x, float(times[0]), float(times[1]), None,
                                                                     w.guidance), 10) if any(guided) else None
    k_min = int(np.argmax(quotas.sum(axis=1)))
    q_min = quotas[k_min].tolist()
    cached_ms = _event_time_ms(torch, lambda: state.cached_step(x, float(times[k_min]), float(times[k_min + 1]),
                                                                q_min), 20) if any(q_min) else None

    if args.log_steps:
        # One trajectory, untimed for `value`: per-step wall time between events
        # on the launch stream, and the library's per-class kernel times.
        state.profile(True)
        for k in range(T):
            state.profile_reset()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            n_act = run.step(k)
            e1.record()
            e1.synchronize()
            cls = state.profile_read()
            rec = {"k": k + 1, "t": float(times[k]), "t_next": float(times[k + 1]),
                   "n_cache": quotas[k].tolist(), "n_active": int(n_act), "guided": bool(guided[k]),
                   "model_flops": run.step_flops(k), "wall_ms": round(e0.elapsed_time(e1), 4),
                   "class_ms": {c: round(v["ms"], 4) for c, v in cls.items() if v["launches"]}}
            print(json.dumps(rec), file=sys.stderr, flush=True)
        state.profile(False)

    peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = prof["flops"] / (prof["ms"] * 1e-3) / 1e12 if prof["ms"] > 0 else 0.0
    timed_ks = [i % T + 1 for i in range(args.steps)]
    traffic, traffic_src = counter_traffic(dominant, w.name, timed_ks)
    roofline = {
        "bound": "mfma",
        "kernel": dominant,
        "achieved": round(achieved, 2),
        "peak": peak,
        "unit": "TFLOP/s",
        "frac": round(achieved / peak, 4),
        **({"measured_peak": MEASURED_BF16_TFLOPS, "frac_of_measured": round(achieved / MEASURED_BF16_TFLOPS, 4)}
           if cfg.dtype == "bf16" else {}),
        "traffic": traffic,
        "traffic_source": traffic_src,
        "algorithmic_bytes_per_launch": round(prof["bytes"] / max(prof["launches"], 1)),
        "launches": prof["launches"],
        "avg_launch_us": round(prof["ms"] * 1e3 / max(prof["launches"], 1), 2),
        "flops_per_launch": prof["flops"] / max(prof["launches"], 1),
        "over": f"the {prof['launches']} launches of the timed steps (k = {timed_ks[0]}..{timed_ks[-1]})",
    }
    step_tflops = flop_total / elapsed / 1e12
    out = {
        "metric": "denoising steps/s (cached flow-DiT sampler)",
        "value": round(args.steps / elapsed, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded weights, noise and condition tokens)",
        "config": {"workload": w.name, "grid": cfg.grid, "tokens": cfg.tokens, "width": cfg.width,
                   "depth": cfg.depth, "heads": cfg.heads, "cond_tokens": cfg.cond_tokens, "batch": w.batch,
                   "steps_per_trajectory": T, "quota": w.schedule, "parallelism": "single GPU",
                   **({"guidance": w.guidance, "guided_steps": int(sum(guided))} if any(guided) else {})},
        "active_tokens_per_s": round(active / elapsed, 1),
        "trajectory_ms": round(traj_ms, 3),
        "samples_per_s": round(w.batch * 1e3 / traj_ms, 4),
        "full_step_ms": round(full_ms, 4),
        **({"guided_full_step_ms": round(guided_full_ms, 4)} if guided_full_ms is not None else {}),
        "cached_step_ms": round(cached_ms, 4) if cached_ms is not None else None,
        "cached_step_active_tokens": int(sum(cfg.tokens - c for c in q_min)),
        "step_model_tflops": round(step_tflops, 2),
        "step_mfma_frac": round(step_tflops / peak, 4),
        "roofline": roofline,
    }
    W_host, cond_host, x_T_host = run.W, run.cond, run.x_T
    if args.secondary and args.secondary != w.name:
        del run, state, x
        torch.cuda.empty_cache()
        r2 = Runner(args.secondary)
        r2.trajectory_ms(1)                         # warm-up trajectory
        ms2 = r2.trajectory_ms(2)
        fl2 = sum(r2.step_flops(i) for i in range(r2.T))
        out["secondary"] = {"workload": r2.w.name, "steps_per_s": round(r2.T * 1e3 / ms2, 3),
                            "ms_per_step": round(ms2 / r2.T, 4), "trajectory_ms": round(ms2, 3),
                            "step_model_tflops": round(fl2 / (ms2 * 1e-3) / 1e12, 2),
                            "timed": "two whole trajectories after one warm-up trajectory"}
        print(f"[bench] secondary {r2.w.name}: {ms2:.1f} ms per trajectory", file=sys.stderr, flush=True)
        del r2
    if not args.no_cpu:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, W_host, cond_host, x_T_host, quotas, times, args.cpu_depth,
                                           guided if any(guided) else None)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
