"""Write the oracle's full-depth trajectories of the measured workloads.

Algorithm 1 run end to end by the CPU oracle (oracle.sampler.step with the
float64 transformer of oracle.dit) on the seeded inputs of
paper_2511_22533_amd.synth: the 25-step cached trajectories of the 24-block
16^3 model (the logistic quota to 80% cached; its first five steps are full
steps, so they are also the first steps of the uncached 16^3 trajectory), of
the same model at batch 4 with ragged per-sample quotas, and of the 12-block
32^3 model with the fixed 70% quota.

This script calls only the oracle and the seeded input generators; nothing
here comes from the HIP library. One file per workload and sample,
``<workload>.s<b>.npz`` (float32 / uint8 arrays, no pickles):

  quotas      int32 [T]          cached count of each step (this sample)
  times       float64 [T+1]      the step times (Eq. S1 shift)
  active      uint8 [T][N/8]     active-token mask of each step, np.packbits
                                 (little bit order): bit i = token i active
  v_act_k<k>  float32 [n_k][8]   the step's fresh velocities of its active
                                 tokens (ascending token order), k in STORED
  x_before_k<k>, v_cache_before_k<k>, v_prev_before_k<k>
              float32 [N][8]     the sampler state entering step k, k in STATE
  x_final     float32 [N][8]     the latent after the last step

A batch-4 workload's samples are independent trajectories (each has its own
noise, condition and quota column), so each is written from a batch-1 run.

The oracle takes minutes per step at these sizes (about 40 minutes per full
step of the 32^3 model); ``--checkpoint DIR`` keeps the sampler state after
every step there and the residual stream after every transformer block of the
step in progress, and a rerun resumes from the last of them.

Usage (repository root):
    python tests/golden/make_trajectories.py --workload trellis16_cached
    python tests/golden/make_trajectories.py --workload trellis16_cached_b4 --sample 2
    python tests/golden/make_trajectories.py --workload trellis32_cached --checkpoint /tmp/ck
"""
from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import dit, sampler, schedule  # noqa: E402
from paper_2511_22533_amd import synth  # noqa: E402

STORED = (1, 6, 15, 25)      # steps whose fresh velocities are kept
STATE = (15,)                # steps whose incoming sampler state is kept
WORKLOADS = ("trellis16_cached", "trellis16_cached_b4", "trellis32_cached")


def out_path(workload: str, sample: int) -> str:
    return os.path.join(HERE, f"{workload}.s{sample}.npz")


def sample_inputs(workload: str, sample: int):
    """Model config, weights, and this sample's x_T [1][N][8], cond [1][Nc][dc], quota column."""
    w = synth.WORKLOADS[workload]
    cfg = w.model
    W = synth.make_weights(cfg)
    x_T = synth.make_noise(cfg, w.batch)[sample:sample + 1]
    cond = synth.make_cond(cfg, w.batch)[sample:sample + 1]
    quotas = synth.quota_schedule(w)[:, sample].astype(np.int32)
    times = np.array(schedule.time_grid(w.steps, w.shift), dtype=np.float64)
    return w, cfg, W, x_T, cond, quotas, times


def resumable_velocity(model: dit.Model, cond: np.ndarray, path: str | None):
    """The velocity of oracle.sampler.model_velocity, with the residual stream
    kept at ``path`` after every block: the same calls of the oracle in the
    same order as dit.Model.forward (modulation, embedding, the blocks, the
    final norm and projection), so a resumed step returns the same array."""
    if path is None:
        return sampler.model_velocity(model, cond)

    def fn(b, x_active, idx, t):
        mod = model.modulation(t)
        tag = np.array([float(t), float(b), float(idx.size), float(np.sum(idx, dtype=np.int64))])
        l0, h = 0, None
        if os.path.exists(path):
            with np.load(path) as z:
                if np.array_equal(z["tag"], tag) and np.array_equal(z["idx"], idx):
                    l0, h = int(z["blocks_done"]), z["h"].copy()
                    print(f"[golden]   resuming the step after block {l0}", flush=True)
        if h is None:
            h = model.embed(x_active, idx)
        for l in range(l0, model.cfg.depth):
            ck, cv = model.cond_kv(cond[b], l)
            h = model.block(l, h, mod[l], ck, cv)
            tmp = path + ".tmp.npz"
            np.savez(tmp, tag=tag, idx=idx, blocks_done=np.int64(l + 1), h=h)
            os.replace(tmp, path)
        return dit.linear(dit.layer_norm(h), model.w["out_w"], model.w["out_b"])
    return fn


def run(workload: str, sample: int, checkpoint: str | None) -> str:
    w, cfg, W, x_T, cond, quotas, times = sample_inputs(workload, sample)
    T, N = w.steps, cfg.tokens
    bpath = os.path.join(checkpoint, f"{workload}.s{sample}.block.npz") if checkpoint else None
    velocity = resumable_velocity(dit.Model(cfg, W), cond, bpath)
    st = sampler.State.start(x_T)
    out = {"quotas": quotas, "times": times, "active": np.zeros((T, N // 8), np.uint8)}
    k0 = 0
    ck = os.path.join(checkpoint, f"{workload}.s{sample}.ckpt.npz") if checkpoint else None
    if ck and os.path.exists(ck):
        with np.load(ck) as z:
            k0 = int(z["k_done"])
            st.x[:], st.v_cache[:], st.v_prev[:] = z["x"], z["v_cache"], z["v_prev"]
            for key in z.files:
                if key not in ("k_done", "x", "v_cache", "v_prev"):
                    out[key] = z[key]
        print(f"[golden] {workload} s{sample}: resuming after step {k0}", flush=True)
    for k in range(k0 + 1, T + 1):
        if k in STATE:
            out[f"x_before_k{k}"] = st.x[0].copy()
            out[f"v_cache_before_k{k}"] = st.v_cache[0].copy()
            out[f"v_prev_before_k{k}"] = st.v_prev[0].copy()
        t0 = time.time()
        rec = sampler.step(st, velocity, times[k - 1], times[k], [int(quotas[k - 1])])
        mask = np.zeros(N, dtype=bool)
        mask[rec.active[0]] = True
        out["active"][k - 1] = np.packbits(mask, bitorder="little")
        if k in STORED:
            out[f"v_act_k{k}"] = np.asarray(rec.v_active[0], np.float32)
        print(f"[golden] {workload} s{sample} step {k}/{T}: {int(mask.sum())} active, {time.time() - t0:.1f} s",
              flush=True)
        if ck:
            tmp = ck + ".tmp.npz"
            np.savez(tmp, k_done=np.int64(k), x=st.x, v_cache=st.v_cache, v_prev=st.v_prev, **out)
            os.replace(tmp, ck)
    out["x_final"] = st.x[0].copy()
    path = out_path(workload, sample)
    np.savez_compressed(path, **out)
    return path


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", required=True, choices=WORKLOADS)
    ap.add_argument("--sample", type=int, default=None, help="one sample (default: every sample)")
    ap.add_argument("--checkpoint", default=None, help="directory for per-step resumable state")
    args = ap.parse_args()
    if args.checkpoint:
        os.makedirs(args.checkpoint, exist_ok=True)
    B = synth.WORKLOADS[args.workload].batch
    for b in ([args.sample] if args.sample is not None else range(B)):
        print("[golden] wrote", run(args.workload, b, args.checkpoint), flush=True)


if __name__ == "__main__":
    main()
