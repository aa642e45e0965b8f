"""Host-side checks of the C ABI (no GPU needed).

* the library loads and exports every function include/f3c.h declares;
* the canonical weight list matches the seeded generator's parameter list;
* argument validation rejects bad shapes before any device work;
* the host schedules (Eq. S1 time grid, ceil ratios, Algorithm 1 phase rule,
  Eqs. 4-5 quota) and the FLOPs model agree with the oracle's restatement.
"""
import ctypes
import math
import os
import subprocess

import numpy as np
import pytest

from oracle import flops as oflops
from oracle import schedule as osched
from paper_2511_22533_amd import f3c, synth


@pytest.fixture(scope="module")
def L():
    return f3c.lib()


def test_exports_every_declared_symbol(L):
    declared = f3c.header_symbols()
    assert len(declared) >= 30
    out = subprocess.run(["nm", "-D", "--defined-only", f3c.LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [s for s in declared if s not in exported]
    assert not missing, missing
    for s in declared:
        assert hasattr(L, s)
    assert set(f3c._SIGS) == set(declared)


@pytest.mark.parametrize("wname", sorted(synth.WORKLOADS))
def test_weight_list_matches_generator(wname):
    cfg = synth.WORKLOADS[wname].model
    m = f3c.Model(cfg)
    got = m.weight_names()
    want = [(n, int(np.prod(s))) for n, s in synth.weight_specs(cfg)]
    assert got == want


def _cfg(**kw):
    base = dict(grid=8, width=128, depth=2, heads=4, cond_tokens=64, cond_width=128, dtype="f32")
    base.update(kw)
    return synth.ModelConfig(**base)


@pytest.mark.parametrize("kw,msg", [
    (dict(width=96, heads=3), "multiple of 128"),
    (dict(heads=8), "head_dim"),
    (dict(grid=33), "exceeds"),
    (dict(cond_width=100), "cond_width"),
    (dict(depth=0), "depth"),
    (dict(in_ch=4), "in_ch"),
    (dict(width=384, heads=6), "power of two"),
])
def test_model_create_rejects_bad_shapes(kw, msg):
    with pytest.raises(f3c.F3CError) as e:
        f3c.Model(_cfg(**kw))
    assert e.value.code == f3c.F3C_EINVAL and msg in str(e.value)


def test_state_bytes_and_batch_limits(L):
    m = f3c.Model(synth.TRELLIS16)
    b = ctypes.c_size_t()
    assert L.f3c_state_bytes(m.h, 1, ctypes.byref(b)) == 0 and b.value > 0
    b4 = ctypes.c_size_t()
    assert L.f3c_state_bytes(m.h, 4, ctypes.byref(b4)) == 0 and b4.value > 3 * b.value
    assert L.f3c_state_bytes(m.h, 0, ctypes.byref(b)) == f3c.F3C_EINVAL
    assert L.f3c_state_bytes(m.h, 65, ctypes.byref(b)) == f3c.F3C_EINVAL


def test_guided_state_bytes_and_limits(L):
    m = f3c.Model(synth.TRELLIS16)
    plain, guided = ctypes.c_size_t(), ctypes.c_size_t()
    assert L.f3c_state_bytes_ex(m.h, 2, 0, ctypes.byref(plain)) == 0
    assert L.f3c_state_bytes_ex(m.h, 2, f3c.F3C_STATE_GUIDED, ctypes.byref(guided)) == 0
    legacy = ctypes.c_size_t()
    assert L.f3c_state_bytes(m.h, 2, ctypes.byref(legacy)) == 0 and legacy.value == plain.value
    # activations and condition K/V double; caches and selection buffers do not
    assert plain.value < guided.value < 2 * plain.value
    assert L.f3c_state_bytes_ex(m.h, 32, f3c.F3C_STATE_GUIDED, ctypes.byref(guided)) == 0
    assert L.f3c_state_bytes_ex(m.h, 33, f3c.F3C_STATE_GUIDED, ctypes.byref(guided)) == f3c.F3C_EINVAL
    assert b"guided" in L.f3c_last_error()
    assert L.f3c_state_bytes_ex(m.h, 1, 6, ctypes.byref(guided)) == f3c.F3C_EINVAL
    assert L.f3c_guided_step(None, None, 1.0, 0.5, None, 3.0, None) == f3c.F3C_EINVAL
    assert L.f3c_set_uncond(None, None, None) == f3c.F3C_EINVAL


def test_modulation_plan_bytes_and_host_checks(L):
    """Plan size: the trajectory's modulation vectors [n][L][6][width] and the
    time-embedding scratch [n][2][width], each 256-byte aligned; a 25-step
    plan of the 24-block width-1024 model holds 14.2 MiB."""
    m = f3c.Model(synth.TRELLIS16)
    b = ctypes.c_size_t()
    assert L.f3c_plan_bytes(m.h, 25, ctypes.byref(b)) == 0
    assert b.value == 25 * 24 * 6 * 1024 * 4 + 25 * 2 * 1024 * 4
    assert L.f3c_plan_bytes(m.h, 0, ctypes.byref(b)) == 0 and b.value == 0
    assert L.f3c_plan_bytes(m.h, 1, ctypes.byref(b)) == 0 and b.value == 147456 * 4 + 8192
    assert L.f3c_plan_bytes(m.h, 1024, ctypes.byref(b)) == 0
    assert L.f3c_plan_bytes(m.h, 1025, ctypes.byref(b)) == f3c.F3C_EINVAL
    assert L.f3c_plan_bytes(m.h, -1, ctypes.byref(b)) == f3c.F3C_EINVAL
    assert L.f3c_plan_bytes(None, 1, ctypes.byref(b)) == f3c.F3C_EINVAL
    assert L.f3c_state_plan_times(None, None, 0, None, 0, None) == f3c.F3C_EINVAL


def test_guidance_interval_matches_oracle():
    from oracle import schedule as osched
    for eta in (1.0, 2.0, 3.0):
        for t in f3c.time_grid(25, eta):
            for lo, hi in ((0.5, 1.0), (0.0, 1.0), (0.25, 0.75)):
                assert f3c.guidance_active(t, lo, hi) == osched.cfg_active(t, lo, hi)
    for t in (0.5, 1.0, np.nextafter(0.5, 0.0), 0.0):
        assert f3c.guidance_active(t) == osched.cfg_active(t)


def test_steps_need_loaded_weights_and_valid_quota(L):
    # state creation needs device memory; the checks below fail before touching it
    assert L.f3c_full_step(None, None, 1.0, 0.5, None) == f3c.F3C_EINVAL
    assert L.f3c_cached_step(None, None, 1.0, 0.5, None, None) == f3c.F3C_EINVAL


def test_op_entry_validation_is_host_side(L):
    q = f3c._i32([0, 5])
    assert L.f3c_op_select(0, 512, 1, 1, 0.7, q, 1, 1, None, 256, 1 << 20, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select(1, 512, 1, 1, 1.5, q, 1, 1, None, 256, 1 << 20, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select(1, 4, 1, 1, 0.7, f3c._i32([5]), 1, 1, None, 256, 1 << 20, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select(1, 40000, 1, 1, 0.7, f3c._i32([5]), 1, 1, None, 256, 1 << 20, None) == f3c.F3C_EINVAL
    # workspace: missing, misaligned, too small
    assert L.f3c_op_select(1, 512, 1, 1, 0.7, q, 1, 1, None, None, 1 << 20, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select(1, 512, 1, 1, 0.7, q, 1, 1, None, 128, 1 << 20, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select(1, 512, 1, 1, 0.7, q, 1, 1, None, 256, 64, None) == f3c.F3C_ENOMEM
    # selection from given scores: NULL scores, quota outside [0, N], bad shapes
    assert L.f3c_op_select_scores(1, 512, None, q, 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select_scores(1, 4, 1, f3c._i32([5]), 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select_scores(1, 4, 1, f3c._i32([-1]), 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select_scores(65, 4, 1, f3c._i32([0] * 65), 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select_scores(1, 40000, 1, f3c._i32([5]), 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_select_scores(1, 512, 1, q, None, 1, None) == f3c.F3C_EINVAL
    assert f3c.select_workspace_bytes(1, 512) == 512 * 8 + 16
    assert f3c.select_workspace_bytes(4, 32768) == 4 * 32768 * 8 + 4 * 32 * 16
    assert L.f3c_op_gemm(1, 0, 16, 100, 64, 1, 64, 1, 64, 1, None, 1, 100, None, 0, None) == f3c.F3C_EINVAL
    assert L.f3c_op_gemm(1, 0, 16, 128, 40, 1, 40, 1, 40, 1, None, 1, 128, None, 0, None) == f3c.F3C_EINVAL
    assert L.f3c_op_gemm(1, 0, 16, 128, 64, 1, 64, 1, 64, 1, None, 1, 130, None, 0, None) == f3c.F3C_EINVAL
    assert L.f3c_op_attention(1, 4, 48, 1, q, q, 1, 192, 1, 192, 1, 192, 1, 192, None, 0, 0, None) == f3c.F3C_EINVAL
    assert L.f3c_op_attention(1, 4, 64, 1, q, q, 16, 256, 16, 256, 16, 256, 16, 256, None, 0, 2, None) == f3c.F3C_EINVAL
    assert L.f3c_op_attention(1, 4, 64, 1, f3c._i32([0, 3]), f3c._i32([0, 0]), 1, 256, 1, 256, 1, 256, 1, 256,
                              None, 0, 0, None) == f3c.F3C_EINVAL
    assert L.f3c_op_attention(1, 4, 64, 1, f3c._i32([0, 3]), f3c._i32([0, 3]), 16, 256, 16, 256, 16, 256, 16, 256,
                              4, 1024, 0, None) == f3c.F3C_EINVAL
    assert b"16-byte aligned" in L.f3c_last_error()
    # bf16, 64-wide heads: one sample's key rows must span less than 2 GiB (32-bit DMA offsets)
    assert L.f3c_op_attention(1, 1, 64, 1, f3c._i32([0, 1]), f3c._i32([0, 32768]), 16, 64, 16, 32768, 16, 64,
                              16, 64, None, 0, 0, None) == f3c.F3C_EINVAL
    assert b"2 GiB" in L.f3c_last_error()
    assert L.f3c_op_ln_mod(1, 4, 96, 1, None, None, 1, None) == f3c.F3C_EINVAL
    assert b"unsupported d" in L.f3c_last_error()
    m = f3c.Model(_cfg())                                   # no weights loaded
    assert L.f3c_op_embed(m.h, 1, 1, None, f3c._i32([0, 512]), 1, None) == f3c.F3C_ESTATE
    assert L.f3c_op_final(m.h, 4, 1, 1, None) == f3c.F3C_ESTATE
    off = f3c._i32([0, 10, 20])
    assert L.f3c_op_euler(2, 16, 1, 2, 3, 4, off, 1.0, 0.5, 2, None) == f3c.F3C_EINVAL     # v_new aliases v_cache
    assert b"alias" in L.f3c_last_error()
    assert L.f3c_op_euler(2, 16, 1, 2, 3, 4, off, math.inf, 0.5, 5, None) == f3c.F3C_EINVAL
    assert L.f3c_op_euler(2, 8, 1, 2, 3, 4, off, 1.0, 0.5, 5, None) == f3c.F3C_EINVAL     # segment > n_tokens
    assert L.f3c_op_euler(2, 16, 1, 2, 3, None, off, 1.0, 0.5, 5, None) == f3c.F3C_EINVAL  # pos NULL, partial
    assert L.f3c_op_euler(2, 16, 1, 2, None, 4, off, 1.0, 0.5, 5, None) == f3c.F3C_EINVAL  # rows but no v_act
    assert L.f3c_op_euler(2, 16, 1, 2, 3, 4, f3c._i32([0, 10, 5]), 1.0, 0.5, 5, None) == f3c.F3C_EINVAL
    assert L.f3c_op_pack_occupancy(1, 64, None, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_pack_occupancy(0, 64, 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_pack_occupancy(1, 0, 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_pack_occupancy(65536, 64, 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_dynamic_voxels(1, 2, 1, None, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_dynamic_voxels(1, 0, 1, 1, 1, None) == f3c.F3C_EINVAL
    assert L.f3c_op_dynamic_voxels(0, 2, 1, 1, 1, None) == f3c.F3C_EINVAL


@pytest.mark.parametrize("steps,eta", [(10, 1.0), (25, 3.0), (25, 2.0), (50, 1.5)])
def test_time_grid_matches_oracle_bitwise(steps, eta):
    got = f3c.time_grid(steps, eta)
    want = np.array(osched.time_grid(steps, eta))
    assert np.array_equal(got, want)


def test_ceil_ratio_and_phase_rule_match_oracle():
    for T in (10, 20, 25, 40, 50):
        for rho in (0.1, 0.2, 0.25, 0.3, 0.5, 0.6, 0.7, 0.75, 0.8):
            assert f3c.ceil_ratio(T, rho) == osched.ceil_ratio(T, rho)
    for T in (10, 25):
        for f_corr in (0, 1, 2, 3, 4):
            for xi in (0.7, 0.8, 0.9):
                for k in range(1, T + 1):
                    assert f3c.phase_quota(k, T, 4096, 1234, 0.2, 0.75, xi, f_corr) == \
                        osched.phase_quota(k, T, 4096, 1234, 0.2, 0.75, xi, f_corr)


def test_ceil_ratio_is_exact_on_decimals():
    # ratios are decimals: a ratio a hair above a fraction that lands on an
    # integer must take the next integer, exactly as the oracle's exact ceiling
    assert f3c.ceil_ratio(25, 0.2) == osched.ceil_ratio(25, 0.2) == 5
    assert f3c.ceil_ratio(25, 0.2000000001) == osched.ceil_ratio(25, 0.2000000001) == 6
    assert f3c.ceil_ratio(10, 0.30000000001) == osched.ceil_ratio(10, 0.30000000001) == 4
    assert f3c.ceil_ratio(25, 0.7599999999999999) == osched.ceil_ratio(25, 0.7599999999999999) == 19
    assert f3c.ceil_ratio(25, 0.76) == osched.ceil_ratio(25, 0.76) == 19
    assert f3c.ceil_ratio(25, 0.0) == 0 and f3c.ceil_ratio(0, 0.5) == 0
    assert f3c.ceil_ratio(25, 5e-324) == osched.ceil_ratio(25, 5e-324) == 1
    rng = np.random.default_rng(7)
    cases = [float(v) for v in rng.random(3000)]
    cases += [round(float(v), int(p)) for v, p in zip(rng.random(3000), rng.integers(1, 17, 3000))]
    cases += [2.0 ** -e for e in range(1, 60)] + [1.0 - 2.0 ** -e for e in range(1, 53)]
    cases += [np.nextafter(v, 1.0) for v in (0.2, 0.25, 0.3, 0.75, 0.7)]
    cases += [np.nextafter(v, 0.0) for v in (0.2, 0.25, 0.3, 0.75, 0.7)]
    for rho in cases:
        for T in (1, 7, 25, 1000, 2 ** 31 - 1):
            assert f3c.ceil_ratio(T, rho) == min(osched.ceil_ratio(T, rho), 2 ** 31 - 1), (T, rho)


def test_phase_quota_floor_is_exact_on_decimals():
    # N * xi just below and at an integer: the floor of the exact decimal product
    k3 = 20                                   # a Phase 3 step at T = 25, no correction with f_corr = 0
    for N, xi in [(32768, 0.7), (4096, 0.7), (10, 0.3), (10, 0.29999999999), (10, 0.30000000001),
                  (3, 1.0 / 3.0), (1000, 0.0009999999999999998), (1000, 0.001), (7, 0.9999999999999999)]:
        got = f3c.phase_quota(k3, 25, N, 0, 0.2, 0.75, xi, 0)
        want = osched.phase_quota(k3, 25, N, 0, 0.2, 0.75, xi, 0)
        assert got == want, (N, xi, got, want)
    assert f3c.phase_quota(k3, 25, 10, 0, 0.2, 0.75, 0.29999999999, 0) == 2
    assert f3c.phase_quota(k3, 25, 10, 0, 0.2, 0.75, 0.3, 0) == 3
    rng = np.random.default_rng(11)
    for xi in [round(float(v), int(p)) for v, p in zip(rng.random(2000), rng.integers(1, 17, 2000))]:
        for N in (512, 4096, 32768):
            assert f3c.phase_quota(k3, 25, N, 0, 0.2, 0.75, xi, 0) == osched.phase_quota(k3, 25, N, 0, 0.2, 0.75,
                                                                                         xi, 0), (N, xi)


def test_pcsc_quota_matches_oracle():
    for N in (512, 4096, 32768):
        for sigma in (0.0, 100.0, 6400.0, 2e5, 1e9):
            for mu in (-0.7, -0.07, -0.007):
                for k in range(5, 26):
                    assert f3c.pcsc_quota(k, N, sigma, mu, 5, 64.0) == osched.pcsc_quota(k, N, sigma, mu, 5, 64.0)


@pytest.mark.parametrize("wname", sorted(synth.WORKLOADS))
def test_forward_flops_matches_oracle(wname):
    cfg = synth.WORKLOADS[wname].model
    for n in (0, 1, 820, cfg.tokens):
        for B in (1, 4):
            assert math.isclose(f3c.forward_flops(cfg, n, B), oflops.forward_flops(cfg, n, B), rel_tol=1e-12)


def test_driver_is_built_and_checks_arguments():
    # argument errors are reported before any HIP call, so this runs without a GPU
    from paper_2511_22533_amd import build
    for args, msg in [(["--bogus"], "unknown argument"), (["--quotas", "1,2"], "one count per step"),
                      (["--steps", "2", "--quotas", "0,-1"], "quota outside")]:
        r = subprocess.run([build.DRIVER, *args], capture_output=True, text=True)
        assert r.returncode == 1 and msg in r.stderr, (args, r.stderr)


def test_bench_counter_traffic_lookup(tmp_path, monkeypatch):
    import bench
    v, why = bench.counter_traffic("attn_self", "no_such_workload", [1])
    assert v is None and "no counter summary" in why
    # a planted summary: per-step lines, averaged over the timed steps' launches
    import hashlib
    csrc = os.path.join(bench.ROOT, "paper_2511_22533_amd", "csrc")
    digest = hashlib.sha256(open(os.path.join(csrc, "k_attn.hip"), "rb").read()).hexdigest()
    prof = tmp_path / "profiles"
    prof.mkdir()
    lines = [f"traffic attn_self k={k}: {1000 * k} bytes over 2 calls; sources k_attn.hip sha256 {digest}"
             for k in (1, 2, 3)]
    (prof / "demo_traffic.md").write_text("\n".join(lines) + "\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "paper_2511_22533_amd", exist_ok=True)
    os.symlink(csrc, tmp_path / "paper_2511_22533_amd" / "csrc")
    v, why = bench.counter_traffic("attn_self", "demo", [1, 2, 3])
    assert v == round((1000 + 2000 + 3000) / 6)
    v, why = bench.counter_traffic("attn_self", "demo", [3, 3])
    assert v == 1500
    v, why = bench.counter_traffic("attn_self", "demo", [4])
    assert v is None and "every timed step" in why
    v, why = bench.counter_traffic("gemm_o", "demo", [1])
    assert v is None and "no counter line" in why
    (prof / "demo_traffic.md").write_text(lines[0].replace(digest, "0" * 64) + "\n")
    v, why = bench.counter_traffic("attn_self", "demo", [1])
    assert v is None and "changed" in why


@pytest.mark.parametrize("steps", [10, 25, 50])
@pytest.mark.parametrize("tau,reading", [(0, 0), (1, 0), (1, 1), (2, 0), (3, 0), (3, 1), (5, 0), (8, 1)])
@pytest.mark.parametrize("f_corr", [0, 1, 3])
def test_schedule_plan_matches_oracle(steps, tau, reading, f_corr):
    for n, sigma, mu, g, xi in [(512, 40.0, -0.07, 1.0, 0.7), (4096, 900.0, -0.05, 4.0, 0.55),
                                (32768, 30000.0, -0.12, 64.0, 0.8), (4096, 1e7, -0.07, 1.0, 0.7)]:
        got = f3c.schedule_plan(steps, n, sigma, mu=mu, gamma_up=g, xi=xi, f_corr=f_corr, tau=tau, reading=reading)
        want = osched.plan(steps, n, sigma, mu=mu, gamma_up=g, xi=xi, f_corr=f_corr, tau=tau, reading=reading)
        assert got.tolist() == want
    for run in range(12):
        assert f3c.tau_forces_full(run, tau, reading) == osched.tau_forces_full(run, tau, reading)


def test_schedule_plan_validation(L):
    with pytest.raises(f3c.F3CError):
        f3c.schedule_plan(25, 4096, 10.0, gamma_up=0.0)
    with pytest.raises(f3c.F3CError):
        f3c.schedule_plan(25, 4096, 10.0, reading=7)
    with pytest.raises(f3c.F3CError):
        f3c.schedule_plan(0, 4096, 10.0)
    with pytest.raises(f3c.F3CError):
        f3c.schedule_plan(25, 4096, float("nan"))
