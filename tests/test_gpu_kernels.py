"""GPU parity of each kernel of the step, through the C ABI, against the oracle.

* scoring + selection: bit-exact scores, index sets and position map (Eqs. 2,
  6, 7; Algorithm 1 SSC), including ties, NaN, quota 0 / N and ragged batches,
  up to 32768 tokens per sample;
* projections (MFMA GEMM, each epilogue) and attention (self, ragged varlen,
  cross with a non-tile-multiple key count) against float64 on the same
  bf16-rounded operands; bf16 bound 2e-2 max-rel, f32 bound 1e-4;
* LayerNorm/modulation and the timestep modulation path;
* gather + embedding and the final LayerNorm + output projection against
  float64; merge + Euler + cache rotation bit-exact against the oracle step.
"""
import numpy as np
import pytest

from helpers import bf16_round, max_rel, oracle_selection, say, to_dev
from oracle import dit, ssc
from paper_2511_22533_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    from paper_2511_22533_amd import f3c
    f3c.lib()
    return t


def _run_select(torch, vc, vp, n_cache, omega):
    from paper_2511_22533_amd import f3c
    B, N = vc.shape[:2]
    total = int(sum(N - c for c in n_cache))
    d_vc, d_vp = to_dev(vc), to_dev(vp)
    idx = torch.full((max(total, 1),), -7, dtype=torch.int32, device="cuda")
    pos = torch.full((B, N), -7, dtype=torch.int32, device="cuda")
    score = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    f3c.op_select(d_vc, d_vp, omega, n_cache, idx, pos, score)
    torch.cuda.synchronize()
    return idx.cpu().numpy()[:total], pos.cpu().numpy(), score.cpu().numpy()


def _check_select(torch, vc, vp, n_cache, omega=0.7):
    B, N = vc.shape[:2]
    idx, pos, score = _run_select(torch, vc, vp, n_cache, omega)
    ref = oracle_selection(vc, vp, n_cache, omega)
    row = 0
    for b in range(B):
        s_ref, active = ref[b]
        n = len(active)
        assert n == N - n_cache[b]
        assert np.array_equal(idx[row:row + n], active), f"sample {b}"
        want_pos = np.full(N, -1, np.int64)
        want_pos[active] = row + np.arange(n)
        assert np.array_equal(pos[b], want_pos), f"sample {b}"
        if s_ref is not None:
            assert np.array_equal(score[b].view(np.uint32), s_ref.view(np.uint32)), f"scores sample {b}"
        row += n


@pytest.mark.parametrize("B,N", [(1, 512), (1, 4096), (4, 4096), (1, 32768), (3, 1000), (2, 1), (5, 3000), (16, 32768)])
def test_select_bit_exact_random(torch, B, N):
    rng = np.random.default_rng(N + B)
    vc = rng.standard_normal((B, N, 8)).astype(np.float32)
    vp = (vc + 0.1 * rng.standard_normal((B, N, 8))).astype(np.float32)
    for quotas in ([0] * B, [N] * B, [1] * B, [N - 1] * B,
                   [int(q) for q in rng.integers(0, N + 1, size=B)],
                   [int(N * f) for f in np.linspace(0.4, 0.85, B)]):
        say("select", B, N, quotas)
        _check_select(torch, vc, vp, quotas)


@pytest.mark.parametrize("omega", [0.0, 0.3, 0.7, 1.0])
def test_select_ties_and_sticky_cache(torch, omega):
    rng = np.random.default_rng(11)
    B, N = 2, 4096
    vc = (rng.integers(-2, 3, size=(B, N, 8)) * 0.5).astype(np.float32)   # many equal scores
    vp = vc.copy()
    moved = rng.random((B, N)) < 0.3
    vp[moved] += 0.5                                                      # A = 0 for the rest
    say("select ties", omega)
    _check_select(torch, vc, vp, [1000, 3000], omega)


def test_select_degenerate_and_nan(torch):
    B, N = 3, 2048
    vc = np.ones((B, N, 8), np.float32)
    vp = np.ones((B, N, 8), np.float32)             # max == min for both terms
    rng = np.random.default_rng(3)
    vc[1] = rng.standard_normal((N, 8)).astype(np.float32)
    vp[1] = rng.standard_normal((N, 8)).astype(np.float32)
    vc[1, 17, 3] = np.nan
    vc[1, 900, :] = np.inf
    vc[2] = rng.standard_normal((N, 8)).astype(np.float32)
    vp[2] = vc[2]
    say("select degenerate/nan")
    _check_select(torch, vc, vp, [100, 1500, 2047])


# The selection alone from given scores (f3c_op_select_scores) against the
# oracle's stable sort of the same scores: ragged quotas including 0, 1, N - 1
# and N; heavy ties (a few distinct values), NaN, +-inf, +-0 and subnormals.
@pytest.mark.parametrize("B,N", [(1, 1), (3, 1000), (4, 4096), (2, 32768)])
def test_select_from_given_scores(torch, B, N):
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(7 * N + B)
    cases = {
        "continuous": rng.standard_normal((B, N)).astype(np.float32),
        "ties": (rng.integers(0, 5, size=(B, N)) * 0.25).astype(np.float32),
    }
    special = rng.random((B, N)).astype(np.float32)
    picks = rng.integers(0, N, size=(B, 6 * max(1, N // 64)))
    for b in range(B):
        for j, i in enumerate(picks[b]):
            special[b, i] = [np.nan, np.inf, -np.inf, 0.0, -0.0, np.float32(1e-45)][j % 6]
    cases["special"] = special
    for name, sc in cases.items():
        quota_sets = [[0] * B, [N] * B, [min(1, N)] * B, [max(N - 1, 0)] * B,
                      [int(q) for q in rng.integers(0, N + 1, size=B)]]
        for quotas in quota_sets:
            say("select scores", name, B, N, quotas)
            tot = sum(N - c for c in quotas)
            idx = torch.full((max(tot, 1),), -7, dtype=torch.int32, device="cuda")
            pos = torch.full((B, N), -7, dtype=torch.int32, device="cuda")
            f3c.op_select_scores(to_dev(sc), quotas, idx, pos)
            torch.cuda.synchronize()
            got_idx, got_pos = idx.cpu().numpy(), pos.cpu().numpy()
            row = 0
            for b in range(B):
                _, active = ssc.select(sc[b], quotas[b])
                n = len(active)
                assert np.array_equal(got_idx[row:row + n], active), (name, quotas, b)
                want_pos = np.full(N, -1, np.int64)
                want_pos[active] = row + np.arange(n)
                assert np.array_equal(got_pos[b], want_pos), (name, quotas, b)
                row += n


def _gemm_case(torch, dt, epi, M, N, K, seed):
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (0.05 * rng.standard_normal((N, K))).astype(np.float32)
    bias = rng.standard_normal(N).astype(np.float32)
    gate = rng.standard_normal(N).astype(np.float32)
    if dt == f3c.F3C_BF16:
        A, W = bf16_round(A), bf16_round(W)
        tdt = torch.bfloat16
    else:
        tdt = torch.float32
    ref = A.astype(np.float64) @ W.astype(np.float64).T + bias
    dA, dW, db, dg = to_dev(A, tdt), to_dev(W, tdt), to_dev(bias), to_dev(gate)
    say("gemm", dt, epi, M, N, K)
    if epi == 2:
        r0 = rng.standard_normal((M, N)).astype(np.float32)
        dr = to_dev(r0)
        f3c.op_gemm(dt, 2, dA, dW, db, resid=dr, gate=dg)
        torch.cuda.synchronize()
        got = dr.cpu().numpy().astype(np.float64) - r0
        want = gate * ref
    else:
        out = torch.empty((M, N), dtype=tdt, device="cuda")
        f3c.op_gemm(dt, epi, dA, dW, db, out=out)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
        want = dit.gelu_tanh(ref) if epi == 1 else ref
    return got, want


# Tile shapes picked: 64 x 64 for the first four, 128 x 128 for 4096 x 1024 x
# 4096 and 2057 x 4096, 64 x 128 for 1310 x 3072.
@pytest.mark.parametrize("M,N,K", [(1, 128, 64), (37, 384, 128), (128, 1024, 1024), (820, 3072, 1024),
                                   (4096, 1024, 4096), (2057, 4096, 1024), (1310, 3072, 1024)])
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_gemm_bf16(torch, M, N, K, epi):
    from paper_2511_22533_amd import f3c
    got, want = _gemm_case(torch, f3c.F3C_BF16, epi, M, N, K, seed=M * 7 + N + epi)
    assert max_rel(got, want) < 1e-2


# Long K: one round of 64 x 64 workgroups (M up to 1024 at N = 1024) or of
# 64 x 128 (up to 2048) goes to the kernel whose waves split each K tile in
# four groups and sum the groups' partial blocks through LDS in a fixed order:
# ragged M, both tile shapes, every epilogue, and bit-reproducible repeats.
@pytest.mark.parametrize("M,N,K", [(1, 128, 4096), (37, 1024, 4096), (820, 1024, 4096), (1500, 1024, 4096),
                                   (2048, 1024, 4096), (300, 2048, 8192)])
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_gemm_bf16_long_k(torch, M, N, K, epi):
    from paper_2511_22533_amd import f3c
    got, want = _gemm_case(torch, f3c.F3C_BF16, epi, M, N, K, seed=M + K + epi)
    assert max_rel(got, want) < 1e-2
    got2, _ = _gemm_case(torch, f3c.F3C_BF16, epi, M, N, K, seed=M + K + epi)
    assert np.array_equal(got, got2)


def _gemm_big_case(torch, epi, M, N, K, seed, rows=None):
    """bf16 projection at many rows; the float64 reference on sampled rows."""
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(seed)
    A = bf16_round(rng.standard_normal((M, K)).astype(np.float32))
    W = bf16_round((0.05 * rng.standard_normal((N, K))).astype(np.float32))
    bias = rng.standard_normal(N).astype(np.float32)
    gate = rng.standard_normal(N).astype(np.float32)
    dA, dW, db, dg = to_dev(A, torch.bfloat16), to_dev(W, torch.bfloat16), to_dev(bias), to_dev(gate)
    say("gemm big", epi, M, N, K)
    if epi == 2:
        r0 = rng.standard_normal((M, N)).astype(np.float32)
        dr = to_dev(r0)
        f3c.op_gemm(f3c.F3C_BF16, 2, dA, dW, db, resid=dr, gate=dg)
        torch.cuda.synchronize()
        got = dr.cpu().numpy()
        base = r0
    else:
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        f3c.op_gemm(f3c.F3C_BF16, epi, dA, dW, db, out=out)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
        base = None
    if rows is None:
        rows = np.unique(np.concatenate([rng.choice(M, 384, replace=False), np.arange(M - 130, M)]))
    ref = A[rows].astype(np.float64) @ W.astype(np.float64).T + bias
    if epi == 2:
        return got, (got[rows].astype(np.float64) - base[rows], gate * ref)
    return got, (got[rows], dit.gelu_tanh(ref) if epi == 1 else ref)


# Many rows (the 32^3 workload's active sets) go to the 256 x 256 tiles for the
# QKV projection shape and both MLP projections from 8192 rows: ragged row
# counts, every epilogue, sampled rows against float64.
@pytest.mark.parametrize("M,N,K", [(8300, 3072, 1024), (9831, 1024, 4096), (16500, 1024, 4096),
                                   (9831, 4096, 1024), (16400, 4096, 1024)])
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_gemm_bf16_many_rows(torch, M, N, K, epi):
    _, (got, want) = _gemm_big_case(torch, epi, M, N, K, seed=M + epi)
    assert max_rel(got, want) < 1e-2


# The tile choice moves with the row count, not the results: the 256 x 256
# kernel sums K in the same order with the same instruction as the 128 x 128
# one, so the rows shared by a run just below the switch and one at it agree
# bit for bit.
@pytest.mark.parametrize("M,N,K", [(8192, 3072, 1024), (8192, 1024, 4096), (8192, 4096, 1024)])
@pytest.mark.parametrize("epi", [0, 2])
def test_gemm_bf16_tile_switch_bit_identical(torch, M, N, K, epi):
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(M + N + epi)
    A = to_dev(rng.standard_normal((M, K)).astype(np.float32), torch.bfloat16)
    W = to_dev((0.05 * rng.standard_normal((N, K))).astype(np.float32), torch.bfloat16)
    bias = to_dev(rng.standard_normal(N).astype(np.float32))
    gate = to_dev(rng.standard_normal(N).astype(np.float32))
    outs = []
    for rows in (M, M - 1):          # at the switch (256 x 256 tiles), just below it
        say("gemm tile switch", epi, rows, N, K)
        if epi == 2:
            r = torch.zeros((rows, N), dtype=torch.float32, device="cuda")
            f3c.op_gemm(f3c.F3C_BF16, 2, A[:rows], W, bias, resid=r, gate=gate)
        else:
            r = torch.empty((rows, N), dtype=torch.bfloat16, device="cuda")
            f3c.op_gemm(f3c.F3C_BF16, epi, A[:rows], W, bias, out=r)
        torch.cuda.synchronize()
        outs.append(r.float().cpu().numpy())
    assert np.array_equal(outs[0][:M - 1].view(np.uint32), outs[1].view(np.uint32))


@pytest.mark.parametrize("M,N,K", [(1, 128, 32), (300, 384, 128), (513, 512, 128)])
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_gemm_f32(torch, M, N, K, epi):
    from paper_2511_22533_amd import f3c
    got, want = _gemm_case(torch, f3c.F3C_F32, epi, M, N, K, seed=M + N + K + epi)
    assert max_rel(got, want) < 1e-5


def _attn_case(torch, dt, heads, hd, q_lens, k_lens, seed, sample_queries=None, workspace=False, outputs=None,
               key_ramp=0.0, prescaled=False):
    """key_ramp > 0 scales key j of each sample by 1 + key_ramp * (j // 64): every
    64-key tile then has larger scores than the ones before it. prescaled: the
    queries go in multiplied by log2(e)/sqrt(hd) (rounded once, as the step's
    projections store them) and the reference takes the stored values divided
    by that factor."""
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(seed)
    d = heads * hd
    q_off = np.concatenate([[0], np.cumsum(q_lens)]).astype(int)
    k_off = np.concatenate([[0], np.cumsum(k_lens)]).astype(int)
    q = (1.5 * rng.standard_normal((q_off[-1], d))).astype(np.float32)
    k = (1.5 * rng.standard_normal((k_off[-1], d))).astype(np.float32)
    v = rng.standard_normal((k_off[-1], d)).astype(np.float32)
    if key_ramp:
        j = np.concatenate([np.arange(n) for n in k_lens]) if k_off[-1] else np.zeros(0, int)
        k *= (1.0 + key_ramp * (j // 64)).astype(np.float32)[:, None]
    tdt = torch.bfloat16 if dt == f3c.F3C_BF16 else torch.float32
    cq = f3c.attention_q_scale(hd) if prescaled else 1.0
    q_in = (q * np.float32(cq)).astype(np.float32)
    if dt == f3c.F3C_BF16:
        q_in, k, v = bf16_round(q_in), bf16_round(k), bf16_round(v)
    q = (q_in.astype(np.float64) / cq) if prescaled else q_in     # what the kernel's input means
    o = torch.zeros((max(q_off[-1], 1), d), dtype=tdt, device="cuda")
    ws = torch.empty(8 << 20, dtype=torch.float32, device="cuda") if workspace else None
    say("attention", dt, heads, hd, list(q_lens), list(k_lens), "workspace" if workspace else "")
    f3c.op_attention(dt, heads, hd, q_off.tolist(), k_off.tolist(), to_dev(q_in, tdt), to_dev(k, tdt),
                     to_dev(v, tdt), o, workspace=ws, q_prescaled=prescaled)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    if outputs is not None:
        outputs.append(got)
    worst = 0.0
    for b in range(len(q_lens)):
        if q_lens[b] == 0:
            continue
        rows = np.arange(q_off[b], q_off[b + 1])
        if sample_queries and len(rows) > sample_queries:
            rows = np.sort(rng.choice(rows, sample_queries, replace=False))
        kk = k[k_off[b]:k_off[b + 1]].astype(np.float64)
        vv = v[k_off[b]:k_off[b + 1]].astype(np.float64)
        want = dit.attention(q[rows].astype(np.float64), kk, vv, heads)
        worst = max(worst, max_rel(got[rows], want))
    return worst


# 1024 and 1025 queries sit on either side of the switch from four-wave to
# eight-wave key-group workgroups (16 x 16 = 256 workgroups of 64 queries is
# the last grid that fits one round).
@pytest.mark.parametrize("q_lens,k_lens", [([64], [64]), ([1], [1]), ([200], [200]), ([0, 37, 300], [0, 37, 300]),
                                           ([820], [820]), ([615, 1536, 2458, 1003], [615, 1536, 2458, 1003]),
                                           ([1024], [1024]), ([1025], [1025])])
@pytest.mark.parametrize("prescaled", [False, True])
def test_self_attention_bf16(torch, q_lens, k_lens, prescaled):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_BF16, 16, 64, q_lens, k_lens, seed=sum(q_lens), prescaled=prescaled) < 2e-2


@pytest.mark.parametrize("prescaled", [False, True])
def test_self_attention_bf16_full_size_sampled(torch, prescaled):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_BF16, 16, 64, [4096], [4096], seed=5, sample_queries=96,
                      prescaled=prescaled) < 2e-2
    assert _attn_case(torch, f3c.F3C_BF16, 16, 64, [9831], [9831], seed=6, sample_queries=64,
                      prescaled=prescaled) < 2e-2


@pytest.mark.parametrize("q_lens", [[820], [5, 1000, 0, 77]])
@pytest.mark.parametrize("prescaled", [False, True])
def test_cross_attention_bf16(torch, q_lens, prescaled):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_BF16, 16, 64, q_lens, [1374] * len(q_lens), seed=len(q_lens),
                      prescaled=prescaled) < 2e-2


# With a workspace, launches with few query tiles may split the key range
# over workgroups and merge the partial results in a fixed order; they do
# when that shortens each wave's chain of key tiles by more than five tiles
# against two key groups in one workgroup. Chosen for these cases (bf16, 16
# heads): key groups of four waves for the first four, 4 splits, 8 splits,
# key groups of eight waves, key groups of four waves.
@pytest.mark.parametrize("q_lens,k_lens", [([1000], [1000]), ([820], [1374]), ([5, 300, 0, 77], [1374] * 4),
                                           ([300], [1374]), ([1, 40], [4096, 2000]), ([64], [8192]),
                                           ([1310], [1310]), ([820], [820])])
@pytest.mark.parametrize("prescaled", [False, True])
def test_attention_bf16_split_keys(torch, q_lens, k_lens, prescaled):
    from paper_2511_22533_amd import f3c
    outs = []
    for rep in range(2):
        assert _attn_case(torch, f3c.F3C_BF16, 16, 64, q_lens, k_lens, seed=sum(k_lens), workspace=True,
                          outputs=outs, prescaled=prescaled) < 2e-2
    assert np.array_equal(outs[0], outs[1])


# Scores that grow from tile to tile: the running reference max of the
# matrix-core path is too small for later tiles, so its fix-up branch
# (rescale what was accumulated, redo the tile) runs, for some queries of a
# wave and not others; in the four-wave key-group, eight-wave and key-split
# (300 x 4096 keys: 4 splits) launches.
@pytest.mark.parametrize("q_lens,k_lens,ramp,ws", [([300], [300], 2.0, False), ([1000], [1000], 0.5, False),
                                                   ([820], [1374], 1.0, False), ([300], [4096], 0.5, True),
                                                   ([37, 3000], [37, 3000], 0.3, False), ([640], [640], 0.12, False)])
@pytest.mark.parametrize("prescaled", [False, True])
def test_attention_bf16_growing_scores(torch, q_lens, k_lens, ramp, ws, prescaled):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_BF16, 16, 64, q_lens, k_lens, seed=int(10 * ramp) + len(q_lens),
                      workspace=ws, key_ramp=ramp, sample_queries=128, prescaled=prescaled) < 2e-2


# Two key groups with one or two key tiles: the second group's only tile lies
# past the end (all keys masked) or is the ragged last one; four-wave
# workgroups up to 1024 queries, eight-wave ones at 1100.
@pytest.mark.parametrize("q_lens,k_lens", [([600], [50]), ([600], [64]), ([700], [100]), ([5, 600], [1, 65]),
                                           ([1100], [50]), ([1100], [100])])
@pytest.mark.parametrize("prescaled", [False, True])
def test_attention_bf16_key_groups_short_keys(torch, q_lens, k_lens, prescaled):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_BF16, 16, 64, q_lens, k_lens, seed=sum(k_lens), prescaled=prescaled) < 2e-2


@pytest.mark.parametrize("hd,heads", [(32, 4), (64, 2)])
def test_attention_f32_split_keys(torch, hd, heads):
    from paper_2511_22533_amd import f3c
    # 2 key splits
    assert _attn_case(torch, f3c.F3C_F32, heads, hd, [512, 70], [2048, 1100], seed=hd, workspace=True) < 1e-4


@pytest.mark.parametrize("hd,heads", [(32, 4), (64, 2)])
@pytest.mark.parametrize("q_lens,k_lens", [([512], [512]), ([3, 256, 130], [64, 64, 64]), ([100], [1])])
@pytest.mark.parametrize("prescaled", [False, True])
def test_attention_f32(torch, hd, heads, q_lens, k_lens, prescaled):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_F32, heads, hd, q_lens, k_lens, seed=hd + len(q_lens),
                      prescaled=prescaled) < 1e-4


def test_attention_f32_eight_waves_sampled(torch):
    # enough query tiles (21 x 8 heads) for the 8-wave workgroup
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_F32, 8, 64, [5200], [5200], seed=11, sample_queries=64) < 1e-4


def test_attention_bf16_hd32(torch):
    from paper_2511_22533_amd import f3c
    assert _attn_case(torch, f3c.F3C_BF16, 4, 32, [300, 64], [300, 64], seed=9) < 2e-2


@pytest.mark.parametrize("dt_name,d", [("f32", 128), ("bf16", 1024), ("bf16", 2048)])
def test_ln_mod(torch, dt_name, d):
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(d)
    rows = 333
    h = (3 * rng.standard_normal((rows, d)) + 1).astype(np.float32)
    shift = rng.standard_normal(d).astype(np.float32)
    scale = rng.standard_normal(d).astype(np.float32)
    dt = f3c.F3C_BF16 if dt_name == "bf16" else f3c.F3C_F32
    tdt = torch.bfloat16 if dt_name == "bf16" else torch.float32
    for mod in (True, False):
        out = torch.empty((rows, d), dtype=tdt, device="cuda")
        say("ln", dt_name, d, mod)
        f3c.op_ln_mod(dt, to_dev(h), out, to_dev(shift) if mod else None, to_dev(scale) if mod else None)
        torch.cuda.synchronize()
        want = dit.layer_norm(h.astype(np.float64))
        if mod:
            want = want * (1 + scale) + shift
        tol = 8e-3 if dt_name == "bf16" else 1e-5
        assert max_rel(out.float().cpu().numpy(), want) < tol


@pytest.mark.parametrize("cfg", [synth.TINY, synth.ModelConfig(grid=4, width=1024, depth=3, heads=16, cond_tokens=8,
                                                              cond_width=64, dtype="bf16")])
def test_modulation(torch, cfg):
    from paper_2511_22533_amd import f3c
    W = synth.make_weights(cfg, seed=2, scale=0.05)
    m = f3c.Model(cfg).load(W)
    om = dit.Model(cfg, W)
    for t in (1.0, 0.73, 0.111, 0.0):
        say("modulation", cfg.dtype, t)
        got = m.modulation(t).cpu().numpy()
        torch.cuda.synchronize()
        tol = 1e-4 if cfg.dtype == "f32" else 5e-3
        assert max_rel(got, om.modulation(t)) < tol


_EMBED_CFGS = [synth.TINY, synth.ModelConfig(grid=16, width=1024, depth=1, heads=16, cond_tokens=8, cond_width=64,
                                             dtype="bf16")]


@pytest.mark.parametrize("cfg", _EMBED_CFGS, ids=["tiny_f32", "g16_w1024_bf16"])
def test_embed_gather(torch, cfg):
    from paper_2511_22533_amd import f3c
    W = synth.make_weights(cfg, seed=4, scale=0.05)
    m = f3c.Model(cfg).load(W)
    om = dit.Model(cfg, W)
    N, d = cfg.grid ** 3, cfg.width
    rng = np.random.default_rng(17)
    B = 3
    x = rng.standard_normal((B, N, 8)).astype(np.float32)
    # ragged active sets: a large one, a tiny one, an empty one (ascending indices)
    sets = [np.sort(rng.choice(N, N - N // 5, replace=False)), np.array([0, N - 1]), np.zeros(0, np.int64)]
    off = np.concatenate([[0], np.cumsum([len(a) for a in sets])]).astype(int)
    idx = np.concatenate(sets).astype(np.int32)
    h = torch.full((off[-1], d), float("nan"), dtype=torch.float32, device="cuda")
    say("embed", cfg.dtype, off.tolist())
    f3c.op_embed(m, to_dev(x), off.tolist(), h, idx_active=to_dev(idx))
    torch.cuda.synchronize()
    got = h.cpu().numpy()
    for b in range(B):
        if len(sets[b]):
            want = om.embed(x[b][sets[b]], sets[b])
            assert max_rel(got[off[b]:off[b + 1]], want) < 1e-5
    # identity gather (full step): every token of each sample, no index list
    h2 = torch.empty((2 * N, d), dtype=torch.float32, device="cuda")
    say("embed identity", cfg.dtype)
    f3c.op_embed(m, to_dev(x[:2]), [0, N, 2 * N], h2)
    torch.cuda.synchronize()
    got2 = h2.cpu().numpy()
    for b in range(2):
        assert max_rel(got2[b * N:(b + 1) * N], om.embed(x[b], np.arange(N))) < 1e-5


@pytest.mark.parametrize("cfg", _EMBED_CFGS, ids=["tiny_f32", "g16_w1024_bf16"])
@pytest.mark.parametrize("rows", [1, 333])
def test_final_projection(torch, cfg, rows):
    from paper_2511_22533_amd import f3c
    W = synth.make_weights(cfg, seed=5, scale=0.05)
    m = f3c.Model(cfg).load(W)
    rng = np.random.default_rng(rows)
    h = (2 * rng.standard_normal((rows, cfg.width)) + 0.5).astype(np.float32)
    v = torch.full((rows, 8), float("nan"), dtype=torch.float32, device="cuda")
    say("final", cfg.dtype, rows)
    f3c.op_final(m, to_dev(h), v)
    torch.cuda.synchronize()
    want = dit.linear(dit.layer_norm(h.astype(np.float64)), W["out_w"], W["out_b"])
    assert max_rel(v.cpu().numpy(), want) < 1e-5


@pytest.mark.parametrize("N,n_cache", [(512, [0, 100, 512]), (4096, [3276, 0]), (32768, [22937])])
def test_euler_merge_rotate_bit_exact(torch, N, n_cache):
    """Merge + Euler + rotation equal the oracle's step bit for bit, with the
    oracle's own selection and the same fresh velocities for the active rows."""
    from oracle import sampler
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(N)
    B = len(n_cache)
    x = rng.standard_normal((B, N, 8)).astype(np.float32)
    vc = rng.standard_normal((B, N, 8)).astype(np.float32)
    vp = rng.standard_normal((B, N, 8)).astype(np.float32)
    sel = oracle_selection(vc, vp, n_cache)
    act = [a for _, a in sel]
    off = np.concatenate([[0], np.cumsum([len(a) for a in act])]).astype(int)
    v_act = rng.standard_normal((max(off[-1], 1), 8)).astype(np.float32)
    pos = np.full((B, N), -1, np.int32)
    for b in range(B):
        pos[b, act[b]] = off[b] + np.arange(len(act[b]))
    t, t_next = 0.7310585786, 0.6224593312
    st = sampler.State(x.copy(), vc.copy(), vp.copy())
    sampler.step(st, lambda b, xa, idx, tt: v_act[off[b]:off[b + 1]], t, t_next, n_cache)
    d_x, d_vn = to_dev(x), torch.full((B, N, 8), float("nan"), dtype=torch.float32, device="cuda")
    say("euler", N, n_cache)
    f3c.op_euler(d_x, to_dev(vc), to_dev(v_act), to_dev(pos), off.tolist(), t, t_next, d_vn)
    torch.cuda.synchronize()
    assert np.array_equal(d_x.cpu().numpy(), st.x)
    assert np.array_equal(d_vn.cpu().numpy(), st.v_cache)


def test_euler_all_active_without_pos(torch):
    from oracle import sampler
    from paper_2511_22533_amd import f3c
    rng = np.random.default_rng(3)
    B, N = 2, 512
    x = rng.standard_normal((B, N, 8)).astype(np.float32)
    vc = rng.standard_normal((B, N, 8)).astype(np.float32)
    v_act = rng.standard_normal((B * N, 8)).astype(np.float32)
    st = sampler.State(x.copy(), vc.copy(), vc.copy())
    sampler.step(st, lambda b, xa, idx, tt: v_act[b * N:(b + 1) * N], 1.0, 0.96, [0, 0])
    d_x, d_vn = to_dev(x), torch.empty((B, N, 8), dtype=torch.float32, device="cuda")
    say("euler identity")
    f3c.op_euler(d_x, to_dev(vc), to_dev(v_act), None, [0, N, 2 * N], 1.0, 0.96, d_vn)
    torch.cuda.synchronize()
    assert np.array_equal(d_x.cpu().numpy(), st.x)
    assert np.array_equal(d_vn.cpu().numpy(), st.v_cache)


def _occupancy_logits(B, n, seed):
    """Decoder-like logits: a smooth blob (occupied core) plus noise, with the
    comparison's edge values planted: 0, -0, NaN, +-inf, the smallest subnormal."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, n)).astype(np.float32)
    x += np.linspace(1.5, -1.5, n, dtype=np.float32)[None, :]
    special = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, 1e-45, -1e-45], np.float32)
    for b in range(B):
        at = rng.choice(n, size=min(n, len(special)), replace=False)
        x[b, at] = special[:len(at)]
    return x


@pytest.mark.parametrize("B,n", [(1, 1), (2, 31), (1, 32), (3, 33), (3, 1028), (2, 8191), (1, 8192), (2, 8193), (2, 8196),
                                 (2, 64 ** 3), (1, 64 ** 3 + 5)])
def test_pack_occupancy_bit_exact(torch, B, n):
    """Packed occupancy equals the oracle's packing word for word, tail bits zero."""
    from oracle import occupancy
    from paper_2511_22533_amd import f3c
    say(f"pack_occupancy B={B} n={n}")
    x = _occupancy_logits(B, n, seed=B * 1000 + n)
    n_words = (n + 31) // 32
    bits = torch.full((B, n_words), -1, dtype=torch.int32, device="cuda")
    f3c.op_pack_occupancy(to_dev(x), bits)
    torch.cuda.synchronize()
    got = bits.cpu().numpy().view(np.uint32)
    for b in range(B):
        assert np.array_equal(got[b], occupancy.pack(occupancy.occupancy(x[b]))), f"sample {b}"


@pytest.mark.parametrize("B,n,offset", [(1, 1, 0), (3, 33, 0), (2, 64 ** 3, 0), (2, 64 ** 3, 1),
                                        (1, 64 ** 3 + 5, 0), (4, 1000, 3)])
def test_dynamic_voxels_exact(torch, B, n, offset):
    """Eq. (1) count per sample equals the oracle's, for grids that differ in a
    few voxels (late steps) and in many (early steps); offset shifts the rows
    off 16-byte alignment so the word-at-a-time path runs too."""
    from oracle import occupancy
    from paper_2511_22533_amd import f3c
    say(f"dynamic_voxels B={B} n={n} offset={offset}")
    rng = np.random.default_rng(n + offset)
    prev = _occupancy_logits(B, n, seed=7 + n)
    nxt = prev.copy()
    for b in range(B):
        flips = rng.choice(n, size=max(1, n // (10 ** (b + 1))), replace=False)
        nxt[b, flips] = -nxt[b, flips]
    n_words = (n + 31) // 32
    packed = torch.zeros(2, B * n_words + offset, dtype=torch.int32, device="cuda")
    a = packed[0, offset:].view(B, n_words)
    p = packed[1, offset:].view(B, n_words)
    f3c.op_pack_occupancy(to_dev(nxt), a)
    f3c.op_pack_occupancy(to_dev(prev), p)
    counts = torch.full((B,), -1, dtype=torch.int64, device="cuda")
    f3c.op_dynamic_voxels(a, p, counts)
    torch.cuda.synchronize()
    got = counts.cpu().numpy()
    for b in range(B):
        want = occupancy.dynamic_voxels(occupancy.occupancy(nxt[b]), occupancy.occupancy(prev[b]))
        assert got[b] == want, f"sample {b}"


def test_dynamic_voxels_all_bits(torch):
    """Complementary grids: every voxel counts, including full 32-bit words."""
    from paper_2511_22533_amd import f3c
    n_words = 4096 + 3
    a = torch.zeros((2, n_words), dtype=torch.int32, device="cuda")
    b = torch.full((2, n_words), -1, dtype=torch.int32, device="cuda")
    b[1] = 0
    counts = torch.full((2,), -1, dtype=torch.int64, device="cuda")
    f3c.op_dynamic_voxels(a, b, counts)
    torch.cuda.synchronize()
    assert counts.cpu().tolist() == [32 * n_words, 0]


def test_sigma_calibration_drives_schedule(torch):
    """sigma of the predictive schedule (Sec. 3.2) from two decoded 64^3 grids
    at the anchor step and the step before it: count on the GPU, then the host
    plan for a 16^3 latent (64 output voxels per latent token), equal to the
    oracle's plan from the oracle's count."""
    from oracle import occupancy
    from oracle import schedule as osched
    from paper_2511_22533_amd import f3c
    G = 64
    z, y, x = np.meshgrid(*(np.arange(G, dtype=np.float32),) * 3, indexing="ij")
    r = np.sqrt((z - 31.5) ** 2 + (y - 30.0) ** 2 + (x - 33.0) ** 2)
    rng = np.random.default_rng(11)
    prev = (20.0 - r + 0.8 * rng.standard_normal(r.shape)).astype(np.float32).reshape(1, -1)
    nxt = (20.6 - r + 0.8 * rng.standard_normal(r.shape)).astype(np.float32).reshape(1, -1)
    words = torch.zeros((2, 1, G ** 3 // 32), dtype=torch.int32, device="cuda")
    f3c.op_pack_occupancy(to_dev(nxt), words[0])
    f3c.op_pack_occupancy(to_dev(prev), words[1])
    counts = torch.zeros((1,), dtype=torch.int64, device="cuda")
    f3c.op_dynamic_voxels(words[0], words[1], counts)
    torch.cuda.synchronize()
    sigma = int(counts.item())
    want_sigma = occupancy.dynamic_voxels(occupancy.occupancy(nxt), occupancy.occupancy(prev))
    assert sigma == want_sigma and sigma > 0
    for tau in (0, 3):
        got = f3c.schedule_plan(25, 16 ** 3, float(sigma), gamma_up=64.0, tau=tau)
        assert got.tolist() == osched.plan(25, 16 ** 3, float(want_sigma), gamma_up=64.0, tau=tau)
