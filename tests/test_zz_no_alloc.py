"""The no-allocation selection entry (f3c_op_select_noalloc) against the
workspace entry (f3c_op_select), through the C ABI: bit-identical indices,
positions and scores on two calls in a row, the second with a smaller
input (the static scratch keeps the first call's contents), and the size
limit rejected before any work."""
import numpy as np
import pytest

from helpers import say, to_dev

pytestmark = pytest.mark.gpu


def _inputs(B, N, seed):
    rng = np.random.default_rng(seed)
    vc = rng.standard_normal((B, N, 8)).astype(np.float32)
    vp = (vc + 0.1 * rng.standard_normal((B, N, 8))).astype(np.float32)
    q = [int(x) for x in rng.integers(0, N + 1, size=B)]
    return vc, vp, q


def _both(torch, f3c, vc, vp, q, omega=0.7):
    B, N = vc.shape[:2]
    d_vc, d_vp = to_dev(vc), to_dev(vp)
    total = max(1, sum(N - c for c in q))
    out = []
    for fn in ("ws", "noalloc"):
        idx = torch.full((total,), -7, dtype=torch.int32, device="cuda")
        pos = torch.full((B, N), -7, dtype=torch.int32, device="cuda")
        score = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
        if fn == "ws":
            f3c.op_select(d_vc, d_vp, omega, q, idx, pos, score)
        else:
            f3c.op_select_noalloc(d_vc, d_vp, omega, q, idx, pos, score)
        torch.cuda.synchronize()
        out.append((idx.cpu().numpy(), pos.cpu().numpy(), score.cpu().numpy().view(np.uint32)))
    return out


def test_noalloc_select_matches_workspace_entry():
    import torch
    from paper_2511_22533_amd import f3c
    f3c.lib()
    for B, N, seed in ((16, 32768, 1), (3, 3000, 2)):     # the second call is smaller
        say("noalloc select", B, N)
        vc, vp, q = _inputs(B, N, seed)
        (i0, p0, s0), (i1, p1, s1) = _both(torch, f3c, vc, vp, q)
        assert np.array_equal(i0, i1) and np.array_equal(p0, p1)
        for b in range(B):
            if q[b] > 0:
                assert np.array_equal(s0[b], s1[b])
    # beyond the static scratch: rejected before any device work
    big = torch.zeros((17, 32768, 8), dtype=torch.float32, device="cuda")
    idx = torch.zeros((17 * 32768,), dtype=torch.int32, device="cuda")
    pos = torch.zeros((17, 32768), dtype=torch.int32, device="cuda")
    with pytest.raises(f3c.F3CError) as e:
        f3c.op_select_noalloc(big, big, 0.7, [1] * 17, idx, pos)
    assert e.value.code == f3c.F3C_EINVAL and "static scratch" in str(e.value)
