"""Pins for the oracle's flow transformer (float64).

* attention equals a scalar-loop softmax on tiny inputs;
* the forward equals an independent scalar-loop transformer on a tiny model;
* permutation equivariance over the active set (positions travel with tokens);
* cached tokens never influence active ones (self-attention on the active
  subset only, Sec. 4.2);
* with zero modulation and zero cross-attention output every block is the
  identity, leaving a closed form for embed -> LayerNorm -> output;
* closed forms of LayerNorm, GELU (tanh form) and the timestep features.
"""
import math

import numpy as np

from oracle import dit
from paper_2511_22533_amd import synth


def _tiny_cfg(**kw):
    base = dict(grid=2, width=8, depth=1, heads=2, cond_tokens=3, cond_width=6, dtype="f32")
    base.update(kw)
    return synth.ModelConfig(**base)


def test_layer_norm_moments():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((50, 64)) * 3 + 7
    y = dit.layer_norm(x)
    assert np.allclose(y.mean(-1), 0, atol=1e-12)
    var = x.var(-1)
    assert np.allclose((y * y).mean(-1), var / (var + dit.LN_EPS), atol=1e-12)


def test_gelu_tanh_identities():
    x = np.linspace(-6, 6, 101)
    g = dit.gelu_tanh(x)
    assert dit.gelu_tanh(np.array([0.0]))[0] == 0.0
    assert np.allclose(g - dit.gelu_tanh(-x), x, atol=1e-14)   # tanh is odd
    assert abs(dit.gelu_tanh(np.array([30.0]))[0] - 30.0) < 1e-12


def test_gelu_tanh_approximates_exact_gelu():
    # The tanh form approximates GELU(x) = x * Phi(x), with Phi the standard
    # normal CDF written through math.erf, to within 4.8e-4 on [-8, 8]. A bound
    # of 5e-4 rejects the plausible slips: a cubic coefficient of 0.04 or 0.05
    # (2.9e-3, 3.0e-3), a dropped cubic term (3.4e-2), sqrt(1/pi) for sqrt(2/pi)
    # (0.10), or the sigmoid form x * sigmoid(1.702 x) (2.0e-2).
    x = np.linspace(-8.0, 8.0, 16001)
    exact = np.array([v * 0.5 * (1.0 + math.erf(v / math.sqrt(2.0))) for v in x])
    err = np.max(np.abs(dit.gelu_tanh(x) - exact))
    assert err < 5e-4, err
    assert err > 4e-4, err      # the tanh form, not the exact one


def test_silu_closed_form():
    assert dit.silu(np.array([0.0]))[0] == 0.0
    assert np.isclose(dit.silu(np.array([1.0]))[0], 1.0 / (1.0 + math.exp(-1.0)))


def test_timestep_features_closed_forms():
    f0 = dit.timestep_features(0.0)
    assert f0.shape == (256,)
    assert np.all(f0[:128] == 1.0) and np.all(f0[128:] == 0.0)
    f = dit.timestep_features(0.37)
    assert np.allclose(f[:128] ** 2 + f[128:] ** 2, 1.0)
    assert np.isclose(f[0], math.cos(370.0)) and np.isclose(f[128], math.sin(370.0))
    assert np.isclose(f[127], math.cos(370.0 * 10000.0 ** (-127 / 128)))


def _attention_loops(q, k, v, heads):
    n, d = q.shape
    m = k.shape[0]
    hd = d // heads
    out = np.zeros((n, d))
    for h in range(heads):
        for i in range(n):
            logits = []
            for j in range(m):
                logits.append(sum(q[i, h * hd + e] * k[j, h * hd + e] for e in range(hd)) / math.sqrt(hd))
            mx = max(logits)
            ws = [math.exp(s - mx) for s in logits]
            tot = sum(ws)
            for e in range(hd):
                out[i, h * hd + e] = sum(ws[j] * v[j, h * hd + e] for j in range(m)) / tot
    return out


def test_attention_matches_scalar_loops():
    rng = np.random.default_rng(1)
    for n, m, d, heads in [(5, 7, 8, 2), (1, 1, 4, 1), (8, 3, 6, 3)]:
        q, k, v = (rng.standard_normal((r, d)) * 2 for r in (n, m, m))
        assert np.allclose(dit.attention(q, k, v, heads), _attention_loops(q, k, v, heads), atol=1e-12)


def _scalar_linear(x, w, b):
    return [sum(w[o][i] * x[i] for i in range(len(x))) + b[o] for o in range(len(b))]


def _scalar_ln(x):
    mu = sum(x) / len(x)
    var = sum((a - mu) ** 2 for a in x) / len(x)
    return [(a - mu) / math.sqrt(var + 1e-6) for a in x]


def _scalar_forward(cfg, W, x_act, idx, t, cond):
    """Independent per-scalar restatement of the block for tiny shapes."""
    d, H = cfg.width, cfg.heads
    Wl = {k: v.tolist() for k, v in W.items()}
    half = 128
    phi = [math.cos(1000 * t * 10000 ** (-j / half)) for j in range(half)] + \
          [math.sin(1000 * t * 10000 ** (-j / half)) for j in range(half)]
    silu = lambda a: a / (1 + math.exp(-a))
    temb = _scalar_linear([silu(a) for a in _scalar_linear(phi, Wl["t1_w"], Wl["t1_b"])], Wl["t2_w"], Wl["t2_b"])
    st = [silu(a) for a in temb]
    hs = []
    for r, n in enumerate(idx):
        e = _scalar_linear(list(x_act[r]), Wl["in_w"], Wl["in_b"])
        hs.append([e[o] + Wl["pos"][n][o] for o in range(d)])

    def mha(qs, ks, vs):
        hd = d // H
        outs = []
        for qi in qs:
            o = [0.0] * d
            for h in range(H):
                sl = range(h * hd, (h + 1) * hd)
                lg = [sum(qi[e] * kj[e] for e in sl) / math.sqrt(hd) for kj in ks]
                mx = max(lg)
                ws = [math.exp(a - mx) for a in lg]
                tot = sum(ws)
                for e in sl:
                    o[e] = sum(w_ * vj[e] for w_, vj in zip(ws, vs)) / tot
            outs.append(o)
        return outs

    gelu = lambda a: 0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3)))
    for l in range(cfg.depth):
        p = f"blk{l}."
        m = _scalar_linear(st, Wl[p + "mod_w"], Wl[p + "mod_b"])
        sh1, sc1, g1, sh2, sc2, g2 = (m[i * d:(i + 1) * d] for i in range(6))
        us = [[a * (1 + sc1[o]) + sh1[o] for o, a in enumerate(_scalar_ln(h))] for h in hs]
        qkv = [_scalar_linear(u, Wl[p + "qkv_w"], Wl[p + "qkv_b"]) for u in us]
        att = mha([r[:d] for r in qkv], [r[d:2 * d] for r in qkv], [r[2 * d:] for r in qkv])
        so = [_scalar_linear(a, Wl[p + "o_w"], Wl[p + "o_b"]) for a in att]
        hs = [[h[o] + g1[o] * s[o] for o in range(d)] for h, s in zip(hs, so)]
        qs = [_scalar_linear(_scalar_ln(h), Wl[p + "q_w"], Wl[p + "q_b"]) for h in hs]
        kv = [_scalar_linear(list(c), Wl[p + "kv_w"], Wl[p + "kv_b"]) for c in cond]
        ca = mha(qs, [r[:d] for r in kv], [r[d:] for r in kv])
        co = [_scalar_linear(a, Wl[p + "co_w"], Wl[p + "co_b"]) for a in ca]
        hs = [[h[o] + c[o] for o in range(d)] for h, c in zip(hs, co)]
        us = [[a * (1 + sc2[o]) + sh2[o] for o, a in enumerate(_scalar_ln(h))] for h in hs]
        f1 = [[gelu(a) for a in _scalar_linear(u, Wl[p + "fc1_w"], Wl[p + "fc1_b"])] for u in us]
        f2 = [_scalar_linear(f, Wl[p + "fc2_w"], Wl[p + "fc2_b"]) for f in f1]
        hs = [[h[o] + g2[o] * f[o] for o in range(d)] for h, f in zip(hs, f2)]
    return np.array([_scalar_linear(_scalar_ln(h), Wl["out_w"], Wl["out_b"]) for h in hs])


def test_forward_matches_scalar_transformer():
    cfg = _tiny_cfg(depth=2)
    W = synth.make_weights(cfg, seed=11, scale=0.3)    # large scale: every sublayer matters
    model = dit.Model(cfg, W)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((cfg.tokens, 8)).astype(np.float32)
    cond = rng.standard_normal((cfg.cond_tokens, cfg.cond_width)).astype(np.float32)
    idx = np.array([0, 2, 3, 6, 7])
    got = model.forward(x[idx], idx, 0.6, cond)
    want = _scalar_forward(cfg, W, x[idx].astype(np.float64), idx.tolist(), 0.6, cond.astype(np.float64))
    assert np.allclose(got, want, rtol=1e-10, atol=1e-12)


def test_forward_permutation_equivariant():
    cfg = _tiny_cfg(grid=3, width=16, heads=4, depth=2)
    W = synth.make_weights(cfg, seed=12, scale=0.3)
    model = dit.Model(cfg, W)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((cfg.tokens, 8)).astype(np.float32)
    cond = rng.standard_normal((cfg.cond_tokens, cfg.cond_width)).astype(np.float32)
    idx = np.array([1, 4, 5, 9, 13, 20, 26])
    perm = rng.permutation(len(idx))
    a = model.forward(x[idx], idx, 0.3, cond)
    b = model.forward(x[idx[perm]], idx[perm], 0.3, cond)
    assert np.allclose(a[perm], b, rtol=1e-12, atol=1e-13)


def test_cached_tokens_do_not_influence_active_tokens():
    cfg = _tiny_cfg(grid=3, width=16, heads=4)
    W = synth.make_weights(cfg, seed=13, scale=0.3)
    model = dit.Model(cfg, W)
    rng = np.random.default_rng(4)
    x = rng.standard_normal((cfg.tokens, 8)).astype(np.float32)
    cond = rng.standard_normal((cfg.cond_tokens, cfg.cond_width)).astype(np.float32)
    idx = np.array([0, 3, 8, 17])
    a = model.forward(x[idx], idx, 0.5, cond)
    x2 = x.copy()
    others = np.setdiff1d(np.arange(cfg.tokens), idx)
    x2[others] += 100.0
    b = model.forward(x2[idx], idx, 0.5, cond)
    assert np.array_equal(a, b)
    # while the full forward of an active token does depend on the others
    full_a = model.forward(x, np.arange(cfg.tokens), 0.5, cond)
    full_b = model.forward(x2, np.arange(cfg.tokens), 0.5, cond)
    assert not np.allclose(full_a[idx], full_b[idx])


def test_identity_blocks_reduce_to_closed_form():
    cfg = _tiny_cfg(grid=3, width=16, heads=4, depth=3)
    W = synth.make_weights(cfg, seed=14, scale=0.3)
    for l in range(cfg.depth):
        for k in ("mod_w", "mod_b", "co_w", "co_b"):
            W[f"blk{l}.{k}"] = np.zeros_like(W[f"blk{l}.{k}"])
    model = dit.Model(cfg, W)
    rng = np.random.default_rng(5)
    x = rng.standard_normal((cfg.tokens, 8))
    cond = rng.standard_normal((cfg.cond_tokens, cfg.cond_width))
    idx = np.arange(0, cfg.tokens, 2)
    got = model.forward(x[idx], idx, 0.8, cond)
    e = x[idx] @ W["in_w"].astype(np.float64).T + W["in_b"] + W["pos"][idx]
    mu = e.mean(1, keepdims=True)
    sd = np.sqrt(((e - mu) ** 2).mean(1, keepdims=True) + 1e-6)
    want = ((e - mu) / sd) @ W["out_w"].astype(np.float64).T + W["out_b"]
    assert np.allclose(got, want, rtol=1e-12, atol=1e-13)
