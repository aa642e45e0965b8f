"""Sparse-structure flow transformer on a token subset, float64 (Sec. 3.2; Sec. 4.2).

The paper accelerates the TRELLIS sparse-structure flow transformer G_S and
states, in its FLOPs model (supplement, FLOPs Calculation), what each block
contains: a per-sample 6*D modulation, three LayerNorms, self-attention with a
QKV and an output projection, cross-attention whose queries come from the
tokens and whose keys/values come from the D_cond-wide condition tokens, and a
ratio-4 MLP. The index-based selection of Sec. 4.2 runs the transformer, self
attention included, on the active tokens only; the grid's positional
information travels with each token.

Readings where the paper is silent (it prints no architecture details):
* LayerNorm without affine parameters, eps 1e-6;
* block: u = LN(h)(1+scale1)+shift1, h += gate1 * SA(u);
         h += CA(LN(h), cond);
         u = LN(h)(1+scale2)+shift2, h += gate2 * MLP(u);
  with (shift1, scale1, gate1, shift2, scale2, gate2) = split6(W_mod SiLU(temb) + b_mod);
* MLP: GELU (tanh form) between two biased linears;
* timestep embedding: [cos(1000 t f_j), sin(1000 t f_j)], f_j = 10000^(-j/128),
  j < 128, followed by Linear -> SiLU -> Linear;
* input: h = x W_in^T + b_in + P[n] with a learned absolute position table P
  gathered by original token index n; output: v = LN(h) W_out^T + b_out;
* attention: per head softmax(Q K^T / sqrt(d_head)) V, no QK normalisation.

All linear weights are stored [out][in] and applied as y = x W^T + b.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict

import numpy as np
from threadpoolctl import threadpool_limits

F64 = np.float64
LN_EPS = 1e-6
QUERY_CHUNK = 2048


def _matmul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Every dense contraction of the transformer goes through here (counted by the FLOPs pin)."""
    return a @ b


def linear(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    return _matmul(x, w.T) + b


def layer_norm(x: np.ndarray) -> np.ndarray:
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    return xc / np.sqrt(var + LN_EPS)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x * x * x)))


def timestep_features(t: float, n_freq: int = 256) -> np.ndarray:
    half = n_freq // 2
    freqs = np.power(10000.0, -np.arange(half, dtype=F64) / half)
    arg = 1000.0 * float(t) * freqs
    return np.concatenate([np.cos(arg), np.sin(arg)])


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """Multi-head softmax attention: q [n][d], k/v [m][d] -> [n][d] (heads split along d).

    Per head: S = Q K^T / sqrt(d_head); P = exp(S - rowmax(S)) / rowsum(...);
    O = P V, with the query rows taken QUERY_CHUNK at a time (the scores of
    one chunk are materialised in full). The heads are independent, so they
    run concurrently on threads, each with a one-thread BLAS; every head's
    arithmetic is the same sequence of whole-array operations as in a serial
    loop (done in place on the chunk's score array), so the result does not
    depend on the thread count."""
    n, d = q.shape
    hd = d // heads
    out = np.empty((n, d), dtype=F64)
    scale = 1.0 / math.sqrt(hd)

    def one_head(h: int) -> None:
        sl = slice(h * hd, (h + 1) * hd)
        kh_t = np.ascontiguousarray(k[:, sl].T)
        vh = v[:, sl]
        for q0 in range(0, n, QUERY_CHUNK):
            qh = q[q0:q0 + QUERY_CHUNK, sl]
            s = _matmul(qh, kh_t)
            np.multiply(s, scale, out=s)
            np.subtract(s, s.max(axis=1, keepdims=True), out=s)
            np.exp(s, out=s)
            np.divide(s, s.sum(axis=1, keepdims=True), out=s)
            out[q0:q0 + QUERY_CHUNK, sl] = _matmul(s, vh)

    workers = max(1, min(heads, len(os.sched_getaffinity(0))))
    with threadpool_limits(limits=1, user_api="blas"), ThreadPoolExecutor(workers) as ex:
        list(ex.map(one_head, range(heads)))
    return out


class Model:
    """Holds float64 copies of the (already rounded) weights and the shapes."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.w = {k: np.asarray(v, dtype=F64) for k, v in weights.items()}

    def modulation(self, t: float) -> np.ndarray:
        """Per-block (shift1, scale1, gate1, shift2, scale2, gate2), shape [L][6][d]."""
        w, d = self.w, self.cfg.width
        phi = timestep_features(t)
        temb = linear(silu(linear(phi, w["t1_w"], w["t1_b"])), w["t2_w"], w["t2_b"])
        a = silu(temb)
        mods = [linear(a, w[f"blk{l}.mod_w"], w[f"blk{l}.mod_b"]).reshape(6, d)
                for l in range(self.cfg.depth)]
        return np.stack(mods)

    def cond_kv(self, cond: np.ndarray, l: int):
        """Cross-attention keys/values of block l from condition tokens [Nc][dc]."""
        kv = linear(np.asarray(cond, dtype=F64), self.w[f"blk{l}.kv_w"], self.w[f"blk{l}.kv_b"])
        d = self.cfg.width
        return kv[:, :d], kv[:, d:]

    def embed(self, x_active: np.ndarray, idx: np.ndarray) -> np.ndarray:
        w = self.w
        return linear(np.asarray(x_active, dtype=F64), w["in_w"], w["in_b"]) + w["pos"][idx]

    def self_attention_sublayer(self, l: int, h: np.ndarray, mod_l: np.ndarray) -> np.ndarray:
        """SA(LN(h)(1+scale1)+shift1) after its output projection, before the gate g1."""
        w, heads, d = self.w, self.cfg.heads, self.cfg.width
        p = f"blk{l}."
        sh1, sc1 = mod_l[0], mod_l[1]
        u = layer_norm(h) * (1.0 + sc1) + sh1
        qkv = linear(u, w[p + "qkv_w"], w[p + "qkv_b"])
        sa = attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], heads)
        return linear(sa, w[p + "o_w"], w[p + "o_b"])

    def cross_attention_sublayer(self, l: int, h: np.ndarray, cond_k: np.ndarray,
                                 cond_v: np.ndarray) -> np.ndarray:
        """CA(LN(h), cond) after its output projection (no gate)."""
        w, heads = self.w, self.cfg.heads
        p = f"blk{l}."
        q = linear(layer_norm(h), w[p + "q_w"], w[p + "q_b"])
        ca = attention(q, cond_k, cond_v, heads)
        return linear(ca, w[p + "co_w"], w[p + "co_b"])

    def mlp_sublayer(self, l: int, h: np.ndarray, mod_l: np.ndarray) -> np.ndarray:
        """MLP(LN(h)(1+scale2)+shift2) after the second linear, before the gate g2."""
        w = self.w
        p = f"blk{l}."
        sh2, sc2 = mod_l[3], mod_l[4]
        u = layer_norm(h) * (1.0 + sc2) + sh2
        return linear(gelu_tanh(linear(u, w[p + "fc1_w"], w[p + "fc1_b"])), w[p + "fc2_w"], w[p + "fc2_b"])

    def block(self, l: int, h: np.ndarray, mod_l: np.ndarray, cond_k: np.ndarray,
              cond_v: np.ndarray, trace: dict | None = None) -> np.ndarray:
        g1, g2 = mod_l[2], mod_l[5]
        sa_out = self.self_attention_sublayer(l, h, mod_l)
        h = h + g1 * sa_out
        ca_out = self.cross_attention_sublayer(l, h, cond_k, cond_v)
        h = h + ca_out
        mlp = self.mlp_sublayer(l, h, mod_l)
        h = h + g2 * mlp
        if trace is not None:
            trace[l] = {"sa_out": sa_out, "ca_out": ca_out, "mlp_out": mlp, "h": h.copy()}
        return h

    def forward(self, x_active: np.ndarray, idx: np.ndarray, t: float, cond: np.ndarray,
                trace: dict | None = None) -> np.ndarray:
        """Velocity of the active tokens x_active [n][C] at original indices idx, float64 [n][C]."""
        mod = self.modulation(t)
        h = self.embed(x_active, idx)
        if trace is not None:
            trace["embed"] = h.copy()
            trace["mod"] = mod
        for l in range(self.cfg.depth):
            ck, cv = self.cond_kv(cond, l)
            h = self.block(l, h, mod[l], ck, cv, trace)
        return linear(layer_norm(h), self.w["out_w"], self.w["out_b"])
