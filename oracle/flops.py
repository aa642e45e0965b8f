"""FLOPs model of the supplement (FLOPs Calculation), per flow-transformer block.

Terms as itemised there, with B samples, N_tok tokens per sample, model width
D, H heads, N_cond condition tokens of width D_cond and MLP width 4 D. Under the
cached sampler N_tok is the active-token count.
"""
from __future__ import annotations


def block_terms(B, n_tok, d, heads, n_cond, d_cond, d_mlp=None):
    d_mlp = 4 * d if d_mlp is None else d_mlp
    hd = d / heads
    return {
        "mod": 5 * B * d + 2 * B * d * (6 * d),
        "ln": 3 * (7 * B * n_tok * d),
        "sa_qkv": 2 * B * n_tok * d * (3 * d),
        "sa_qk": 2 * B * heads * n_tok ** 2 * hd,
        "sa_softmax": 5 * B * heads * n_tok ** 2,
        "sa_av": 2 * B * heads * n_tok ** 2 * hd,
        "sa_out": 2 * B * n_tok * d * d,
        "ca_q": 2 * B * n_tok * d * d,
        "ca_kv": 2 * B * n_cond * d_cond * (2 * d),
        "ca_qk": 2 * B * heads * n_tok * n_cond * hd,
        "ca_softmax": 5 * B * heads * n_tok * n_cond,
        "ca_av": 2 * B * heads * n_tok * n_cond * hd,
        "ca_out": 2 * B * n_tok * d * d,
        "fc1": 2 * B * n_tok * d * d_mlp,
        "act": 5 * B * n_tok * d_mlp,
        "fc2": 2 * B * n_tok * d_mlp * d,
    }


def block_flops(B, n_tok, d, heads, n_cond, d_cond, d_mlp=None) -> float:
    return float(sum(block_terms(B, n_tok, d, heads, n_cond, d_cond, d_mlp).values()))


def forward_flops(cfg, n_tok: int, B: int = 1) -> float:
    """All blocks of one forward over n_tok tokens per sample."""
    return cfg.depth * block_flops(B, n_tok, cfg.width, cfg.heads, cfg.cond_tokens, cfg.cond_width,
                                   cfg.mlp_width)
