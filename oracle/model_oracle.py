"""CPU oracle for the whole-model prefill timing study (§4.1, §4.3, §5.3).

TEST INFRASTRUCTURE ONLY.  Only the test suite may import this module; the
product path never imports, calls or links it, and it imports nothing from
the product path.

The paper times time-to-first-token of a Qwen3-0.6B decoder stack (28 layers,
16 query heads, 8 kv-heads, head dimension 128, §4.1) with its attention
layers on the dense causal path, with eight middle layers on the BF1 route,
and with every layer on the BF1 route (§4.3, §5.3).  This module is that
stack written out plainly in float64: per layer an RMSNorm, the Q/K/V
projections, an RMSNorm of every query and key head, the rotary position
embedding, attention (the BF1 route of Eq. 1 or dense causal attention, both
from bf1_oracle), the output projection added to the residual stream, an
RMSNorm and a SwiGLU MLP added to the residual stream; then a final RMSNorm
and the logits of the last position through the tied embedding matrix.  The
layer structure beyond the paper's geometry follows the public Qwen3
architecture; its weights are not available, so callers pass seeded random
ones.
"""

import math

import numpy as np

from oracle import bf1_oracle as orc

__all__ = ["rms_norm", "rope", "silu", "prefill_last_logits_fp64"]


def rms_norm(x, w, eps):
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def rope(x, theta):
    """Rotary position embedding of x [n, heads, d] at positions 0..n-1:
    the pair (x_i, x_{i+d/2}) of position p turns by p * theta^(-2i/d)."""
    n, _, d = x.shape
    half = d // 2
    inv = theta ** (-np.arange(0, d, 2, dtype=np.float64) / d)
    ang = np.arange(n, dtype=np.float64)[:, None] * inv[None, :]
    cos = np.concatenate([np.cos(ang), np.cos(ang)], axis=-1)[:, None, :]
    sin = np.concatenate([np.sin(ang), np.sin(ang)], axis=-1)[:, None, :]
    rotated = np.concatenate([-x[..., half:], x[..., :half]], axis=-1)
    return x * cos + rotated * sin


def silu(x):
    return x / (1.0 + np.exp(-x))


def prefill_last_logits_fp64(ids, weights, cfg, bf1_layers, b=64, L=2):
    """Logits [vocab] of the last position after a prefill of token ids.

    weights: float arrays named as by the input generator ("embed",
    "final_norm", "<layer>.<name>", projections stored [in, out]);
    bf1_layers: indices of the layers whose attention takes the BF1 route
    (block width b, local width L); the others are dense causal.
    """
    w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
    ids = np.asarray(ids)
    n = len(ids)
    H, Hkv, d = cfg.heads, cfg.kv_heads, cfg.head_dim
    h = w["embed"][ids]
    for l in range(cfg.layers):
        p = f"{l}."
        a = rms_norm(h, w[p + "in_norm"], cfg.eps)
        q = rms_norm((a @ w[p + "wq"]).reshape(n, H, d), w[p + "q_norm"], cfg.eps)
        k = rms_norm((a @ w[p + "wk"]).reshape(n, Hkv, d), w[p + "k_norm"], cfg.eps)
        v = (a @ w[p + "wv"]).reshape(n, Hkv, d)
        q, k = rope(q, cfg.rope_theta), rope(k, cfg.rope_theta)
        Q, K, V = (t.transpose(1, 0, 2)[None] for t in (q, k, v))
        if l in bf1_layers:
            O, _ = orc.attn_gathered_fp64(Q, K, V, b, L)
        else:
            O, _ = orc.dense_causal_fp64(Q, K, V)
        h = h + O[0].transpose(1, 0, 2).reshape(n, H * d) @ w[p + "wo"]
        a = rms_norm(h, w[p + "post_norm"], cfg.eps)
        h = h + (silu(a @ w[p + "wg"]) * (a @ w[p + "wu"])) @ w[p + "wd"]
    last = rms_norm(h[-1], w["final_norm"], cfg.eps)
    return last @ w["embed"].T
