"""Whole-model prefill of the paper's timing study (§4.3, §5.3) on one GPU.

A decoder stack of the evaluated geometry (Qwen3-0.6B: 28 layers, 16 query
heads, 8 kv-heads, head dimension 128, §4.1) whose attention layers run this
library's kernels: bf1_attn_fwd on the BF1 route for the chosen layers, the
in-house dense causal kernel (bf1_dense_causal_fwd) for the others.  The
projections, norms, rotary embedding and MLP around them are plain PyTorch
operators on the GPU (hipBLASLt GEMMs and eager elementwise kernels), as in
the paper's eager harness; the study measures the time to first token (the
last position's logits) with no, the middle eight, or all layers on the BF1
route.  The trained weights are not available: callers pass seeded random
weights of the published shapes (timing does not depend on their values).
"""

import torch

from . import attn_fwd, dense_causal_fwd

__all__ = ["middle_layers", "PrefillStack"]


def middle_layers(cfg, count=8):
    """Indices of the `count` central layers of the stack (the paper converts
    eight middle layers of 28, §4.4; here layers 10..17)."""
    start = (cfg.layers - count) // 2
    return set(range(start, start + count))


class PrefillStack:
    """cfg: a synth.ModelConfig; weights: the generator's bf16 tensors
    (projections stored [in, out]); B, L: block width and local width of the
    BF1 layers."""

    def __init__(self, cfg, weights, device="cuda", B=64, L=2):
        self.cfg, self.B, self.L = cfg, B, L
        self.w = {k: v.to(device).contiguous() for k, v in weights.items()}
        self.device = device
        self._rope_n = -1

    def _rope_tables(self, n):
        if n != self._rope_n:
            d = self.cfg.head_dim
            inv = self.cfg.rope_theta ** (-torch.arange(0, d, 2, dtype=torch.float64, device=self.device) / d)
            ang = torch.arange(n, dtype=torch.float64, device=self.device)[:, None] * inv[None, :]
            self._cos = torch.cat([ang.cos(), ang.cos()], dim=-1).float()[:, None, :]
            self._sin = torch.cat([ang.sin(), ang.sin()], dim=-1).float()[:, None, :]
            self._rope_n = n
        return self._cos, self._sin

    def _rms(self, x, w):
        xf = x.float()
        y = xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + self.cfg.eps)
        return (y * w.float()).to(torch.bfloat16)

    def _rope(self, x, cos, sin):
        xf = x.float()
        half = xf.shape[-1] // 2
        rot = torch.cat([-xf[..., half:], xf[..., :half]], dim=-1)
        return (xf * cos + rot * sin).to(torch.bfloat16)

    def last_logits(self, ids, bf1_layers, dense_attention=None):
        """Logits (float32, [vocab]) of the last position after the prefill of
        token ids (int64 device tensor [n]).  dense_attention, if given,
        replaces the in-house dense kernel for the non-BF1 layers: a callable
        (Q, K, V) -> O on [1, heads, n, d] bf16 tensors (a comparator)."""
        cfg, w = self.cfg, self.w
        n = ids.shape[0]
        H, Hkv, d = cfg.heads, cfg.kv_heads, cfg.head_dim
        cos, sin = self._rope_tables(n)
        h = w["embed"][ids]
        for l in range(cfg.layers):
            p = f"{l}."
            a = self._rms(h, w[p + "in_norm"])
            q = self._rms((a @ w[p + "wq"]).view(n, H, d), w[p + "q_norm"])
            k = self._rms((a @ w[p + "wk"]).view(n, Hkv, d), w[p + "k_norm"])
            v = (a @ w[p + "wv"]).view(n, Hkv, d)
            q, k = self._rope(q, cos, sin), self._rope(k, cos, sin)
            Q = q.transpose(0, 1).contiguous().unsqueeze(0)
            K = k.transpose(0, 1).contiguous().unsqueeze(0)
            V = v.transpose(0, 1).contiguous().unsqueeze(0)
            if l in bf1_layers:
                O, _ = attn_fwd(Q, K, V, self.B, self.L, want_lse=False)
            elif dense_attention is not None:
                O = dense_attention(Q, K, V)
            else:
                O, _ = dense_causal_fwd(Q, K, V, want_lse=False)
            h = h + O[0].transpose(0, 1).reshape(n, H * d) @ w[p + "wo"]
            a = self._rms(h, w[p + "post_norm"])
            h = h + (torch.nn.functional.silu(a @ w[p + "wg"]) * (a @ w[p + "wu"])) @ w[p + "wd"]
        last = self._rms(h[-1:], w["final_norm"])
        return (last @ w["embed"].t()).float()[0]
