"""Seeded synthetic inputs for BF1 attention.

This module only draws random tensors.  It holds none of the attention
arithmetic, and it is the one module that both the HIP path's tests and the
CPU oracle's tests take their inputs from: the same bf16 bits go to the GPU
and (converted exactly to float64) to the oracle.

Recipe: a NumPy ``Generator(PCG64(seed))`` draws Q, then K, then V as float32
standard normals in [batch, heads, n, head_dim] order; each tensor is
rounded to bf16 (round-to-nearest-even) by PyTorch on the CPU.  The peaked
workload additionally multiplies K by a factor at a random 5% of the token
positions of each batch element (all kv-heads, all dims), in float32 before
the bf16 rounding, so that some softmax rows are dominated by a few keys.

The workloads follow the paper's evaluated attention geometry (Qwen3-0.6B:
16 query heads, 8 kv-heads, head dimension 128, block width 64 and two local
blocks, §3.1 and §4.1); the paper's model activations and corpus are not
available, so seeded normals of that exact shape stand in for them.
"""

from dataclasses import dataclass, field, replace

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "sweep", "make_qkv", "make_qkv_device", "to_f64", "DecodeWorkload",
           "DECODE_WORKLOADS", "decode_seq_lens", "make_decode_host", "page_cache",
           "make_decode_device", "ModelConfig", "QWEN3_06B", "make_model_weights", "make_tokens"]


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n: int
    Hq: int
    Hkv: int
    d: int
    b: int
    L: int
    seed: int
    peak_frac: float = 0.0  # fraction of token positions whose K is scaled
    peak_mul: float = 3.0
    note: str = field(default="", compare=False)

    def with_(self, **kw):
        return replace(self, **kw)


# The named workloads: a tiny case, the Qwen3-0.6B layer geometry at 4K and
# at 32K (the headline point), and a batched case with a partial final block
# (30001 = 468 * 64 + 49) and peaked rows.
WORKLOADS = {
    "tiny_n512": Workload("tiny_n512", 1, 512, 2, 1, 64, 64, 1, 0,
                          note="tiny: batch 1, n=512, Hq=2, Hkv=1, d=64, b=64, L=1"),
    "qwen_n4096": Workload("qwen_n4096", 1, 4096, 16, 8, 128, 64, 2, 1,
                           note="Qwen3-0.6B layer geometry, n=4096"),
    "qwen_n32768": Workload("qwen_n32768", 1, 32768, 16, 8, 128, 64, 2, 2,
                            note="Qwen3-0.6B layer geometry, n=32768"),
    "qwen_n30001_b2_peaked": Workload("qwen_n30001_b2_peaked", 2, 30001, 16, 8, 128, 64, 2, 3,
                                      peak_frac=0.05, peak_mul=3.0,
                                      note="batch 2, n=30001 (partial last block), K x3 on 5% of positions"),
}


def sweep(b=64):
    """The length sweep 1K..64K in the Qwen3-0.6B geometry, seed 1000+log2(n)."""
    out = []
    for lg in range(10, 17):
        n = 1 << lg
        out.append(Workload(f"sweep_n{n}_b{b}", 1, n, 16, 8, 128, b, 2, 1000 + lg,
                            note=f"sweep point n={n}, b={b}"))
    return out


def make_qkv(w, device="cpu"):
    """Draw Q, K, V for workload ``w`` as bf16 torch tensors.

    Q: [batch, Hq, n, d]; K, V: [batch, Hkv, n, d].  Drawing happens on the
    host so that the bits do not depend on the device.
    """
    rng = np.random.Generator(np.random.PCG64(w.seed))
    q = rng.standard_normal((w.batch, w.Hq, w.n, w.d), dtype=np.float32)
    k = rng.standard_normal((w.batch, w.Hkv, w.n, w.d), dtype=np.float32)
    v = rng.standard_normal((w.batch, w.Hkv, w.n, w.d), dtype=np.float32)
    if w.peak_frac > 0.0 and w.n > 0:
        count = int(round(w.peak_frac * w.n))
        for beta in range(w.batch):
            pos = rng.choice(w.n, size=count, replace=False)
            k[beta, :, pos, :] *= np.float32(w.peak_mul)
    tq = torch.from_numpy(q).to(torch.bfloat16)
    tk = torch.from_numpy(k).to(torch.bfloat16)
    tv = torch.from_numpy(v).to(torch.bfloat16)
    if device != "cpu":
        tq, tk, tv = tq.to(device), tk.to(device), tv.to(device)
    return tq, tk, tv


def make_qkv_device(w, device="cuda"):
    """Q, K, V of workload w drawn on the device by a seeded torch generator
    (for lengths whose float32 host draws would not fit in host memory):
    bf16 standard normals in [batch, heads, n, head_dim] order, Q then K then
    V.  Not bit-identical to make_qkv; a test gives the oracle the device's
    bits by copying the rows it needs."""
    g = torch.Generator(device=device)
    g.manual_seed(w.seed)
    q = torch.randn((w.batch, w.Hq, w.n, w.d), generator=g, device=device, dtype=torch.bfloat16)
    k = torch.randn((w.batch, w.Hkv, w.n, w.d), generator=g, device=device, dtype=torch.bfloat16)
    v = torch.randn((w.batch, w.Hkv, w.n, w.d), generator=g, device=device, dtype=torch.bfloat16)
    return q, k, v


def make_qkv_large_logits(w, q_mul=8.0, k_ramp=9.0, diag=0.0, device="cpu"):
    """Inputs with scores in the hundreds whose row maximum keeps growing
    along a row: Q ~ q_mul N(0, 1) and K[s] ~ (1 + k_ramp s / n) N(0, 1), so
    later key blocks carry larger scores and a route visited in ascending
    block order sees its running maximum jump many times.  With diag > 0,
    K[s] also gets diag * (1 + k_ramp s / n) * sign(sum of the group's Q[s])
    added, which makes the diagonal key the largest score of most rows: the
    row maximum then arrives in the self block, visited last.  V ~ N(0, 1).
    All drawn as float32 on the host (PCG64 of the workload seed, stream 2)
    and rounded to bf16."""
    rng = np.random.Generator(np.random.PCG64([w.seed, 2]))
    q = rng.standard_normal((w.batch, w.Hq, w.n, w.d), dtype=np.float32) * np.float32(q_mul)
    k = rng.standard_normal((w.batch, w.Hkv, w.n, w.d), dtype=np.float32)
    if diag > 0.0:
        G = w.Hq // w.Hkv
        qsum = q.reshape(w.batch, w.Hkv, G, w.n, w.d).sum(axis=2)
        k += np.float32(diag) * np.sign(qsum).astype(np.float32)
    ramp = (1.0 + k_ramp * np.arange(w.n, dtype=np.float64) / max(w.n, 1)).astype(np.float32)
    k *= ramp[None, None, :, None]
    v = rng.standard_normal((w.batch, w.Hkv, w.n, w.d), dtype=np.float32)
    out = [torch.from_numpy(x).to(torch.bfloat16) for x in (q, k, v)]
    return tuple(t.to(device) if device != "cpu" else t for t in out)


def make_grad_out(w, device="cpu"):
    """Upstream gradient dO for workload ``w`` (bf16, Q's shape): standard
    normal from its own seeded stream (PCG64 of the workload seed, stream 1),
    so that Q, K, V are the same with or without it."""
    rng = np.random.Generator(np.random.PCG64([w.seed, 1]))
    g = rng.standard_normal((w.batch, w.Hq, w.n, w.d), dtype=np.float32)
    t = torch.from_numpy(g).to(torch.bfloat16)
    return t.to(device) if device != "cpu" else t


def to_f64(t):
    """Exact float64 copy of a bf16 tensor as a NumPy array."""
    return t.detach().to("cpu").to(torch.float64).numpy()


# ---------------------------------------------------------------------------
# Decode: paged key/value caches
# ---------------------------------------------------------------------------
# The paper characterises one-token decode at contexts 32K and 64K for batch
# 1, 8 and 32 in the same attention geometry (§5.4, Table 3).  A cache page
# holds one block of b tokens of one sequence; pages are handed out in a
# seeded random order (a fragmented pool, as a serving allocator leaves it),
# and pages no sequence owns ("decoys") hold other values.

@dataclass(frozen=True)
class DecodeWorkload:
    name: str
    batch: int
    ctx: int          # tokens in the cache of the longest sequence (newest included)
    Hq: int
    Hkv: int
    d: int
    b: int
    L: int
    seed: int
    ragged: bool = False   # lengths uniform in [ctx/2, ctx] instead of all ctx
    note: str = ""


DECODE_WORKLOADS = {
    f"decode_n{ctx}_batch{bt}": DecodeWorkload(f"decode_n{ctx}_batch{bt}", bt, ctx, 16, 8, 128, 64, 2,
                                               4000 + bt + ctx // 1024,
                                               note=f"Qwen3-0.6B geometry, {bt} sequences of {ctx} tokens")
    for ctx in (32768, 65536) for bt in (1, 8, 32)
}


def decode_seq_lens(w):
    """Sequence lengths (int32 numpy) of a decode workload."""
    if not w.ragged:
        return np.full(w.batch, w.ctx, dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64([w.seed, 2]))
    return rng.integers(max(1, w.ctx // 2), w.ctx + 1, size=w.batch).astype(np.int32)


def make_decode_host(w, seq_lens=None):
    """Host draw for small decode cases: the newest token's query
    [batch, Hq, d] and logical caches K, V [batch, Hkv, n_max, d] (bf16
    torch tensors), n_max = the longest sequence; positions past a
    sequence's length hold values it must never read."""
    if seq_lens is None:
        seq_lens = decode_seq_lens(w)
    n_max = int(max(seq_lens))
    rng = np.random.Generator(np.random.PCG64(w.seed))
    q = rng.standard_normal((w.batch, w.Hq, w.d), dtype=np.float32)
    k = rng.standard_normal((w.batch, w.Hkv, n_max, w.d), dtype=np.float32)
    v = rng.standard_normal((w.batch, w.Hkv, n_max, w.d), dtype=np.float32)
    return (torch.from_numpy(q).to(torch.bfloat16), torch.from_numpy(k).to(torch.bfloat16),
            torch.from_numpy(v).to(torch.bfloat16), np.asarray(seq_lens, dtype=np.int32))


def page_cache(k, v, seq_lens, b, seed, spare_pages=3, decoy=float("nan")):
    """Scatter logical caches [batch, Hkv, n_max, d] into pages
    [num_pages, Hkv, b, d] in a seeded random page order.  Returns
    (k_pages, v_pages, page_table [batch, max_pages] int32, num_pages).
    Page-table slots past a sequence's last block hold -1; spare pages and
    the unused tail of each sequence's last page hold ``decoy``."""
    batch, Hkv, n_max, d = k.shape
    max_pages = -(-n_max // b)
    owned = [-(-int(n) // b) for n in seq_lens]
    num_pages = sum(owned) + spare_pages
    rng = np.random.Generator(np.random.PCG64([seed, 3]))
    order = rng.permutation(num_pages)
    kp = torch.full((num_pages, Hkv, b, d), decoy, dtype=torch.bfloat16)
    vp = torch.full((num_pages, Hkv, b, d), decoy, dtype=torch.bfloat16)
    table = np.full((batch, max_pages), -1, dtype=np.int32)
    nxt = 0
    for beta in range(batch):
        n = int(seq_lens[beta])
        for i in range(owned[beta]):
            page = int(order[nxt])
            nxt += 1
            table[beta, i] = page
            lo, hi = i * b, min((i + 1) * b, n)
            kp[page, :, : hi - lo] = k[beta, :, lo:hi]
            vp[page, :, : hi - lo] = v[beta, :, lo:hi]
    return kp, vp, torch.from_numpy(table), num_pages


def make_decode_device(w, device="cuda"):
    """Full-size decode inputs drawn on the device (a seeded torch generator;
    the caches are gigabytes): q [batch, Hq, d], k_pages, v_pages
    [num_pages, Hkv, b, d] bf16 standard normals, page_table [batch,
    max_pages] int32 (a seeded random page order), seq_lens int32."""
    seq_lens = decode_seq_lens(w)
    max_pages = -(-w.ctx // w.b)
    owned = [-(-int(n) // w.b) for n in seq_lens]
    num_pages = sum(owned)
    g = torch.Generator(device=device)
    g.manual_seed(w.seed)
    q = torch.randn((w.batch, w.Hq, w.d), generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)
    kp = torch.randn((num_pages, w.Hkv, w.b, w.d), generator=g, device=device, dtype=torch.bfloat16)
    vp = torch.randn((num_pages, w.Hkv, w.b, w.d), generator=g, device=device, dtype=torch.bfloat16)
    rng = np.random.Generator(np.random.PCG64([w.seed, 3]))
    order = rng.permutation(num_pages).astype(np.int32)
    table = np.full((w.batch, max_pages), -1, dtype=np.int32)
    at = 0
    for beta in range(w.batch):
        table[beta, :owned[beta]] = order[at:at + owned[beta]]
        at += owned[beta]
    return (q, kp, vp, torch.from_numpy(seq_lens).to(device), torch.from_numpy(table).to(device),
            num_pages)


# ---------------------------------------------------------------------------
# Whole-model prefill timing: a decoder stack of the evaluated geometry
# ---------------------------------------------------------------------------
# The paper times whole-model prefill (time to first token) of Qwen3-0.6B with
# 8 or all 28 attention layers on the BF1 route (§4.3, §5.3).  The trained
# weights are not available here, so the stack gets seeded random weights of
# the published Qwen3-0.6B shapes: timing does not depend on their values.

@dataclass(frozen=True)
class ModelConfig:
    layers: int = 28
    hidden: int = 1024
    heads: int = 16
    kv_heads: int = 8
    head_dim: int = 128
    intermediate: int = 3072
    vocab: int = 151936
    rope_theta: float = 1.0e6
    eps: float = 1.0e-6


QWEN3_06B = ModelConfig()

_WEIGHT_SHAPES = {
    "in_norm": lambda c: (c.hidden,),
    "wq": lambda c: (c.hidden, c.heads * c.head_dim),
    "wk": lambda c: (c.hidden, c.kv_heads * c.head_dim),
    "wv": lambda c: (c.hidden, c.kv_heads * c.head_dim),
    "q_norm": lambda c: (c.head_dim,),
    "k_norm": lambda c: (c.head_dim,),
    "wo": lambda c: (c.heads * c.head_dim, c.hidden),
    "post_norm": lambda c: (c.hidden,),
    "wg": lambda c: (c.hidden, c.intermediate),
    "wu": lambda c: (c.hidden, c.intermediate),
    "wd": lambda c: (c.intermediate, c.hidden),
}


def make_model_weights(cfg, seed, device="cpu"):
    """Seeded random weights (bf16): "embed" [vocab, hidden] (tied output
    head), "final_norm" [hidden], and per layer l the entries "l.<name>" of
    _WEIGHT_SHAPES, projections stored [in, out] (x @ W).  Projection entries
    are N(0, 1/in), norm gains 1 + N(0, 0.1^2), embeddings N(0, 1).  Drawn on
    the host with PCG64 for device "cpu", else with a seeded torch generator
    on the device (the full-size stack holds 0.6 G parameters)."""
    out = {}
    if device == "cpu":
        rng = np.random.Generator(np.random.PCG64([seed, 4]))
        draw = lambda shape: torch.from_numpy(rng.standard_normal(shape, dtype=np.float32))
    else:
        g = torch.Generator(device=device)
        g.manual_seed(seed)
        draw = lambda shape: torch.randn(shape, generator=g, device=device, dtype=torch.float32)

    def put(name, shape):
        x = draw(shape)
        if name.endswith("norm"):
            x = 1.0 + 0.1 * x
        elif name != "embed":
            x = x / float(np.sqrt(shape[0]))
        out[name] = x.to(torch.bfloat16)

    put("embed", (cfg.vocab, cfg.hidden))
    for l in range(cfg.layers):
        for name, shape in _WEIGHT_SHAPES.items():
            put(f"{l}.{name}", shape(cfg))
    put("final_norm", (cfg.hidden,))
    return out


def make_tokens(cfg, n, seed):
    """n token ids (int64 numpy), uniform over the vocabulary."""
    rng = np.random.Generator(np.random.PCG64([seed, 5]))
    return rng.integers(0, cfg.vocab, size=n, dtype=np.int64)
