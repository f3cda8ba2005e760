"""Pins of the oracle's attention values (CPU only).

The oracle computes exact softmax attention restricted to the BF1 token mask
(§3.1).  Its arithmetic is pinned against things other than itself:

* PyTorch's own scaled-dot-product attention (float64, CPU) under a boolean
  mask built here from the hand-derived routes of Eq. 1 (golden fixture);
* the textbook dense causal softmax when the route covers every block;
* closed forms at K = 0 (uniform weights over the selected set);
* single-key rows, future-token isolation (§4.2) and GQA head grouping.
"""

import math

import numpy as np
import pytest
import torch

from conftest import read_golden
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

F = torch.nn.functional


def sdpa_ref(q, k, v, mask=None, causal=False):
    """Library reference: torch SDPA in float64 on the CPU with GQA."""
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(x)).double() for x in (q, k, v))
    G = tq.shape[1] // tk.shape[1]
    tk = tk.repeat_interleave(G, dim=1)
    tv = tv.repeat_interleave(G, dim=1)
    am = None if mask is None else torch.from_numpy(mask)
    o = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=am, is_causal=causal)
    return o.numpy()


def sdpa_lse(q, k, mask=None, causal=False):
    """log-sum-exp of the scaled scores by torch.logsumexp (float64)."""
    tq, tk = (torch.from_numpy(np.ascontiguousarray(x)).double() for x in (q, k))
    G = tq.shape[1] // tk.shape[1]
    tk = tk.repeat_interleave(G, dim=1)
    x = tq @ tk.transpose(-1, -2) / math.sqrt(tq.shape[-1])
    n = x.shape[-1]
    if causal:
        mask = np.tril(np.ones((n, n), dtype=bool))
    if mask is not None:
        x = x.masked_fill(~torch.from_numpy(mask), float("-inf"))
    return torch.logsumexp(x, dim=-1).numpy()


def hand_mask(n, b):
    """Token mask built from the hand-derived L=2 routes (golden fixture),
    independent of the oracle's route enumeration."""
    routes = {}
    for row in read_golden("routes_hand.txt"):
        if int(row[0]) == 2:
            routes[int(row[1])] = [int(x) for x in row[3:]]
    NB = -(-n // b)
    assert all(j in routes for j in range(NB)), "fixture too short for this n"
    mask = np.zeros((n, n), dtype=bool)
    for t in range(n):
        j = t // b
        for i in routes[j]:
            for s in range(i * b, min((i + 1) * b, n)):
                if i < j or s <= t:
                    mask[t, s] = True
    return mask


def rand_qkv(batch, Hq, Hkv, n, d, seed):
    w = synth.Workload("t", batch, n, Hq, Hkv, d, 64, 2, seed)
    q, k, v = synth.make_qkv(w)
    return synth.to_f64(q), synth.to_f64(k), synth.to_f64(v)


@pytest.mark.parametrize("n,b", [(70, 4), (72, 4), (35, 2), (144, 8)])
def test_oracle_equals_library_sdpa_on_hand_mask(n, b):
    q, k, v = rand_qkv(2, 4, 2, n, 16, seed=11 + n)
    mask = hand_mask(n, b)
    ref_o = sdpa_ref(q, k, v, mask=mask)
    ref_l = sdpa_lse(q, k, mask=mask)
    o1, l1 = orc.attn_full_mask_fp64(q, k, v, b, 2)
    o2, l2 = orc.attn_gathered_fp64(q, k, v, b, 2)
    for o, l in ((o1, l1), (o2, l2)):
        assert np.abs(o - ref_o).max() < 1e-12
        assert np.abs(l - ref_l).max() < 1e-12


@pytest.mark.parametrize("n,b,L", [(512, 64, 1), (257, 64, 2), (777, 64, 3), (1000, 32, 2), (130, 8, 0)])
def test_full_mask_equals_gathered(n, b, L):
    q, k, v = rand_qkv(1, 2, 1, n, 32, seed=n + L)
    o1, l1 = orc.attn_full_mask_fp64(q, k, v, b, L)
    o2, l2 = orc.attn_gathered_fp64(q, k, v, b, L)
    assert np.abs(o1 - o2).max() < 1e-12
    assert np.abs(l1 - l2).max() < 1e-12


@pytest.mark.parametrize("n,b,L", [(256, 64, 2), (200, 64, 2), (640, 64, 8), (64, 64, 0), (40, 64, 0)])
def test_route_covering_every_block_is_dense_causal(n, b, L):
    # When NB <= L + 2 (or n <= b) every earlier block is selected, so the
    # BF1 operator reduces to textbook dense causal attention.
    assert orc.num_blocks(n, b) <= L + 2 or n <= b
    q, k, v = rand_qkv(1, 4, 2, n, 32, seed=5 + n)
    o, l = orc.attn_gathered_fp64(q, k, v, b, L)
    assert np.abs(o - sdpa_ref(q, k, v, causal=True)).max() < 1e-12
    assert np.abs(l - sdpa_lse(q, k, causal=True)).max() < 1e-12
    od, ld = orc.dense_causal_fp64(q, k, v)
    assert np.abs(od - o).max() < 1e-12 and np.abs(ld - l).max() < 1e-12


def test_route_not_covering_differs_from_dense():
    # Sanity: at NB = L + 3 some earlier block is dropped, so rows differ.
    n, b = 5 * 64, 64
    q, k, v = rand_qkv(1, 2, 1, n, 32, seed=3)
    o, _ = orc.attn_gathered_fp64(q, k, v, b, 2)
    od, _ = orc.dense_causal_fp64(q, k, v)
    assert np.abs(o[:, :, 4 * 64:] - od[:, :, 4 * 64:]).max() > 1e-3
    assert np.abs(o[:, :, : 4 * 64] - od[:, :, : 4 * 64]).max() < 1e-12


@pytest.mark.parametrize("n,b,L", [(777, 64, 2), (512, 64, 1), (300, 16, 0)])
def test_zero_keys_closed_form(n, b, L):
    # K = 0: every visible score is 0, so softmax is uniform over the
    # selected set S(t): LSE_t = ln |S(t)| with
    # |S(t)| = (t mod b) + 1 + b * (number of earlier selected blocks), and O_t
    # is the mean of V over S(t).
    q, k, v = rand_qkv(1, 2, 1, n, 16, seed=7)
    k = np.zeros_like(k)
    o, l = orc.attn_gathered_fp64(q, k, v, b, L)
    t = np.arange(n)
    size = np.array([(tt % b) + 1 + b * (len(orc.route(tt // b, L)) - 1) for tt in t])
    assert np.abs(l[0, 0] - np.log(size)).max() < 1e-12
    for tt in [0, 1, b - 1, b, n - 1, n // 2, 3 * b + 5]:
        if tt >= n:
            continue
        j = tt // b
        keys = [s for i in orc.route(j, L) for s in range(i * b, min((i + 1) * b, n)) if i < j or s <= tt]
        assert len(keys) == size[tt]
        assert np.abs(o[0, 1, tt] - v[0, 0, keys].mean(axis=0)).max() < 1e-12


def test_first_row_is_first_value():
    q, k, v = rand_qkv(1, 2, 1, 130, 16, seed=9)
    o, l = orc.attn_gathered_fp64(q, k, v, 64, 2)
    assert np.array_equal(o[0, :, 0], v[0, [0, 0], 0])
    for h in range(2):
        assert abs(l[0, h, 0] - q[0, h, 0] @ k[0, 0, 0] / 4.0) < 1e-14


@pytest.mark.parametrize("t0", [1, 63, 64, 100, 511])
def test_future_token_isolation_oracle(t0):
    # §4.2: mutating future tokens must leave earlier outputs unchanged.
    n, b = 512, 64
    q, k, v = rand_qkv(1, 2, 1, n, 32, seed=21)
    o, l = orc.attn_gathered_fp64(q, k, v, b, 2)
    rng = np.random.default_rng(5)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for x in (q2, k2, v2):
        x[:, :, t0:] = rng.standard_normal(x[:, :, t0:].shape) * 4
    o2, l2 = orc.attn_gathered_fp64(q2, k2, v2, b, 2)
    assert np.array_equal(o[:, :, :t0], o2[:, :, :t0])
    assert np.array_equal(l[:, :, :t0], l2[:, :, :t0])
    assert not np.array_equal(o[:, :, t0:], o2[:, :, t0:])


def test_gqa_grouping_contiguous():
    # q-head h reads kv-head h // (Hq/Hkv): with distinct K/V per kv-head a
    # wrong mapping fails the comparison with per-head dense attention.
    n, b = 256, 64
    q, k, v = rand_qkv(1, 8, 2, n, 16, seed=4)
    o, _ = orc.attn_gathered_fp64(q, k, v, b, 2)
    for h in range(8):
        g = h // 4
        oh = sdpa_ref(q[:, h:h + 1], k[:, g:g + 1], v[:, g:g + 1], causal=True)
        assert np.abs(o[:, h:h + 1] - oh).max() < 1e-12


def test_partial_last_block_rows():
    # n = 257 (the paper's partial-block gate, §4.2): the last block has one
    # token, which sees itself plus every earlier selected block.
    q, k, v = rand_qkv(1, 2, 1, 257, 16, seed=8)
    mask = orc.token_mask(257, 64, 2)
    assert mask[256].sum() == 1 + 64 * (len(orc.route(4, 2)) - 1)
    o, l = orc.attn_gathered_fp64(q, k, v, 64, 2)
    ref = sdpa_ref(q, k, v, mask=mask)
    assert np.abs(o - ref).max() < 1e-12


def test_csr_attention_matches_route_attention():
    n, b = 640, 64
    q, k, v = rand_qkv(1, 2, 1, n, 16, seed=10)
    rp, ci = orc.csr(n, b, 2)
    o1, l1 = orc.attn_csr_fp64(q, k, v, b, rp, ci)
    o2, l2 = orc.attn_full_mask_fp64(q, k, v, b, 2)
    assert np.abs(o1 - o2).max() < 1e-12 and np.abs(l1 - l2).max() < 1e-12


def test_block_subset():
    n, b = 640, 64
    q, k, v = rand_qkv(1, 2, 1, n, 16, seed=12)
    o, l = orc.attn_gathered_fp64(q, k, v, b, 2)
    os_, ls_ = orc.attn_gathered_fp64(q, k, v, b, 2, blocks=[0, 7, 9])
    for j in [0, 7, 9]:
        sl = slice(j * b, (j + 1) * b)
        assert np.array_equal(o[:, :, sl], os_[:, :, sl])
    assert np.isnan(os_[:, :, 64:128]).all()


def test_input_generator_is_seeded_and_bf16():
    w = synth.WORKLOADS["tiny_n512"]
    a = synth.make_qkv(w)
    b = synth.make_qkv(w)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16 and torch.equal(x, y)
    assert a[0].shape == (1, 2, 512, 64) and a[1].shape == (1, 1, 512, 64)
    # The peaked draw equals the plain draw except that K is scaled on exactly
    # round(0.05 n) token positions of each batch element (all heads, dims).
    wp = synth.Workload("p", 2, 1000, 2, 1, 16, 64, 2, 3, peak_frac=0.05)
    _, kp, _ = synth.make_qkv(wp)
    _, k0, _ = synth.make_qkv(wp.with_(peak_frac=0.0))
    changed = (kp != k0).any(dim=-1)          # [batch, Hkv, n]
    for beta in range(2):
        pos = changed[beta].all(dim=0).nonzero().flatten()
        assert len(pos) == 50
        assert torch.equal(changed[beta].any(dim=0), changed[beta].all(dim=0))
        ratio = kp[beta][:, pos].float() / k0[beta][:, pos].float()
        assert (ratio - 3).abs().max() < 0.02
