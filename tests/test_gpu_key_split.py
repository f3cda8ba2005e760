"""The forward's two key-group path (short sequences: two groups of waves take
alternate key tiles of each route and merge their softmax states) against the
fp64 oracle, forced on and off for the same inputs; the automatic choice must
be bitwise one of the two forced paths, the split one exactly when the launch
has at most one work item per compute unit."""

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
import test_gpu_parity as TP
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()
    yield
    bf1.set_forward_key_split(0)
    torch.cuda.synchronize()


CASES = [
    # batch, n, Hq, Hkv, d, B, L
    (1, 1024, 16, 8, 128, 64, 2),     # the 1K sweep point (128 items)
    (1, 2048, 16, 8, 128, 128, 2),    # 2K, b = 128
    (2, 1337, 4, 2, 64, 64, 2),       # ragged, batch 2, d = 64
    (1, 512, 2, 1, 64, 64, 1),        # the tiny workload
    (1, 700, 2, 2, 128, 64, 3),       # G = 1 (two-wave groups)
    (1, 901, 16, 2, 128, 128, 2),     # G = 8, B = 128 (chunks)
    (1, 1, 2, 1, 128, 64, 2),         # one tile: the second group only has a dummy
    (1, 130, 2, 1, 128, 64, 2),       # three tiles: odd count
    (1, 257, 4, 2, 128, 64, 0),       # L = 0
]


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: "x".join(map(str, c)))
def test_both_paths_against_oracle(cfg):
    w = synth.Workload("ks", *cfg, seed=70 + cfg[1])
    q, k, v = synth.make_qkv(w, device="cuda")
    o_ref, l_ref = orc.attn_gathered_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), w.b, w.L)
    outs = {}
    for mode in (1, 2, 0):
        bf1.set_forward_key_split(mode)
        outs[mode] = bf1.attn_fwd(q, k, v, B=w.b, L=w.L)
        torch.cuda.synchronize()
    bf1.set_forward_key_split(0)
    for mode in (1, 2):
        TP.compare(*outs[mode], o_ref, l_ref, tag=f"key groups mode {mode} {cfg}")
    nchunk = max(1, (w.Hq // w.Hkv) * w.b // 128)      # 128-row chunks per query block
    items = -(-w.n // w.b) * w.batch * w.Hkv * nchunk
    tiles = bf1.plan_size(w.n, w.b, w.L)[1] * (w.b // 64) * w.batch * w.Hkv * nchunk
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    pick = 2 if items <= cus and tiles >= 8 * items else 1
    assert torch.equal(outs[0][0], outs[pick][0]) and torch.equal(outs[0][1], outs[pick][1])


def test_dense_automatic_choice():
    # the dense route averages (NB + 1) / 2 tiles per item: split at 1K (16
    # blocks, 8 kv-heads: 128 items, 8.5 tiles each), not at 8K (1024 items)
    for n, split in ((1024, True), (8192, False)):
        w = synth.Workload("ksa", 1, n, 16, 8, 128, 64, 2, seed=82)
        q, k, v = synth.make_qkv(w, device="cuda")
        outs = {}
        for mode in (0, 1, 2):
            bf1.set_forward_key_split(mode)
            outs[mode] = bf1.dense_causal_fwd(q, k, v)
        torch.cuda.synchronize()
        pick = 2 if split and 128 <= torch.cuda.get_device_properties(0).multi_processor_count else 1
        assert torch.equal(outs[0][0], outs[pick][0]) and torch.equal(outs[0][1], outs[pick][1]), n
    bf1.set_forward_key_split(0)


def test_dense_both_paths_and_covering_route():
    # dense causal through both paths; and with either path forced, the BF1
    # kernel with a covering route equals the dense kernel bitwise
    w = synth.Workload("ksd", 1, 1000, 4, 2, 128, 64, 14, seed=81)
    q, k, v = synth.make_qkv(w, device="cuda")
    rows = np.arange(0, 1000, 7)
    o_ref, l_ref = orc.dense_causal_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), rows=rows)
    for mode in (1, 2):
        bf1.set_forward_key_split(mode)
        od, ld = bf1.dense_causal_fwd(q, k, v)
        ob, lb = bf1.attn_fwd(q, k, v, B=64, L=14)
        torch.cuda.synchronize()
        TP.compare(od, ld, o_ref, l_ref, rows=rows, tag=f"dense mode {mode}")
        assert torch.equal(od, ob) and torch.equal(ld, lb)
    bf1.set_forward_key_split(0)


def test_large_logits_two_groups():
    # the merge of the two groups' running maxima under scores in the hundreds
    w = synth.Workload("ksbig", 1, 2048 + 37, 4, 2, 128, 64, 2, seed=33)
    q, k, v = synth.make_qkv_large_logits(w, diag=0.5, device="cuda")
    o_ref, l_ref = orc.attn_gathered_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), 64, 2)
    for mode in (1, 2):
        bf1.set_forward_key_split(mode)
        o, l = bf1.attn_fwd(q, k, v, B=64, L=2)
        torch.cuda.synchronize()
        TP.compare(o, l, o_ref, l_ref, tag=f"large logits mode {mode}")
    bf1.set_forward_key_split(0)

