"""Every instance the C ABI advertises, compared with the fp64 oracle on the
GPU: forward BF1 (head_dim x group x block width: 16 instances), the dense
comparator (8), the backward (the 14 with G * B >= 128) and decode (16), each
at batch 2 with a ragged length (n = 5 B + 37: several tiles and a partial
last block); plus forward cases whose scores reach the hundreds, so that the
lazily rescaled running maximum moves by more than 2^8 several times per row
and the row maximum often arrives in the last tile visited.

Bars: the forward's (O max-abs 2e-2, mean-abs 2e-3, LSE max-abs 1e-3); the
backward's element-wise bound derived from its arithmetic (see
test_gpu_backward.py)."""

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
import test_gpu_backward as TB
import test_gpu_decode as TD
import test_gpu_parity as TP
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu

D = (64, 128)
GROUPS = (1, 2, 4, 8)
WIDTHS = (64, 128)
GRID = [(d, G, B) for d in D for G in GROUPS for B in WIDTHS]
BWD_GRID = [(d, G, B) for (d, G, B) in GRID if G * B >= 128]
ident = lambda c: "d{}_G{}_B{}".format(*c)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()
    yield
    torch.cuda.synchronize()


def _workload(d, G, B, seed):
    return synth.Workload("grid", 2, 5 * B + 37, 2 * G, 2, d, B, 2, seed=seed)


@pytest.mark.parametrize("cfg", GRID, ids=ident)
def test_forward_every_instance(cfg):
    d, G, B = cfg
    TP.say(f"grid forward {cfg}")
    w = _workload(d, G, B, seed=3000 + d + 10 * G + B)
    q, k, v = synth.make_qkv(w, device="cuda")
    o, lse = bf1.attn_fwd(q, k, v, B=B, L=2)
    torch.cuda.synchronize()
    o_ref, l_ref = orc.attn_gathered_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), B, 2)
    TP.compare(o, lse, o_ref, l_ref, tag=f"forward {cfg}")


@pytest.mark.parametrize("cfg", [(d, G) for d in D for G in GROUPS], ids=lambda c: "d{}_G{}".format(*c))
def test_dense_every_instance(cfg):
    d, G = cfg
    TP.say(f"grid dense {cfg}")
    w = _workload(d, G, 64, seed=3100 + d + G)
    q, k, v = synth.make_qkv(w, device="cuda")
    o, lse = bf1.dense_causal_fwd(q, k, v)
    torch.cuda.synchronize()
    o_ref, l_ref = orc.dense_causal_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v))
    TP.compare(o, lse, o_ref, l_ref, tag=f"dense {cfg}")


@pytest.mark.parametrize("cfg", BWD_GRID, ids=ident)
def test_backward_every_instance(cfg):
    d, G, B = cfg
    TP.say(f"grid backward {cfg}")
    w = _workload(d, G, B, seed=3200 + d + 10 * G + B)
    (dq, dk, dv), ref, terms = TB.run_case(w)
    for name, got, r, t in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref, terms):
        TB.check_bound(got, r, t, tag=f"backward {cfg} {name}")


@pytest.mark.parametrize("cfg", GRID, ids=ident)
def test_decode_every_instance(cfg):
    d, G, B = cfg
    TP.say(f"grid decode {cfg}")
    lens = np.array([5 * B + 37, B + 1], dtype=np.int32)
    w = synth.DecodeWorkload("grid", 2, int(lens.max()), 2 * G, 2, d, B, 2, seed=3300 + d + 10 * G + B)
    (q, k, v, sl, _), dev = TD.setup_case(w, lens)
    o, l, _ = TD.run_decode(w, dev)
    o_ref, l_ref = orc.attn_decode_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), sl, B, 2)
    TD.compare(o, l, o_ref, l_ref, f"decode {cfg}")


@pytest.mark.parametrize("cfg", [(128, 2, 64, 0.0), (128, 2, 64, 0.5), (64, 2, 64, 0.5), (128, 8, 64, 0.5),
                                 (128, 2, 128, 0.5), (64, 1, 128, 0.5)],
                         ids=lambda c: "d{}_G{}_B{}_diag{}".format(*c))
def test_forward_large_logits(cfg):
    # Scores of several hundred (natural-log units): the running maximum of a
    # row jumps past the 2^8 lazy-rescale threshold several times along the
    # ascending route, and with the diagonal planted the row maximum mostly
    # arrives in the self block, the last tile of the row.
    d, G, B, diag = cfg
    TP.say(f"large logits {cfg}")
    w = synth.Workload("big", 1, 4096 + 37, 2 * G, 2, d, B, 2, seed=31)
    q, k, v = synth.make_qkv_large_logits(w, diag=diag, device="cuda")
    o, lse = bf1.attn_fwd(q, k, v, B=B, L=2)
    torch.cuda.synchronize()
    o_ref, l_ref = orc.attn_gathered_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), B, 2)
    assert np.abs(l_ref).max() > 200.0
    TP.compare(o, lse, o_ref, l_ref, tag=f"large logits {cfg}")


def test_dense_large_logits():
    w = synth.Workload("big", 1, 2048 + 37, 4, 2, 128, 64, 2, seed=32)
    q, k, v = synth.make_qkv_large_logits(w, diag=0.5, device="cuda")
    o, lse = bf1.dense_causal_fwd(q, k, v)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, 70), np.arange(w.n - 70, w.n),
                                     np.random.default_rng(2).integers(0, w.n, 100)]))
    o_ref, l_ref = orc.dense_causal_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), rows=rows)
    TP.compare(o, lse, o_ref, l_ref, rows=rows, tag="dense large logits")
