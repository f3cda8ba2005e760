"""GPU parity of the backward (dQ, dK, dV) against the fp64 CPU oracle.

Bar (derived from the arithmetic of the kernels, not from their outputs): the kernels
take exact bf16 inputs, accumulate in fp32 and round only two quantities to
bf16 before a product -- the weights P (for dV = P^T dO) and dS (for
dQ = c dS K and dK = c dS^T Q).  Rounding to bf16 (8 significant bits,
round to nearest) has relative error <= 2^-8.  Every gradient element is a
sum of such products, so its error is at most 2^-8 times the sum of the
magnitudes of its terms (the oracle's attn_bwd_abs_terms_fp64, kind "ds").
The fp32 part of dS = P (dP - D) cancels: its error scales with
P (|dP| + |D|) (kind "pdp") times the fp32 unit roundoff and the length of
the dot products behind dP and D (128 terms: 2^-17).  The test allows 2^-8
times the first sum, 2^-16 times the second, and 1e-5 of the largest first
sum for fp32 accumulation and exponential rounding.

The kernels compute D = rowsum(dO * O) from the O they are given; the parity
cases feed them the oracle's O (rounded to bf16) and LSE, and the oracle uses
the same O.  A separate chained case feeds the GPU forward's outputs.
"""

import sys

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()
    yield
    torch.cuda.synchronize()


def _rows(blocks, b, n):
    return np.concatenate([np.arange(j * b, min((j + 1) * b, n)) for j in blocks])


def check_bound(got, ref, terms, rows=None, tag=""):
    terms, tpdp = terms
    g = got.cpu().double().numpy()
    if rows is not None:
        g, ref, terms, tpdp = g[:, :, rows], ref[:, :, rows], terms[:, :, rows], tpdp[:, :, rows]
    assert np.isfinite(g).all(), tag
    err = np.abs(g - ref)
    bound = 2.0 ** -8 * terms + 2.0 ** -16 * tpdp + 1e-5 * terms.max()
    worst = float((err / bound).max())
    say(f"  {tag}: max err {err.max():.3e}, max err/bound {worst:.3f}")
    assert (err <= bound).all(), (tag, worst)


def run_case(w, q_blocks=None, kv_blocks=None):
    q, k, v = synth.make_qkv(w)
    do = synth.make_grad_out(w)
    qf, kf, vf, dof = (synth.to_f64(t) for t in (q, k, v, do))
    o_ref, lse_ref = orc.attn_gathered_fp64(qf, kf, vf, w.b, w.L,
                                            blocks=None if q_blocks is None and kv_blocks is None else None)
    o_bf = torch.from_numpy(o_ref).to(torch.bfloat16)
    o_used = synth.to_f64(o_bf)
    lse32 = torch.from_numpy(lse_ref.astype(np.float32))
    dev = "cuda"
    dq, dk, dv = bf1.attn_bwd(q.to(dev), k.to(dev), v.to(dev), o_bf.to(dev), do.to(dev),
                              lse32.to(dev), w.b, w.L)
    torch.cuda.synchronize()
    ref = orc.attn_bwd_gathered_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used,
                                     q_blocks=q_blocks, kv_blocks=kv_blocks)
    terms = orc.attn_bwd_abs_terms_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used,
                                        q_blocks=q_blocks, kv_blocks=kv_blocks)
    tpdp = orc.attn_bwd_abs_terms_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used,
                                       q_blocks=q_blocks, kv_blocks=kv_blocks, kind="pdp")
    return (dq, dk, dv), ref, list(zip(terms, tpdp))


SMALL = [
    # batch, n, Hq, Hkv, B, L
    (1, 512, 2, 1, 64, 1),       # tiny geometry with d = 128
    (1, 257, 2, 1, 64, 2),       # partial block of one token
    (2, 1000, 4, 2, 64, 2),      # ragged tail, batch 2
    (1, 777, 4, 1, 64, 3),       # G = 4, L = 3
    (1, 640, 8, 1, 64, 2),       # G = 8
    (1, 900, 2, 2, 128, 2),      # G = 1 with B = 128
    (1, 1500, 4, 2, 128, 2),     # B = 128, ragged
    (2, 1300, 8, 2, 128, 2),     # G = 4 with B = 128 (four 128-row chunks per block), batch 2
    (1, 700, 8, 1, 128, 3),      # G = 8 with B = 128, L = 3
    (1, 2048, 16, 8, 64, 2),     # Qwen geometry, short
    (1, 1, 2, 1, 64, 2),         # a single token
    (1, 65, 2, 1, 64, 2),        # n = B + 1
    (1, 1200, 2, 1, 64, 0),      # L = 0
]


SMALL_D64 = [
    # batch, n, Hq, Hkv, B, L  (head_dim 64)
    (1, 512, 2, 1, 64, 1),       # the tiny workload's geometry
    (2, 1000, 4, 2, 64, 2),      # ragged tail, batch 2
    (1, 900, 2, 2, 128, 2),      # G = 1 with B = 128
    (1, 2048, 16, 8, 64, 2),     # 16 / 8 heads
    (1, 1, 2, 1, 64, 2),         # a single token
    (1, 64 * 40, 8, 1, 64, 3),   # G = 8, key block 0's list split into segments
]


@pytest.mark.parametrize("cfg", SMALL_D64, ids=lambda c: "x".join(map(str, c)))
def test_backward_head_dim_64_full_oracle(cfg):
    batch, n, Hq, Hkv, B, L = cfg
    say(f"backward d=64 {cfg}")
    w = synth.Workload("bwd64", batch, n, Hq, Hkv, 64, B, L, seed=900 + n)
    (dq, dk, dv), ref, terms = run_case(w)
    for name, got, r, t in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref, terms):
        check_bound(got, r, t, tag=f"d64 {cfg} {name}")


def test_backward_tiny_workload_chained():
    # the tiny workload (n = 512, Hq 2, Hkv 1, d 64, L 1) through the GPU forward and backward
    w = synth.WORKLOADS["tiny_n512"]
    q, k, v = synth.make_qkv(w, device="cuda")
    do = synth.make_grad_out(w, device="cuda")
    o, lse = bf1.attn_fwd(q, k, v, w.b, w.L)
    dq, dk, dv = bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L)
    torch.cuda.synchronize()
    ref = orc.attn_bwd_gathered_fp64(*(synth.to_f64(t) for t in (q, k, v, do)), w.b, w.L)
    for name, got, r in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref):
        err = np.abs(got.cpu().double().numpy() - r).max()
        say(f"  tiny chained {name}: max err {err:.3e} (max |ref| {np.abs(r).max():.3e})")
        assert err <= 2e-2 * np.abs(r).max(), name


@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: "x".join(map(str, c)))
def test_backward_small_full_oracle(cfg):
    batch, n, Hq, Hkv, B, L = cfg
    say(f"backward {cfg}")
    w = synth.Workload("bwd", batch, n, Hq, Hkv, 128, B, L, seed=500 + n)
    (dq, dk, dv), ref, terms = run_case(w)
    for name, got, r, t in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref, terms):
        check_bound(got, r, t, tag=f"{cfg} {name}")


def test_backward_long_list_segments():
    # n = 64 * 300: key block 0 is selected by 300 query blocks -> 19 segments
    # summed by the reduce kernel; the other lists fit one segment.
    w = synth.Workload("bwd_long", 1, 64 * 300, 2, 1, 128, 64, 2, seed=77)
    say("backward long lists")
    NB = 300
    kv = [0, 1, 2, 150, 298, 299]
    qb = [0, 1, 150, 299]
    (dq, dk, dv), ref, terms = run_case(w, q_blocks=qb, kv_blocks=kv)
    rows_q, rows_k = _rows(qb, 64, w.n), _rows(kv, 64, w.n)
    check_bound(dq, ref[0], terms[0], rows=rows_q, tag="long dQ")
    check_bound(dk, ref[1], terms[1], rows=rows_k, tag="long dK")
    check_bound(dv, ref[2], terms[2], rows=rows_k, tag="long dV")


def test_backward_deterministic_and_invariants_32k():
    # Full headline geometry: two runs are bitwise equal (fixed-order partial
    # sums), every gradient is finite, and the row-sum invariants hold: the
    # dK rows of a kv-head sum to ~0 and its dV rows to the sum of dO over
    # the group's q-heads.
    w = synth.WORKLOADS["qwen_n32768"]
    say("backward 32K determinism / invariants")
    q, k, v = synth.make_qkv(w, device="cuda")
    do = synth.make_grad_out(w, device="cuda")
    o, lse = bf1.attn_fwd(q, k, v, w.b, w.L)
    a = bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L)
    b = bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
        assert torch.isfinite(x).all()
    dq, dk, dv = a
    G = w.Hq // w.Hkv
    dsum = do.float().reshape(w.batch, w.Hkv, G, w.n, w.d).sum(dim=(2, 3))
    vsum = dv.sum(dim=2)
    assert (vsum - dsum).abs().max().item() <= 2e-2 * dsum.abs().max().item() + 1e-2
    ksum = dk.sum(dim=2)
    assert ksum.abs().max().item() <= 2e-3 * dk.abs().sum(dim=2).max().item()


def test_backward_32k_sampled_blocks():
    w = synth.WORKLOADS["qwen_n32768"]
    say("backward 32K sampled")
    NB = orc.num_blocks(w.n, w.b)
    q, k, v = synth.make_qkv(w)
    do = synth.make_grad_out(w)
    qf, kf, vf, dof = (synth.to_f64(t) for t in (q, k, v, do))
    qb = [0, 1, 17, 300, NB - 1]
    kv = [1, 100, 481, NB - 1]  # key block 0's 512 users are covered by the long-list case
    need = sorted(set(qb) | {int(j) for i in kv for j in orc.csr_transposed(w.n, w.b, w.L)[1][
        orc.csr_transposed(w.n, w.b, w.L)[0][i]:orc.csr_transposed(w.n, w.b, w.L)[0][i + 1]]})
    o_ref, lse_ref = orc.attn_gathered_fp64(qf, kf, vf, w.b, w.L, blocks=need)
    o_ref = np.nan_to_num(o_ref)
    lse_ref = np.nan_to_num(lse_ref)
    o_bf = torch.from_numpy(o_ref).to(torch.bfloat16)
    o_used = synth.to_f64(o_bf)
    dq, dk, dv = bf1.attn_bwd(q.cuda(), k.cuda(), v.cuda(), o_bf.cuda(), do.cuda(),
                              torch.from_numpy(lse_ref.astype(np.float32)).cuda(), w.b, w.L)
    torch.cuda.synchronize()
    ref = orc.attn_bwd_gathered_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used, q_blocks=qb, kv_blocks=kv)
    terms = list(zip(
        orc.attn_bwd_abs_terms_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used, q_blocks=qb, kv_blocks=kv),
        orc.attn_bwd_abs_terms_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used, q_blocks=qb, kv_blocks=kv,
                                    kind="pdp")))
    check_bound(dq, ref[0], terms[0], rows=_rows(qb, w.b, w.n), tag="32K dQ")
    check_bound(dk, ref[1], terms[1], rows=_rows(kv, w.b, w.n), tag="32K dK")
    check_bound(dv, ref[2], terms[2], rows=_rows(kv, w.b, w.n), tag="32K dV")


def test_backward_chained_from_gpu_forward():
    # GPU forward -> GPU backward.  The forward's O (within its own bar)
    # enters D = rowsum(dO * O); the result is compared with the exact
    # gradients at a tolerance of 2e-2 of each tensor's largest magnitude.
    w = synth.Workload("chain", 1, 1000, 4, 2, 128, 64, 2, seed=31)
    q, k, v = synth.make_qkv(w, device="cuda")
    do = synth.make_grad_out(w, device="cuda")
    o, lse = bf1.attn_fwd(q, k, v, w.b, w.L)
    dq, dk, dv = bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L)
    torch.cuda.synchronize()
    ref = orc.attn_bwd_gathered_fp64(*(synth.to_f64(t) for t in (q, k, v, do)), w.b, w.L)
    for name, got, r in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref):
        err = np.abs(got.cpu().double().numpy() - r).max()
        say(f"  chained {name}: max err {err:.3e} (max |ref| {np.abs(r).max():.3e})")
        assert err <= 2e-2 * np.abs(r).max(), name


def test_backward_peaked_rows_ragged_batch():
    # The partial-block / batching workload's structure at a small size: batch
    # 2, a ragged length, K scaled x3 on 5% of the positions (peaked softmax
    # rows, where recomputing P from the LSE is most sensitive).
    w = synth.Workload("bwd_peaked", 2, 1501, 4, 2, 128, 64, 2, seed=3, peak_frac=0.05, peak_mul=3.0)
    say("backward peaked rows, batch 2, n = 1501")
    (dq, dk, dv), ref, terms = run_case(w)
    for name, got, r, t in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref, terms):
        check_bound(got, r, t, tag=f"peaked {name}")


def test_backward_full_size_peaked_sampled():
    # The full n = 30001, batch 2 peaked workload: sampled blocks of both
    # batch elements, including the 49-token last block and key block 0.
    w = synth.WORKLOADS["qwen_n30001_b2_peaked"]
    say("backward n=30001 batch 2 peaked, sampled")
    NB = orc.num_blocks(w.n, w.b)
    q, k, v = synth.make_qkv(w)
    do = synth.make_grad_out(w)
    qf, kf, vf, dof = (synth.to_f64(t) for t in (q, k, v, do))
    qb = [0, 2, 250, NB - 1]
    kv = [3, 200, NB - 2, NB - 1]
    rp_t, ci_t = orc.csr_transposed(w.n, w.b, w.L)
    need = sorted(set(qb) | {int(j) for i in kv for j in ci_t[rp_t[i]:rp_t[i + 1]]})
    o_ref, lse_ref = orc.attn_gathered_fp64(qf, kf, vf, w.b, w.L, blocks=need)
    o_ref, lse_ref = np.nan_to_num(o_ref), np.nan_to_num(lse_ref)
    o_bf = torch.from_numpy(o_ref).to(torch.bfloat16)
    o_used = synth.to_f64(o_bf)
    dq, dk, dv = bf1.attn_bwd(q.cuda(), k.cuda(), v.cuda(), o_bf.cuda(), do.cuda(),
                              torch.from_numpy(lse_ref.astype(np.float32)).cuda(), w.b, w.L)
    torch.cuda.synchronize()
    ref = orc.attn_bwd_gathered_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used, q_blocks=qb, kv_blocks=kv)
    terms = list(zip(
        orc.attn_bwd_abs_terms_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used, q_blocks=qb, kv_blocks=kv),
        orc.attn_bwd_abs_terms_fp64(qf, kf, vf, dof, w.b, w.L, o=o_used, q_blocks=qb, kv_blocks=kv,
                                    kind="pdp")))
    check_bound(dq, ref[0], terms[0], rows=_rows(qb, w.b, w.n), tag="30001 dQ")
    check_bound(dk, ref[1], terms[1], rows=_rows(kv, w.b, w.n), tag="30001 dK")
    check_bound(dv, ref[2], terms[2], rows=_rows(kv, w.b, w.n), tag="30001 dV")


@pytest.mark.parametrize("cfg", [(2, 1000, 4, 2, 64, 2), (2, 1300, 8, 2, 128, 2), (1, 777, 4, 1, 64, 3)],
                         ids=lambda c: "x".join(map(str, c)))
def test_backward_ignores_workspace_contents(cfg):
    # Every workspace byte a kernel reads is written earlier in the same call
    # (D, LSE log2 e, the partial tiles and the dS units of every pair the dQ
    # kernel visits): a workspace filled with NaN bit patterns gives bitwise
    # the result of a zeroed one.
    batch, n, Hq, Hkv, B, L = cfg
    say(f"backward workspace contents {cfg}")
    w = synth.Workload("bwd_ws", batch, n, Hq, Hkv, 128, B, L, seed=1234 + n)
    q, k, v = synth.make_qkv(w, device="cuda")
    do = synth.make_grad_out(w, device="cuda")
    o, lse = bf1.attn_fwd(q, k, v, B, L)
    need = bf1.bwd_workspace_size(batch, n, Hq, Hkv, 128, B, L)
    outs = []
    for fill in (0x00, 0xFF):
        ws = torch.full((need,), fill, dtype=torch.uint8, device="cuda")
        outs.append(bf1.attn_bwd(q, k, v, o, do, lse, B, L, workspace=ws))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.isfinite(a).all()
        assert torch.equal(a, b)
