"""GPU parity of the one-token decode over a paged cache (§3.2, §4.2, §5.4)
against the fp64 oracle.

Bars: decode plan rows bit-exact against the oracle's page lists; O max-abs
<= 2e-2, mean-abs <= 2e-3, LSE max-abs <= 1e-3 (the forward's bars: the
decode row is the forward's last row); page-permutation invariance,
decoy-page isolation and determinism bitwise.
"""

import sys

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu

O_MAX, O_MEAN, LSE_MAX = 2e-2, 2e-3, 1e-3


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


def compare(o, l, o_ref, l_ref, tag, rows=None):
    og = o.float().cpu().double().numpy()
    lg = l.cpu().double().numpy()
    if rows is not None:
        og, lg, o_ref, l_ref = og[rows], lg[rows], o_ref[rows], l_ref[rows]
    assert np.isfinite(og).all() and np.isfinite(lg).all(), tag
    err, lerr = np.abs(og - o_ref), np.abs(lg - l_ref)
    say(f"  [{tag}] O max {err.max():.3e} mean {err.mean():.3e} | LSE max {lerr.max():.3e}")
    assert err.max() <= O_MAX and err.mean() <= O_MEAN and lerr.max() <= LSE_MAX, tag


def setup_case(w, seq_lens, spare=3, decoy=float("nan"), dense=False, page_seed=None):
    q, k, v, sl = synth.make_decode_host(w, seq_lens)
    kp, vp, table, num_pages = synth.page_cache(k, v, sl, w.b, w.seed if page_seed is None else page_seed,
                                                spare_pages=spare, decoy=decoy)
    stride = bf1.decode_plan_stride(int(max(sl)), w.b, w.L, dense)
    dev = dict(q=q.cuda(), kp=kp.cuda(), vp=vp.cuda(), sl=torch.from_numpy(sl).cuda(),
               table=table.cuda(), num_pages=num_pages, stride=stride)
    return (q, k, v, sl, table), dev


def run_decode(w, dev, dense=False, plan=None):
    if plan is None:
        plan = bf1.decode_plan(dev["sl"], dev["table"], dev["num_pages"], dev["stride"], w.b, w.L, dense)
    o, l = bf1.attn_decode(dev["q"], dev["kp"], dev["vp"], dev["sl"], plan, w.b)
    torch.cuda.synchronize()
    return o, l, plan


# ---------------------------------------------------------------------------
# Plan: bit-exact
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("B,L,dense", [(64, 2, False), (128, 2, False), (64, 1, False), (64, 5, False),
                                       (64, 2, True)])
def test_decode_plan_bit_exact(B, L, dense):
    rng = np.random.default_rng(B + L + dense)
    batch, max_pages = 40, 300
    num_pages = batch * max_pages
    sl = rng.integers(1, max_pages * B + 1, size=batch).astype(np.int32)
    sl[:4] = [1, B, B + 1, max_pages * B]
    table = rng.permutation(num_pages).astype(np.int32).reshape(batch, max_pages)
    stride = bf1.decode_plan_stride(max_pages * B, B, L, dense)
    plan = bf1.decode_plan(torch.from_numpy(sl).cuda(), torch.from_numpy(table).cuda(), num_pages, stride,
                           B, L, dense).cpu().numpy()
    for beta in range(batch):
        j, earlier = orc.decode_plan(int(sl[beta]), table[beta], B, L, dense)
        assert plan[beta, 0] == j and plan[beta, 1] == len(earlier), beta
        assert plan[beta, 2:2 + len(earlier)].tolist() == earlier, beta
        assert plan[beta, 2 + len(earlier)] == table[beta, j], beta


def test_decode_plan_marks_unplannable_rows():
    B, L = 64, 2
    sl = np.array([0, 65, 64 * 10 + 1, 200, 130], dtype=np.int32)
    table = np.arange(5 * 10, dtype=np.int32).reshape(5, 10)
    table[3, 0] = 999          # a page outside the pool (block 0 is selected by row 3)
    table[4, 2] = -1           # the self page of row 4 is missing
    stride = bf1.decode_plan_stride(640, B, L)
    plan = bf1.decode_plan(torch.from_numpy(sl).cuda(), torch.from_numpy(table).cuda(), 50, stride, B,
                           L).cpu().numpy()
    assert plan[:, 0].tolist() == [-1, 1, -1, -1, -1]
    assert plan[1, 1] == 1 and plan[1, 2] == table[1, 0] and plan[1, 3] == table[1, 1]


# ---------------------------------------------------------------------------
# Attention parity: small shapes, full oracle
# ---------------------------------------------------------------------------

SMALL = [
    # batch, Hq, Hkv, d, B, L, seq_lens
    (4, 4, 2, 128, 64, 2, [1, 64, 65, 1000]),
    (3, 16, 8, 128, 64, 2, [2048, 4096, 3001]),
    (2, 2, 1, 64, 64, 1, [777, 130]),
    (2, 8, 1, 128, 64, 2, [640, 129]),
    (3, 3, 3, 128, 64, 2, [700, 1, 64]),
    (2, 4, 1, 64, 128, 3, [900, 1500]),
    (2, 4, 2, 128, 128, 2, [1500, 128]),
    (1, 2, 1, 128, 64, 0, [330]),
]


@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: "x".join(map(str, c[:6])))
def test_decode_small_full_oracle(cfg):
    batch, Hq, Hkv, d, B, L, lens = cfg
    w = synth.DecodeWorkload("dec", batch, max(lens), Hq, Hkv, d, B, L, seed=500 + sum(lens))
    say(f"decode small {cfg}")
    (q, k, v, sl, _), dev = setup_case(w, np.array(lens, dtype=np.int32))
    o, l, _ = run_decode(w, dev)
    o_ref, l_ref = orc.attn_decode_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), sl, B, L)
    compare(o, l, o_ref, l_ref, str(cfg))


# Larger batches: more (sequence, kv-head) pairs than pages per list, so
# several pages share a split and the merge folds fewer records.
SPLIT = [
    # batch, Hq, Hkv, d, B, L, seq_lens: 320 / 288 (sequence, kv-head) pairs,
    # so a split holds 3 / 2 pages of each list (about 1024 workgroups)
    (40, 16, 8, 128, 64, 2, [1, 64, 65, 1000, 2048, 3001, 777, 130, 4096, 5] * 4),
    (36, 16, 8, 64, 128, 1, [1, 128, 129, 900, 1500, 60, 3000, 2048, 255, 256, 257, 1024] * 3),
]


@pytest.mark.parametrize("cfg", SPLIT, ids=lambda c: "x".join(map(str, c[:6])))
def test_decode_split_path_full_oracle(cfg):
    batch, Hq, Hkv, d, B, L, lens = cfg
    w = synth.DecodeWorkload("dec", batch, max(lens), Hq, Hkv, d, B, L, seed=700 + batch)
    say(f"decode split path {cfg[:6]}")
    (q, k, v, sl, _), dev = setup_case(w, np.array(lens, dtype=np.int32))
    o, l, _ = run_decode(w, dev)
    o_ref, l_ref = orc.attn_decode_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), sl, B, L)
    compare(o, l, o_ref, l_ref, "split " + str(cfg[:6]))


def test_decode_dense_plan_is_dense_causal():
    w = synth.DecodeWorkload("dec", 3, 2000, 4, 2, 128, 64, 2, seed=77)
    lens = np.array([2000, 65, 1], dtype=np.int32)
    (q, k, v, sl, _), dev = setup_case(w, lens, dense=True)
    dev["stride"] = bf1.decode_plan_stride(2000, 64, 2, dense=True)
    o, l, _ = run_decode(w, dev, dense=True)
    # dense causal row t: the oracle's decode over a route that covers every block
    o_ref, l_ref = orc.attn_decode_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), sl, 64,
                                        L=int(max(lens)) // 64 + 2)
    compare(o, l, o_ref, l_ref, "dense")


def test_decode_matches_gpu_forward_last_row():
    # the decode row is the prefill forward's row t (both on the GPU)
    w = synth.Workload("fw", 1, 3000, 4, 2, 128, 64, 2, seed=21)
    q, k, v = synth.make_qkv(w, device="cuda")
    of, lf = bf1.attn_fwd(q, k, v, B=64, L=2)
    torch.cuda.synchronize()
    for n in (3000, 2049, 64, 1):
        sl = np.array([n], dtype=np.int32)
        kp, vp, table, num_pages = synth.page_cache(k[:, :, :n].cpu(), v[:, :, :n].cpu(), sl, 64, seed=n)
        stride = bf1.decode_plan_stride(n, 64, 2)
        plan = bf1.decode_plan(torch.from_numpy(sl).cuda(), table.cuda(), num_pages, stride, 64, 2)
        qd = q[:, :, n - 1].contiguous()
        o, l = bf1.attn_decode(qd, kp.cuda(), vp.cuda(), torch.from_numpy(sl).cuda(), plan, 64)
        torch.cuda.synchronize()
        err = (o.float() - of[:, :, n - 1].float()).abs().max().item()
        lerr = (l - lf[:, :, n - 1]).abs().max().item()
        say(f"  n={n}: decode vs forward row O {err:.3e} LSE {lerr:.3e}")
        assert err <= 2 * O_MAX and lerr <= 2 * LSE_MAX


# ---------------------------------------------------------------------------
# Paging properties
# ---------------------------------------------------------------------------

def test_page_permutation_invariance_and_decoys():
    w = synth.DecodeWorkload("dec", 3, 3000, 4, 2, 128, 64, 2, seed=88)
    lens = np.array([3000, 1700, 65], dtype=np.int32)
    _, dev1 = setup_case(w, lens, page_seed=1, decoy=float("nan"))
    _, dev2 = setup_case(w, lens, page_seed=2, decoy=1e4, spare=17)
    o1, l1, _ = run_decode(w, dev1)
    o2, l2, _ = run_decode(w, dev2)
    assert torch.isfinite(o1).all() and torch.isfinite(l1).all()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_persistent_plan_across_the_epoch_and_stale_detection():
    w = synth.DecodeWorkload("dec", 2, 1024 + 64, 4, 2, 128, 64, 2, seed=91)
    full = np.array([1024 + 64, 768], dtype=np.int32)      # tokens held by each cache
    q, k, v, _ = synth.make_decode_host(w, full)
    kp, vp, table, num_pages = synth.page_cache(k, v, full, 64, seed=3)
    kp, vp, table = kp.cuda(), vp.cuda(), table.cuda()
    stride = bf1.decode_plan_stride(int(full.max()), 64, 2)
    start = np.array([1024 + 1, 641], dtype=np.int32)     # first token of blocks 16 and 10
    plan = bf1.decode_plan(torch.from_numpy(start).cuda(), table, num_pages, stride, 64, 2)
    qf, kf, vf = synth.to_f64(q), synth.to_f64(k), synth.to_f64(v)
    for step in (0, 1, 31, 59):
        sl = start + step
        o, l = bf1.attn_decode(q.cuda(), kp, vp, torch.from_numpy(sl).cuda(), plan, 64)
        torch.cuda.synchronize()
        o_ref, l_ref = orc.attn_decode_fp64(qf, kf, vf, sl, 64, 2)
        compare(o, l, o_ref, l_ref, f"step {step}")
    # sequence 1 crosses into block 11 at length 705; sequence 0 stays in block 16
    sl = np.array([1024 + 64, 705], dtype=np.int32)
    o, l = bf1.attn_decode(q.cuda(), kp, vp, torch.from_numpy(sl).cuda(), plan, 64)
    torch.cuda.synchronize()
    assert torch.isnan(o[1].float()).all() and torch.isnan(l[1]).all()
    o_ref, l_ref = orc.attn_decode_fp64(qf, kf, vf, sl, 64, 2)
    compare(o, l, o_ref, l_ref, "stale row isolated", rows=[0])
    # re-planning fixes it
    plan = bf1.decode_plan(torch.from_numpy(sl).cuda(), table, num_pages, stride, 64, 2)
    o, l = bf1.attn_decode(q.cuda(), kp, vp, torch.from_numpy(sl).cuda(), plan, 64)
    torch.cuda.synchronize()
    compare(o, l, o_ref, l_ref, "replanned")


def test_decode_deterministic_and_plan_unchanged():
    w = synth.DecodeWorkload("dec", 2, 4096, 16, 8, 128, 64, 2, seed=93)
    _, dev = setup_case(w, np.array([4096, 2500], dtype=np.int32))
    o1, l1, plan = run_decode(w, dev)
    before = plan.clone()
    for _ in range(3):
        o2, l2, _ = run_decode(w, dev, plan=plan)
        assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert torch.equal(plan, before)


# ---------------------------------------------------------------------------
# Full size (the timed configurations), oracle on sampled sequences
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["decode_n32768_batch8", "decode_n65536_batch1", "decode_n32768_batch32"])
def test_decode_full_size_sampled(name):
    w = synth.DECODE_WORKLOADS[name]
    say(f"decode full size {name}")
    q, kp, vp, sl, table, num_pages = synth.make_decode_device(w)
    stride = bf1.decode_plan_stride(w.ctx, w.b, w.L)
    plan = bf1.decode_plan(sl, table, num_pages, stride, w.b, w.L)
    o, l = bf1.attn_decode(q, kp, vp, sl, plan, w.b)
    torch.cuda.synchronize()
    for beta in sorted({0, w.batch - 1}):
        n = int(sl[beta])
        pages = table[beta, : -(-n // w.b)].long()
        kl = kp[pages].permute(1, 0, 2, 3).reshape(w.Hkv, -1, w.d)[:, :n][None]
        vl = vp[pages].permute(1, 0, 2, 3).reshape(w.Hkv, -1, w.d)[:, :n][None]
        o_ref, l_ref = orc.attn_decode_fp64(synth.to_f64(q[beta:beta + 1]), synth.to_f64(kl), synth.to_f64(vl),
                                            [n], w.b, w.L)
        compare(o[beta:beta + 1], l[beta:beta + 1], o_ref, l_ref, f"{name} seq {beta}")


def test_decode_workspace_too_small_and_lse_optional():
    w = synth.DecodeWorkload("dec", 2, 2000, 4, 2, 128, 64, 2, seed=95)
    _, dev = setup_case(w, np.array([2000, 1000], dtype=np.int32))
    plan = bf1.decode_plan(dev["sl"], dev["table"], dev["num_pages"], dev["stride"], 64, 2)
    need = bf1.decode_workspace_size(2, 4, 2, 128, dev["stride"])
    ws = torch.empty(need - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):     # the binding refuses it before the library
        bf1.attn_decode(dev["q"], dev["kp"], dev["vp"], dev["sl"], plan, 64, workspace=ws)
    lib = bf1.load()
    o0 = torch.empty_like(dev["q"])
    st = lib.bf1_decode_attn(bf1._ptr(dev["q"]), bf1._ptr(dev["kp"]), bf1._ptr(dev["vp"]), bf1._ptr(dev["sl"]),
                             dev["num_pages"], bf1._ptr(plan), dev["stride"], bf1._ptr(o0), None, 2, 4, 2, 128,
                             64, bf1._ptr(ws), need - 256, bf1._stream(None))
    assert st == bf1.BF1_ERR_BUFFER_TOO_SMALL   # ... and so does the C ABI
    o1, l1, _ = run_decode(w, dev, plan=plan)
    o2 = torch.empty_like(o1)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    st = lib.bf1_decode_attn(bf1._ptr(dev["q"]), bf1._ptr(dev["kp"]), bf1._ptr(dev["vp"]), bf1._ptr(dev["sl"]),
                             dev["num_pages"], bf1._ptr(plan), dev["stride"], bf1._ptr(o2), None, 2, 4, 2, 128,
                             64, bf1._ptr(ws), need, bf1._stream(None))
    torch.cuda.synchronize()
    assert st == bf1.BF1_OK and torch.equal(o1, o2)


def test_decode_step_replays_in_a_graph():
    # the plan and the step captured in one HIP graph; every replay, with eager
    # work and synchronisations between them, equals the eager result
    w = synth.DecodeWorkload("dec", 4, 3000, 16, 8, 128, 64, 2, seed=97)
    _, dev = setup_case(w, np.array([3000, 1025, 64, 2222], dtype=np.int32))
    o_e, l_e, plan = run_decode(w, dev)
    need = bf1.decode_workspace_size(w.batch, w.Hq, w.Hkv, w.d, dev["stride"])
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    o = torch.empty_like(o_e)
    l = torch.empty_like(l_e)

    def step():
        bf1.decode_plan(dev["sl"], dev["table"], dev["num_pages"], dev["stride"], w.b, w.L, plan=plan)
        bf1.attn_decode(dev["q"], dev["kp"], dev["vp"], dev["sl"], plan, w.b, out=o, lse=l, workspace=ws)

    step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        o.zero_()
        l.zero_()
        plan.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, o_e) and torch.equal(l, l_e), r
        junk = torch.randn(1 << 20, device="cuda").sum()    # eager work between replays
        torch.cuda.synchronize()
        assert torch.isfinite(junk)


def test_decode_ignores_workspace_contents():
    # The merge reads only the records its split kernel wrote in the same call:
    # a workspace filled with NaN bit patterns gives bitwise the result of a
    # zeroed one (batch 40: several pages per split, so the merge runs).
    batch, Hq, Hkv, d, B, L, lens = SPLIT[0]
    w = synth.DecodeWorkload("dec", batch, max(lens), Hq, Hkv, d, B, L, seed=811)
    say("decode workspace contents")
    _, dev = setup_case(w, np.array(lens, dtype=np.int32))
    plan = bf1.decode_plan(dev["sl"], dev["table"], dev["num_pages"], dev["stride"], w.b, w.L)
    need = bf1.decode_workspace_size(w.batch, w.Hq, w.Hkv, w.d, dev["stride"])
    outs = []
    for fill in (0x00, 0xFF):
        ws = torch.full((need,), fill, dtype=torch.uint8, device="cuda")
        outs.append(bf1.attn_decode(dev["q"], dev["kp"], dev["vp"], dev["sl"], plan, w.b, workspace=ws))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.isfinite(a.float()).all()
        assert torch.equal(a, b)
