"""The forward that allocates nothing (bf1_attn_fwd_noalloc), called through
the C ABI: its route table lives in the library's fixed scratch array, so
its output must equal bf1_attn_fwd's bitwise (same planner, same kernel),
and, like it, the fp64 oracle within the forward's bars.  Two calls in a row,
the second on a smaller input, so the second runs over the first one's
leftover table."""

import ctypes

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()
    yield
    torch.cuda.synchronize()


def _noalloc(lib, q, k, v, o, lse, B, L):
    batch, Hq, n, d = q.shape
    return lib.bf1_attn_fwd_noalloc(bf1._ptr(q), bf1._ptr(k), bf1._ptr(v), bf1._ptr(o), bf1._ptr(lse),
                                    batch, n, Hq, k.shape[1], d, B, L, bf1._stream(None))


@pytest.mark.parametrize("first,second", [
    ((1, 32768, 16, 8, 128, 64, 2), (2, 1000, 4, 2, 128, 64, 2)),
    ((2, 3001, 4, 1, 64, 128, 3), (1, 333, 2, 1, 64, 64, 1)),
])
def test_noalloc_matches_cached_plan_forward(first, second):
    lib = bf1.load()
    cases = []
    for cfg in (first, second):
        w = synth.Workload("noalloc", *cfg, seed=61 + cfg[1])
        q, k, v = synth.make_qkv(w, device="cuda")
        o = torch.empty_like(q)
        lse = torch.empty((w.batch, w.Hq, w.n), dtype=torch.float32, device="cuda")
        cases.append((w, q, k, v, o, lse))
    # both no-allocation calls back to back on one stream, the smaller second
    for w, q, k, v, o, lse in cases:
        o.fill_(float("nan"))
        lse.fill_(float("nan"))
    for w, q, k, v, o, lse in cases:
        assert _noalloc(lib, q, k, v, o, lse, w.b, w.L) == bf1.BF1_OK
    torch.cuda.synchronize()
    for w, q, k, v, o, lse in cases:
        o_ref, l_ref = bf1.attn_fwd(q, k, v, B=w.b, L=w.L)
        torch.cuda.synchronize()
        assert torch.equal(o, o_ref) and torch.equal(lse, l_ref), w
    # the small one against the oracle as well
    w, q, k, v, o, lse = cases[1]
    o64, l64 = orc.attn_gathered_fp64(synth.to_f64(q), synth.to_f64(k), synth.to_f64(v), w.b, w.L)
    err = np.abs(o.float().cpu().double().numpy() - o64)
    lerr = np.abs(lse.cpu().double().numpy() - l64)
    assert err.max() <= 2e-2 and err.mean() <= 2e-3 and lerr.max() <= 1e-3


def test_noalloc_binding_and_limit():
    w = synth.Workload("noalloc", 1, 700, 4, 2, 128, 64, 2, seed=62)
    q, k, v = synth.make_qkv(w, device="cuda")
    o = torch.empty_like(q)
    bf1.attn_fwd_noalloc(q, k, v, o, None, 64, 2)      # LSE not written
    o_ref, _ = bf1.attn_fwd(q, k, v, B=64, L=2)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref)
    # a route table larger than the scratch array is refused before any work
    lib = bf1.load()
    fake = ctypes.c_void_p(1 << 20)
    n_big = 1 << 23                                     # NB = 131072 blocks at B = 64
    nb, nnz, _ = bf1.plan_size(n_big, 64, 2)
    assert nb + 1 + nnz > 1 << 20
    st = lib.bf1_attn_fwd_noalloc(fake, fake, fake, fake, None, 1, n_big, 2, 1, 128, 64, 2, None)
    assert st == bf1.BF1_ERR_BUFFER_TOO_SMALL
