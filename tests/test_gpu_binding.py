"""Binding checks with real device operands: every caller buffer that is on
the host, of another shape or dtype, or not contiguous is refused with
ValueError before the library is called (nothing is launched)."""

import pytest
import torch

import paper_2608_20427_amd as bf1

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()


def _qkv(n=200, Hq=4, Hkv=2, d=128):
    g = torch.Generator(device="cpu").manual_seed(5)
    mk = lambda h: torch.randn((1, h, n, d), generator=g).to(torch.bfloat16).cuda()
    return mk(Hq), mk(Hkv), mk(Hkv)


def _bad_like(t):
    """Host copy, wrong shape, wrong dtype, non-contiguous view."""
    wrong_shape = torch.empty(t.shape[:-1] + (t.shape[-1] + 1,), dtype=t.dtype, device=t.device)
    wrong_dtype = torch.empty(t.shape, dtype=torch.float16 if t.dtype != torch.float16 else torch.float32,
                              device=t.device)
    strided = torch.empty(t.shape[:-1] + (2 * t.shape[-1],), dtype=t.dtype, device=t.device)[..., ::2]
    return [t.cpu(), wrong_shape, wrong_dtype, strided]


def test_forward_output_buffers():
    q, k, v = _qkv()
    o, lse = bf1.attn_fwd(q, k, v)
    for bad in _bad_like(o):
        with pytest.raises(ValueError):
            bf1.attn_fwd(q, k, v, out=bad)
        with pytest.raises(ValueError):
            bf1.dense_causal_fwd(q, k, v, out=bad)
    for bad in _bad_like(lse):
        with pytest.raises(ValueError):
            bf1.attn_fwd(q, k, v, lse=bad)
    for bad in _bad_like(k):
        with pytest.raises(ValueError):
            bf1.attn_fwd(q, bad, v)
        with pytest.raises(ValueError):
            bf1.attn_fwd(q, k, bad)


def test_csr_tables():
    q, k, v = _qkv()
    rp, ci = bf1.plan(200, 64, 2)
    with pytest.raises(ValueError):
        bf1.attn_fwd_csr(q, k, v, 64, rp.cpu(), ci)
    with pytest.raises(ValueError):
        bf1.attn_fwd_csr(q, k, v, 64, rp, ci.cpu())
    with pytest.raises(ValueError):
        bf1.attn_fwd_csr(q, k, v, 64, rp[:-1].contiguous(), ci)   # row_ptr needs NB + 1 entries
    with pytest.raises(ValueError):
        bf1.attn_fwd_csr(q, k, v, 64, rp.long(), ci)
    with pytest.raises(ValueError):
        bf1.plan(200, 64, 2, row_ptr=rp.cpu())


def test_backward_buffers():
    q, k, v = _qkv()
    o, lse = bf1.attn_fwd(q, k, v)
    do = torch.randn(q.shape, generator=torch.Generator().manual_seed(1)).to(torch.bfloat16).cuda()
    dq, dk, dv = bf1.attn_bwd(q, k, v, o, do, lse)
    for bad in _bad_like(do):
        with pytest.raises(ValueError):
            bf1.attn_bwd(q, k, v, o, bad, lse)
    for name, ref in (("dq", dq), ("dk", dk), ("dv", dv)):
        for bad in _bad_like(ref):
            with pytest.raises(ValueError):
                bf1.attn_bwd(q, k, v, o, do, lse, **{name: bad})
    need = bf1.bwd_workspace_size(1, 200, 4, 2, 128, 64, 2)
    with pytest.raises(ValueError):
        bf1.attn_bwd(q, k, v, o, do, lse, workspace=torch.empty(need - 1, dtype=torch.uint8, device="cuda"))
    with pytest.raises(ValueError):
        bf1.attn_bwd(q, k, v, o, do, lse, workspace=torch.empty(need, dtype=torch.uint8))
    # a float workspace is sized in bytes, not elements
    ws = torch.empty((need + 3) // 4, dtype=torch.float32, device="cuda")
    dq2, dk2, dv2 = bf1.attn_bwd(q, k, v, o, do, lse, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq2) and torch.equal(dk, dk2) and torch.equal(dv, dv2)


def test_decode_buffers():
    g = torch.Generator().manual_seed(3)
    B, Hq, Hkv, d, pages = 64, 4, 2, 128, 6
    q = torch.randn((1, Hq, d), generator=g).to(torch.bfloat16).cuda()
    kp = torch.randn((pages, Hkv, B, d), generator=g).to(torch.bfloat16).cuda()
    vp = torch.randn((pages, Hkv, B, d), generator=g).to(torch.bfloat16).cuda()
    sl = torch.tensor([300], dtype=torch.int32, device="cuda")
    table = torch.arange(pages, dtype=torch.int32, device="cuda").view(1, pages)
    stride = bf1.decode_plan_stride(6 * B, B, 2)
    plan = bf1.decode_plan(sl, table, pages, stride, B, 2)
    o, lse = bf1.attn_decode(q, kp, vp, sl, plan, B)
    for bad in _bad_like(o):
        with pytest.raises(ValueError):
            bf1.attn_decode(q, kp, vp, sl, plan, B, out=bad)
    for bad in _bad_like(lse):
        with pytest.raises(ValueError):
            bf1.attn_decode(q, kp, vp, sl, plan, B, lse=bad)
    with pytest.raises(ValueError):
        bf1.attn_decode(q, kp, vp, sl, plan, B, workspace=torch.empty(8, dtype=torch.uint8, device="cuda"))
    with pytest.raises(ValueError):
        bf1.attn_decode(q, kp, vp, sl.cpu(), plan, B)
    with pytest.raises(ValueError):
        bf1.decode_plan(sl, table, pages, stride, B, 2, plan=plan.cpu())
    with pytest.raises(ValueError):
        bf1.decode_plan(sl, table.cpu(), pages, stride, B, 2)
    torch.cuda.synchronize()
