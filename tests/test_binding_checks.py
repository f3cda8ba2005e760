"""Tensor checks of the Python binding that need no GPU: every caller buffer
must be a contiguous tensor of the exact shape and dtype on the operands'
device before its pointer reaches the library, and calls that cannot be
served raise ValueError instead of handing the kernels a bad address."""

import pytest
import torch

import paper_2608_20427_amd as bf1

CPU = torch.device("cpu")


def test_check_buffer_accepts_the_exact_buffer():
    t = torch.zeros((2, 3, 5), dtype=torch.float32)
    assert bf1.check_buffer(t, "t", (2, 3, 5), torch.float32, CPU) is t


@pytest.mark.parametrize("bad,why", [
    (torch.zeros((2, 3, 5), dtype=torch.float16), "dtype"),
    (torch.zeros((2, 3, 6), dtype=torch.float32), "shape"),
    (torch.zeros((2, 3 * 5), dtype=torch.float32), "shape"),
    (torch.zeros((2, 5, 3), dtype=torch.float32).transpose(1, 2), "contiguous"),
    (torch.zeros((2, 3, 5), dtype=torch.float32, device="meta"), "device"),
    ([0.0] * 30, "tensor"),
])
def test_check_buffer_rejects(bad, why):
    with pytest.raises(ValueError, match=why):
        bf1.check_buffer(bad, "t", (2, 3, 5), torch.float32, CPU)


def test_check_workspace_counts_bytes_not_elements():
    ws = torch.zeros(100, dtype=torch.float32)         # 400 bytes
    assert bf1.check_workspace(ws, "ws", 400, CPU) == 400
    with pytest.raises(ValueError, match="bytes"):
        bf1.check_workspace(ws, "ws", 401, CPU)
    with pytest.raises(ValueError, match="device"):
        bf1.check_workspace(torch.zeros(1000, dtype=torch.uint8, device="meta"), "ws", 10, CPU)
    with pytest.raises(ValueError, match="contiguous"):
        bf1.check_workspace(torch.zeros((40, 40), dtype=torch.uint8).t(), "ws", 10, CPU)


def _qkv_cpu(n=64):
    q = torch.zeros((1, 2, n, 128), dtype=torch.bfloat16)
    k = torch.zeros((1, 1, n, 128), dtype=torch.bfloat16)
    return q, k, k.clone()


def test_host_operands_are_rejected():
    q, k, v = _qkv_cpu()
    for fn in (lambda: bf1.attn_fwd(q, k, v), lambda: bf1.dense_causal_fwd(q, k, v),
               lambda: bf1.attn_fwd_csr(q, k, v, 64, torch.zeros(2, dtype=torch.int32),
                                        torch.zeros(3, dtype=torch.int32))):
        with pytest.raises(ValueError, match="CUDA"):
            fn()


def test_backward_needs_forward_outputs():
    q, k, v = _qkv_cpu()
    do = torch.zeros_like(q)
    with pytest.raises(ValueError, match="o and lse"):
        bf1.attn_bwd(q, k, v, q.clone(), do, None)
    with pytest.raises(ValueError, match="o and lse"):
        bf1.attn_bwd(q, k, v, None, do, torch.zeros((1, 2, 64)))


def test_decode_host_operands_are_rejected():
    q = torch.zeros((1, 2, 128), dtype=torch.bfloat16)
    kp = torch.zeros((4, 1, 64, 128), dtype=torch.bfloat16)
    sl = torch.ones(1, dtype=torch.int32)
    plan = torch.zeros((1, 8), dtype=torch.int32)
    with pytest.raises(ValueError, match="CUDA"):
        bf1.attn_decode(q, kp, kp, sl, plan)
    with pytest.raises(ValueError, match="CUDA"):
        bf1.decode_plan(sl, torch.zeros((1, 4), dtype=torch.int32), 4, 8)
