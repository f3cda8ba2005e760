"""BF1 causal dyadic block-sparse attention (prefill forward and backward) for MI355X.

Thin ctypes binding over libbf1.so (declared in include/bf1.h).  Every
function here only checks tensor metadata and marshals pointers, sizes and
the current HIP stream; every step of the computation runs in the library's
HIP kernels.  There is no fallback: if the library is not built, or a call
fails, an exception is raised.

Layouts: Q, O [batch, Hq, n, d] bf16; K, V [batch, Hkv, n, d] bf16;
LSE [batch, Hq, n] float32 (natural log).  q-head h reads kv-head
h // (Hq // Hkv).  Block width ``B`` (tokens per block) and local width
``L`` (blocks) define the route of the paper's §3.1, Eq. 1.
"""

import ctypes
import os

__all__ = [
    "BF1Error", "lib_path", "load", "version", "status_string", "plan_size", "plan",
    "attn_fwd", "attn_fwd_csr", "dense_causal_fwd", "release_plans", "selected_flops",
    "plan_transposed", "bwd_workspace_size", "attn_bwd", "selected_bwd_flops", "attn_fwd_noalloc",
    "set_forward_key_split",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

BF1_OK = 0
BF1_ERR_INVALID_ARG = -1
BF1_ERR_UNSUPPORTED = -2
BF1_ERR_BUFFER_TOO_SMALL = -3
BF1_ERR_HIP = -4
BF1_ERR_NOMEM = -5
BF1_ERR_CAPTURE = -6


class BF1Error(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


def lib_path():
    return os.path.join(_HERE, "libbf1.so")


def load():
    """Load libbf1.so (built in-tree by __graft_entry__.build()).  Raises if
    it is missing: there is no other implementation to fall back to."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2608_20427_amd.build`")
    lib = ctypes.CDLL(path)
    i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    lib.bf1_version.restype = ctypes.c_int
    lib.bf1_version.argtypes = []
    lib.bf1_status_string.restype = ctypes.c_char_p
    lib.bf1_status_string.argtypes = [ctypes.c_int]
    lib.bf1_plan_size.restype = ctypes.c_int
    lib.bf1_plan_size.argtypes = [i64, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i64),
                                  ctypes.POINTER(i64)]
    lib.bf1_plan.restype = ctypes.c_int
    lib.bf1_plan.argtypes = [i64, i32, i32, vp, vp, i64, vp]
    attn = [vp, vp, vp, vp, vp, i32, i64, i32, i32, i32]
    lib.bf1_attn_fwd.restype = ctypes.c_int
    lib.bf1_attn_fwd.argtypes = attn + [i32, i32, vp]
    lib.bf1_attn_fwd_noalloc.restype = ctypes.c_int
    lib.bf1_attn_fwd_noalloc.argtypes = attn + [i32, i32, vp]
    lib.bf1_attn_fwd_csr.restype = ctypes.c_int
    lib.bf1_attn_fwd_csr.argtypes = attn + [i32, vp, vp, i64, vp]
    lib.bf1_dense_causal_fwd.restype = ctypes.c_int
    lib.bf1_dense_causal_fwd.argtypes = attn + [vp]
    lib.bf1_set_forward_key_split.restype = ctypes.c_int
    lib.bf1_set_forward_key_split.argtypes = [i32]
    lib.bf1_release_plans.restype = None
    lib.bf1_release_plans.argtypes = []
    lib.bf1_plan_transposed.restype = ctypes.c_int
    lib.bf1_plan_transposed.argtypes = [i64, i32, i32, vp, vp, i64]
    lib.bf1_attn_bwd_workspace_size.restype = ctypes.c_int
    lib.bf1_attn_bwd_workspace_size.argtypes = [i32, i64, i32, i32, i32, i32, i32,
                                                ctypes.POINTER(i64)]
    lib.bf1_attn_bwd.restype = ctypes.c_int
    lib.bf1_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, i64, i32, i32, i32,
                                 i32, i32, vp, i64, vp]
    lib.bf1_plan_variant.restype = ctypes.c_int
    lib.bf1_plan_variant.argtypes = [i32, i64, i32, i32, ctypes.c_uint64, vp, vp, i64]
    lib.bf1_route_depth.restype = ctypes.c_int
    lib.bf1_route_depth.argtypes = [vp, vp, i32, ctypes.POINTER(i32)]
    lib.bf1_decode_plan_stride.restype = ctypes.c_int
    lib.bf1_decode_plan_stride.argtypes = [i64, i32, i32, i32, ctypes.POINTER(i32)]
    lib.bf1_decode_plan.restype = ctypes.c_int
    lib.bf1_decode_plan.argtypes = [i32, vp, vp, i32, i32, i32, i32, i32, vp, i32, vp]
    lib.bf1_decode_workspace_size.restype = ctypes.c_int
    lib.bf1_decode_workspace_size.argtypes = [i32, i32, i32, i32, i32, ctypes.POINTER(i64)]
    lib.bf1_decode_attn.restype = ctypes.c_int
    lib.bf1_decode_attn.argtypes = [vp, vp, vp, vp, i32, vp, i32, vp, vp, i32, i32, i32, i32, i32, vp,
                                    i64, vp]
    _LIB = lib
    return lib


def _check(status, where):
    if status != BF1_OK:
        raise BF1Error(status, where)


def version():
    return load().bf1_version()


def status_string(status):
    return load().bf1_status_string(int(status)).decode()


def plan_size(n, B=64, L=2):
    """(num_blocks, nnz, selected pairs per (batch, head)) in closed form."""
    nb, nnz, pairs = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_int64()
    _check(load().bf1_plan_size(int(n), int(B), int(L), ctypes.byref(nb), ctypes.byref(nnz),
                                ctypes.byref(pairs)), "bf1_plan_size")
    return nb.value, nnz.value, pairs.value


def selected_flops(batch, n, Hq, d, B=64, L=2):
    """Algorithmic flops of the forward: 4 d per selected pair (QK^T and PV),
    per q-head and batch element."""
    return 4 * d * plan_size(n, B, L)[2] * Hq * batch


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def check_buffer(t, name, shape, dtype, device):
    """Raise ValueError unless `t` is a contiguous tensor of exactly `shape`
    and `dtype` on `device`.  Every buffer handed to the library goes through
    this check before its pointer is taken: a host tensor, or one of another
    size, would otherwise become a kernel access outside the intended memory."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor, got {type(t).__name__}")
    if t.device != device:
        raise ValueError(f"{name} must be on device {device}, got {t.device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def check_workspace(t, name, nbytes, device):
    """Raise ValueError unless `t` is a contiguous tensor on `device` holding at
    least `nbytes` bytes; returns its size in bytes."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor, got {type(t).__name__}")
    if t.device != device:
        raise ValueError(f"{name} must be on device {device}, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, {nbytes} needed")
    return have


def _cuda_device(t, name):
    """The CUDA device of input `t` (ValueError if it is not a CUDA tensor)."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA tensor")
    return t.device


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def plan(n, B=64, L=2, row_ptr=None, col_idx=None, stream=None):
    """Route table of Eq. 1 as device CSR (int32 row_ptr[NB+1], col_idx[nnz])."""
    import torch
    nb, nnz, _ = plan_size(n, B, L)
    dev = torch.device("cuda", torch.cuda.current_device())
    if row_ptr is None:
        row_ptr = torch.empty(nb + 1, dtype=torch.int32, device=dev)
    if col_idx is None:
        col_idx = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    check_buffer(row_ptr, "row_ptr", (nb + 1,), torch.int32, dev)
    if col_idx.dim() != 1:
        raise ValueError("col_idx must be 1-D")
    check_buffer(col_idx, "col_idx", col_idx.shape, torch.int32, dev)
    _check(load().bf1_plan(int(n), int(B), int(L), _ptr(row_ptr), _ptr(col_idx),
                           col_idx.numel(), _stream(stream)), "bf1_plan")
    return row_ptr, col_idx[:nnz]


def _prep(q, k, v, out, lse, want_lse):
    """Check the attention operands and the caller's output buffers (or
    allocate them) on q's device; returns (out, lse, sizes)."""
    import torch
    dev = _cuda_device(q, "q")
    if q.dim() != 4:
        raise ValueError("q must be 4-D [batch, Hq, n, d]")
    batch, Hq, n, d = q.shape
    check_buffer(q, "q", q.shape, torch.bfloat16, dev)
    if not isinstance(k, torch.Tensor) or k.dim() != 4:
        raise ValueError("k must be a 4-D tensor [batch, Hkv, n, d]")
    Hkv = k.shape[1]
    check_buffer(k, "k", (batch, Hkv, n, d), torch.bfloat16, dev)
    check_buffer(v, "v", (batch, Hkv, n, d), torch.bfloat16, dev)
    if out is None:
        out = torch.empty_like(q)
    check_buffer(out, "out", q.shape, torch.bfloat16, dev)
    if lse is None and want_lse:
        lse = torch.empty((batch, Hq, n), dtype=torch.float32, device=dev)
    if lse is not None:
        check_buffer(lse, "lse", (batch, Hq, n), torch.float32, dev)
    return out, lse, (batch, n, Hq, Hkv, d)


def attn_fwd(q, k, v, B=64, L=2, out=None, lse=None, want_lse=True, stream=None):
    """BF1 prefill forward; returns (O, LSE)."""
    import torch
    out, lse, (batch, n, Hq, Hkv, d) = _prep(q, k, v, out, lse, want_lse)
    with torch.cuda.device(q.device):
        _check(load().bf1_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), batch, n, Hq,
                                   Hkv, d, int(B), int(L), _stream(stream)), "bf1_attn_fwd")
    return out, lse


def attn_fwd_noalloc(q, k, v, out, lse=None, B=64, L=2, stream=None):
    """BF1 prefill forward that allocates no device memory (the route table
    goes to the library's fixed scratch array): the caller passes O (and
    optionally LSE); returns (O, LSE)."""
    import torch
    if out is None:
        raise ValueError("attn_fwd_noalloc writes into a caller-provided out")
    out, lse, (batch, n, Hq, Hkv, d) = _prep(q, k, v, out, lse, False)
    with torch.cuda.device(q.device):
        _check(load().bf1_attn_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), batch, n,
                                           Hq, Hkv, d, int(B), int(L), _stream(stream)),
               "bf1_attn_fwd_noalloc")
    return out, lse


def attn_fwd_csr(q, k, v, B, row_ptr, col_idx, out=None, lse=None, want_lse=True, stream=None):
    """Forward over a caller-supplied block route (CSR, int32 CUDA tensors)."""
    import torch
    out, lse, (batch, n, Hq, Hkv, d) = _prep(q, k, v, out, lse, want_lse)
    if int(B) < 1:
        raise ValueError("B must be positive")
    nb = -(-n // int(B))
    check_buffer(row_ptr, "row_ptr", (nb + 1,), torch.int32, q.device)
    if not isinstance(col_idx, torch.Tensor) or col_idx.dim() != 1:
        raise ValueError("col_idx must be a 1-D tensor")
    check_buffer(col_idx, "col_idx", col_idx.shape, torch.int32, q.device)
    with torch.cuda.device(q.device):
        _check(load().bf1_attn_fwd_csr(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), batch, n,
                                       Hq, Hkv, d, int(B), _ptr(row_ptr), _ptr(col_idx),
                                       col_idx.numel(), _stream(stream)), "bf1_attn_fwd_csr")
    return out, lse


def dense_causal_fwd(q, k, v, out=None, lse=None, want_lse=True, stream=None):
    """In-house dense causal attention built from the same kernel."""
    import torch
    out, lse, (batch, n, Hq, Hkv, d) = _prep(q, k, v, out, lse, want_lse)
    with torch.cuda.device(q.device):
        _check(load().bf1_dense_causal_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), batch,
                                           n, Hq, Hkv, d, _stream(stream)), "bf1_dense_causal_fwd")
    return out, lse


def release_plans():
    load().bf1_release_plans()


def set_forward_key_split(mode):
    """Forward key split: 0 automatic (default), 1 never, 2 always."""
    _check(load().bf1_set_forward_key_split(int(mode)), "bf1_set_forward_key_split")


def plan_transposed(n, B=64, L=2):
    """Transposed route (host only): for every key block, the ascending query
    blocks whose route selects it, as numpy int32 (row_ptr[NB+1], col_idx)."""
    import numpy as np
    nb, nnz, _ = plan_size(n, B, L)
    row_ptr = np.zeros(nb + 1, dtype=np.int32)
    col_idx = np.zeros(max(nnz, 1), dtype=np.int32)
    _check(load().bf1_plan_transposed(int(n), int(B), int(L), row_ptr.ctypes.data_as(ctypes.c_void_p),
                                      col_idx.ctypes.data_as(ctypes.c_void_p), col_idx.size),
           "bf1_plan_transposed")
    return row_ptr, col_idx[:nnz]


ROUTE_KINDS = {"bf1": 0, "sliding": 1, "static_random": 2}


def plan_variant(kind, n, B=64, L=2, seed=17):
    """Route table (host numpy int32 row_ptr[NB+1], col_idx) of kind "bf1",
    "sliding" (matched local sliding) or "static_random" (static random
    nonlocal graph drawn from `seed`); every kind has BF1's row sizes."""
    import numpy as np
    if kind not in ROUTE_KINDS:
        raise ValueError(f"unknown route kind {kind!r}; one of {sorted(ROUTE_KINDS)}")
    nb, nnz, _ = plan_size(n, B, L)
    row_ptr = np.zeros(nb + 1, dtype=np.int32)
    col_idx = np.zeros(max(nnz, 1), dtype=np.int32)
    _check(load().bf1_plan_variant(ROUTE_KINDS[kind], int(n), int(B), int(L), int(seed),
                                   row_ptr.ctypes.data_as(ctypes.c_void_p),
                                   col_idx.ctypes.data_as(ctypes.c_void_p), col_idx.size),
           "bf1_plan_variant")
    return row_ptr, col_idx[:nnz]


def route_depth(row_ptr, col_idx):
    """Communication depth (largest shortest path between blocks) of a host
    CSR route table; -1 if some later block is unreachable."""
    import numpy as np
    rp = np.ascontiguousarray(row_ptr, dtype=np.int32)
    ci = np.ascontiguousarray(col_idx, dtype=np.int32)
    if ci.size == 0:
        ci = np.zeros(1, dtype=np.int32)
    out = ctypes.c_int32(0)
    _check(load().bf1_route_depth(rp.ctypes.data_as(ctypes.c_void_p), ci.ctypes.data_as(ctypes.c_void_p),
                                  int(rp.size - 1), ctypes.byref(out)), "bf1_route_depth")
    return out.value


def bwd_workspace_size(batch, n, Hq, Hkv, d=128, B=64, L=2):
    """Bytes of device workspace bf1_attn_bwd needs."""
    out = ctypes.c_int64(0)
    _check(load().bf1_attn_bwd_workspace_size(int(batch), int(n), int(Hq), int(Hkv), int(d),
                                              int(B), int(L), ctypes.byref(out)),
           "bf1_attn_bwd_workspace_size")
    return out.value


def selected_bwd_flops(batch, n, Hq, d, B=64, L=2):
    """Algorithmic flops of the backward on the selected pairs: the five
    products S = Q K^T (recomputed), dP = dO V^T, dV = P^T dO, dQ = dS K and
    dK = dS^T Q, 2 d flops per selected pair each."""
    return 10 * d * plan_size(n, B, L)[2] * Hq * batch


def attn_bwd(q, k, v, o, do, lse, B=64, L=2, dq=None, dk=None, dv=None, workspace=None,
             stream=None):
    """BF1 backward; returns float32 (dQ, dK, dV).  o and lse are the
    forward's outputs; do is the upstream gradient of o (bf16, o's shape)."""
    import torch
    if o is None or lse is None:
        raise ValueError("attn_bwd needs the forward's o and lse")
    _, _, (batch, n, Hq, Hkv, d) = _prep(q, k, v, o, lse, True)
    dev = q.device
    check_buffer(do, "do", q.shape, torch.bfloat16, dev)

    def _grad(t, name, shape):
        if t is None:
            return torch.empty(shape, dtype=torch.float32, device=dev)
        return check_buffer(t, name, shape, torch.float32, dev)
    dq = _grad(dq, "dq", q.shape)
    dk = _grad(dk, "dk", k.shape)
    dv = _grad(dv, "dv", v.shape)
    need = bwd_workspace_size(batch, n, Hq, Hkv, d, B, L)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    ws_bytes = check_workspace(workspace, "workspace", need, dev)
    with torch.cuda.device(dev):
        _check(load().bf1_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse), _ptr(dq),
                                   _ptr(dk), _ptr(dv), batch, n, Hq, Hkv, d, int(B), int(L),
                                   _ptr(workspace), ws_bytes, _stream(stream)),
               "bf1_attn_bwd")
    return dq, dk, dv


# ---- one-token decode over a paged cache ------------------------------------

def decode_plan_stride(max_seq_len, B=64, L=2, dense=False):
    """int32 entries per sequence of a decode plan for up to max_seq_len tokens."""
    out = ctypes.c_int32(0)
    _check(load().bf1_decode_plan_stride(int(max_seq_len), int(B), int(L), int(bool(dense)),
                                         ctypes.byref(out)), "bf1_decode_plan_stride")
    return out.value


def _i32_cuda(t, name, dim, device=None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.int32 \
            or t.dim() != dim or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dim}-D int32 CUDA tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} must be on device {device}, got {t.device}")


def decode_plan(seq_lens, page_table, num_pages, stride, B=64, L=2, dense=False, plan=None,
                stream=None):
    """Decode plan [batch, stride] int32 (device) for the current block of
    every sequence: the pages of its earlier selected blocks."""
    import torch
    _i32_cuda(seq_lens, "seq_lens", 1)
    dev = seq_lens.device
    _i32_cuda(page_table, "page_table", 2, dev)
    batch, max_pages = page_table.shape
    if seq_lens.shape[0] != batch:
        raise ValueError("seq_lens and page_table disagree on the batch size")
    if plan is None:
        plan = torch.empty((batch, stride), dtype=torch.int32, device=dev)
    check_buffer(plan, "plan", (batch, stride), torch.int32, dev)
    with torch.cuda.device(dev):
        _check(load().bf1_decode_plan(batch, _ptr(seq_lens), _ptr(page_table), max_pages,
                                      int(num_pages), int(B), int(L), int(bool(dense)), _ptr(plan),
                                      int(stride), _stream(stream)), "bf1_decode_plan")
    return plan


def decode_workspace_size(batch, Hq, Hkv, head_dim, stride):
    out = ctypes.c_int64(0)
    _check(load().bf1_decode_workspace_size(int(batch), int(Hq), int(Hkv), int(head_dim), int(stride),
                                            ctypes.byref(out)), "bf1_decode_workspace_size")
    return out.value


def attn_decode(q, k_pages, v_pages, seq_lens, plan, B=64, out=None, lse=None, workspace=None,
                stream=None):
    """Attention of each sequence's newest token over the paged cache, using
    a decode plan; returns (O [batch, Hq, d] bf16, LSE [batch, Hq] fp32)."""
    import torch
    dev = _cuda_device(q, "q")
    if q.dim() != 3:
        raise ValueError("q must be 3-D [batch, Hq, d]")
    batch, Hq, d = q.shape
    check_buffer(q, "q", q.shape, torch.bfloat16, dev)
    if not isinstance(k_pages, torch.Tensor) or k_pages.dim() != 4:
        raise ValueError("k_pages must be a 4-D tensor [num_pages, Hkv, B, d]")
    num_pages, Hkv, pw, dk = k_pages.shape
    if dk != d or pw != B:
        raise ValueError("k_pages / v_pages must be [num_pages, Hkv, B, d] matching q")
    check_buffer(k_pages, "k_pages", k_pages.shape, torch.bfloat16, dev)
    check_buffer(v_pages, "v_pages", k_pages.shape, torch.bfloat16, dev)
    _i32_cuda(seq_lens, "seq_lens", 1, dev)
    _i32_cuda(plan, "plan", 2, dev)
    if seq_lens.shape[0] != batch or plan.shape[0] != batch:
        raise ValueError("batch sizes disagree")
    if out is None:
        out = torch.empty_like(q)
    check_buffer(out, "out", q.shape, torch.bfloat16, dev)
    if lse is None:
        lse = torch.empty((batch, Hq), dtype=torch.float32, device=dev)
    check_buffer(lse, "lse", (batch, Hq), torch.float32, dev)
    stride = plan.shape[1]
    need = decode_workspace_size(batch, Hq, Hkv, d, stride)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    ws_bytes = check_workspace(workspace, "workspace", need, dev)
    with torch.cuda.device(dev):
        _check(load().bf1_decode_attn(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(seq_lens), num_pages,
                                      _ptr(plan), stride, _ptr(out), _ptr(lse), batch, Hq, Hkv, d,
                                      int(B), _ptr(workspace), ws_bytes, _stream(stream)),
               "bf1_decode_attn")
    return out, lse
