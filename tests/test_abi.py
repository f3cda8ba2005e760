"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, computes route sizes in closed form (host code) that agree
with the oracle's enumeration, and rejects bad arguments before any device
call."""

import ctypes
import os
import re

import pytest

import paper_2608_20427_amd as bf1
from conftest import read_golden
from oracle import bf1_oracle as orc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bf1.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bf1_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bf1.lib_path()):
        pytest.fail("libbf1.so is not built (run __graft_entry__.build())")
    return bf1.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ["bf1_plan", "bf1_plan_size", "bf1_attn_fwd", "bf1_attn_fwd_csr",
                 "bf1_dense_causal_fwd", "bf1_release_plans", "bf1_status_string", "bf1_version"]:
        assert want in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for st in range(-6, 1):
        assert bf1.status_string(st).startswith("BF1")
    assert "unknown" in bf1.status_string(42)
    assert bf1.version() >= 10000


@pytest.mark.parametrize("n,B,L", [(512, 64, 1), (4096, 64, 2), (32768, 64, 2), (30001, 64, 2),
                                   (65536, 128, 2), (1, 64, 2), (0, 64, 2), (777, 5, 0),
                                   (100000, 64, 7)])
def test_plan_size_matches_oracle(lib, n, B, L):
    nb, nnz, pairs = bf1.plan_size(n, B, L)
    rp, ci = orc.csr(n, B, L)
    assert nb == len(rp) - 1 and nnz == len(ci)
    assert pairs == orc.selected_pairs(n, B, L)


def test_selected_flops_headline(lib):
    # 32K tokens, Qwen3-0.6B geometry: 4 * 128 * pairs * 16 q-heads.
    f = bf1.selected_flops(1, 32768, 16, 128, 64, 2)
    assert f == 4 * 128 * orc.selected_pairs(32768, 64, 2) * 16
    assert abs(f / 1e9 - 163.04) < 0.01


def test_invalid_arguments_rejected_without_device(lib):
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: checks come first
    st = lib.bf1_attn_fwd(fake, fake, fake, fake, None, 1, 128, 2, 1, 96, 64, 2, None)
    assert st == bf1.BF1_ERR_UNSUPPORTED
    st = lib.bf1_attn_fwd(fake, fake, fake, fake, None, 1, 128, 2, 1, 128, 48, 2, None)
    assert st == bf1.BF1_ERR_UNSUPPORTED
    st = lib.bf1_attn_fwd(fake, fake, fake, fake, None, 1, 128, 3, 2, 128, 64, 2, None)
    assert st == bf1.BF1_ERR_INVALID_ARG
    st = lib.bf1_attn_fwd(fake, fake, fake, fake, None, 1, 128, 6, 2, 128, 64, 2, None)
    assert st == bf1.BF1_ERR_UNSUPPORTED     # group of 3
    st = lib.bf1_attn_fwd(None, fake, fake, fake, None, 1, 128, 2, 1, 128, 64, 2, None)
    assert st == bf1.BF1_ERR_INVALID_ARG
    st = lib.bf1_attn_fwd(ctypes.c_void_p((1 << 20) + 8), fake, fake, fake, None, 1, 128, 2, 1,
                          128, 64, 2, None)
    assert st == bf1.BF1_ERR_INVALID_ARG     # misaligned
    st = lib.bf1_attn_fwd(fake, fake, fake, fake, None, 1, -5, 2, 1, 128, 64, 2, None)
    assert st == bf1.BF1_ERR_INVALID_ARG
    st = lib.bf1_attn_fwd(fake, fake, fake, fake, None, 1, 128, 2, 1, 128, 64, -1, None)
    assert st == bf1.BF1_ERR_INVALID_ARG
    st = lib.bf1_dense_causal_fwd(fake, fake, fake, fake, None, 1, 128, 2, 1, 80, None)
    assert st == bf1.BF1_ERR_UNSUPPORTED
    st = lib.bf1_attn_fwd_csr(fake, fake, fake, fake, None, 1, 128, 2, 1, 128, 64, None, fake, 4,
                              None)
    assert st == bf1.BF1_ERR_INVALID_ARG
    # plan: capacity below the route size is reported before any launch
    nb, nnz, _ = bf1.plan_size(4096, 64, 2)
    st = lib.bf1_plan(4096, 64, 2, fake, fake, nnz - 1, None)
    assert st == bf1.BF1_ERR_BUFFER_TOO_SMALL
    st = lib.bf1_plan(4096, 0, 2, fake, fake, nnz, None)
    assert st == bf1.BF1_ERR_INVALID_ARG


def test_empty_problems_are_noops(lib):
    # n == 0 / batch == 0 return before touching the device.
    st = lib.bf1_attn_fwd(None, None, None, None, None, 0, 128, 2, 1, 128, 64, 2, None)
    assert st == bf1.BF1_OK
    st = lib.bf1_dense_causal_fwd(None, None, None, None, None, 1, 0, 2, 1, 128, None)
    assert st == bf1.BF1_OK


# ---- backward boundary ------------------------------------------------------

def test_header_declares_the_backward():
    names = declared_functions()
    for want in ["bf1_plan_transposed", "bf1_attn_bwd_workspace_size", "bf1_attn_bwd"]:
        assert want in names


@pytest.mark.parametrize("n,B,L", [(1, 64, 2), (512, 64, 1), (4096, 64, 2), (32768, 64, 2),
                                   (30001, 64, 2), (1500, 128, 2), (5000, 7, 0), (777, 64, 3),
                                   (65536, 128, 2)])
def test_plan_transposed_matches_oracle(lib, n, B, L):
    rp, ci = bf1.plan_transposed(n, B, L)
    rp_o, ci_o = orc.csr_transposed(n, B, L)
    assert rp.tolist() == rp_o.tolist()
    assert ci.tolist() == ci_o.tolist()


def _ds_bytes(batch, n, Hq, B, L):
    # one 64 x 64 bf16 dS unit per (selected block pair, q-head, query and key
    # sub-tile of 64); the pairs are the entries of the transposed route
    _, ci = orc.csr_transposed(n, B, L)
    return batch * Hq * len(ci) * (B // 64) ** 2 * 64 * 64 * 2


def test_bwd_workspace_size_head_dim_64(lib):
    # partial dK/dV slots are 64 x head_dim fp32 tiles
    D = (1 * 16 * 32768 * 4 + 255) // 256 * 256
    assert bf1.bwd_workspace_size(1, 32768, 16, 8, 64, 64, 2) == (
        2 * D + 1 * 8 * 32 * 2 * 64 * 64 * 4 + _ds_bytes(1, 32768, 16, 64, 2))


def test_bwd_workspace_size(lib):
    # D and LSE log2 e (each batch * Hq * n fp32, 256-byte rounded), the
    # partial dK/dV slots of the tiles whose query-block list is longer than
    # one segment of 16 (at 32K / b = 64 only block 0: 512 users -> 32
    # segments), and the dS units.
    D = (1 * 16 * 32768 * 4 + 255) // 256 * 256
    part = 1 * 8 * 32 * 2 * 64 * 128 * 4
    assert bf1.bwd_workspace_size(1, 32768, 16, 8, 128, 64, 2) == 2 * D + part + _ds_bytes(1, 32768, 16, 64, 2)
    # a short sequence has no split lists
    assert bf1.bwd_workspace_size(1, 512, 2, 1, 128, 64, 1) == (
        2 * ((2 * 512 * 4 + 255) // 256 * 256) + _ds_bytes(1, 512, 2, 64, 1))
    # b = 128: four 64 x 64 units per pair and head; block 0's 32 users make two
    # segments for each of its two 64-key sub-tiles (four partial slots)
    assert bf1.bwd_workspace_size(2, 4096, 4, 2, 128, 128, 2) == (
        2 * ((2 * 4 * 4096 * 4 + 255) // 256 * 256) + 2 * 2 * 4 * 2 * 64 * 128 * 4 + _ds_bytes(2, 4096, 4, 128, 2))


def test_backward_invalid_arguments_rejected_without_device(lib):
    fake = ctypes.c_void_p(1 << 20)
    args = [fake] * 9
    def call(*a, ws=fake, wsb=1 << 40):
        return lib.bf1_attn_bwd(*a, ws, wsb, None)
    # head_dims other than 64 and 128 are not built
    assert call(*args, 1, 128, 2, 1, 96, 64, 2) == bf1.BF1_ERR_UNSUPPORTED
    # G * B < 128
    assert call(*args, 1, 128, 2, 2, 128, 64, 2) == bf1.BF1_ERR_UNSUPPORTED
    # missing gradient buffer / workspace, misaligned workspace, too small workspace
    assert call(*args[:6], None, fake, fake, 1, 128, 2, 1, 128, 64, 2) == bf1.BF1_ERR_INVALID_ARG
    assert call(*args, 1, 128, 2, 1, 128, 64, 2, ws=None) == bf1.BF1_ERR_INVALID_ARG
    assert call(*args, 1, 128, 2, 1, 128, 64, 2, ws=ctypes.c_void_p((1 << 20) + 16)) == \
        bf1.BF1_ERR_INVALID_ARG
    assert call(*args, 1, 128, 2, 1, 128, 64, 2, wsb=16) == bf1.BF1_ERR_BUFFER_TOO_SMALL
    assert call(*args, 1, 128, 2, 1, 128, 64, -1) == bf1.BF1_ERR_INVALID_ARG
    # empty problems are no-ops
    assert lib.bf1_attn_bwd(*([None] * 9), 0, 128, 2, 1, 128, 64, 2, None, 0, None) == bf1.BF1_OK
    # transposed plan: capacity check
    nb, nnz, _ = bf1.plan_size(4096, 64, 2)
    import numpy as np
    rp = np.zeros(nb + 1, dtype=np.int32)
    ci = np.zeros(nnz, dtype=np.int32)
    assert lib.bf1_plan_transposed(4096, 64, 2, rp.ctypes.data_as(ctypes.c_void_p),
                                   ci.ctypes.data_as(ctypes.c_void_p), nnz - 1) == \
        bf1.BF1_ERR_BUFFER_TOO_SMALL


# ---- route variants and the depth tool (host entry points) -------------------

VARIANT_CASES = [(1, 64, 2), (257, 64, 2), (4096, 64, 2), (32768, 64, 2), (30001, 64, 2),
                 (65536, 128, 2), (512, 64, 1), (5000, 7, 0), (777, 16, 3), (3000, 8, 5)]


def test_header_declares_the_variants():
    names = declared_functions()
    for want in ["bf1_plan_variant", "bf1_route_depth"]:
        assert want in names


@pytest.mark.parametrize("kind", ["bf1", "sliding", "static_random"])
@pytest.mark.parametrize("n,B,L", VARIANT_CASES)
def test_plan_variant_matches_oracle(lib, kind, n, B, L):
    for seed in (17, 2 ** 64 - 1, 0):
        rp, ci = bf1.plan_variant(kind, n, B, L, seed)
        rp_o, ci_o = orc.variant_csr(kind, n, B, L, seed)
        assert rp.tolist() == rp_o.tolist(), seed
        assert ci.tolist() == ci_o.tolist(), seed
        if kind != "static_random":
            break


@pytest.mark.parametrize("n,B,L", VARIANT_CASES[:6])
def test_plan_variant_bf1_equals_planner_table(lib, n, B, L):
    rp, ci = bf1.plan_variant("bf1", n, B, L)
    rp_o, ci_o = orc.csr(n, B, L)
    assert rp.tolist() == rp_o.tolist() and ci.tolist() == ci_o.tolist()


@pytest.mark.parametrize("kind", ["bf1", "sliding", "static_random"])
@pytest.mark.parametrize("NB,B,L", [(1, 64, 2), (2, 64, 2), (40, 16, 2), (300, 4, 1), (512, 64, 2),
                                    (1024, 64, 2), (200, 8, 4)])
def test_route_depth_matches_oracle(lib, kind, NB, B, L):
    rp, ci = bf1.plan_variant(kind, NB * B, B, L, 17)
    assert bf1.route_depth(rp, ci) == orc.max_shortest_path_csr(*orc.variant_csr(kind, NB * B, B, L, 17))


def test_route_depth_golden(lib):
    for route_kind, NB, L, depth in read_golden("route_variant_depth.txt"):
        rp, ci = bf1.plan_variant(route_kind, int(NB) * 64, 64, int(L))
        assert bf1.route_depth(rp, ci) == int(depth)


def test_route_depth_unreachable_and_invalid(lib):
    import numpy as np
    # rows {0}, {1}, {1, 2}: block 2 is unreachable from block 0
    rp = np.array([0, 1, 2, 4], dtype=np.int32)
    ci = np.array([0, 1, 1, 2], dtype=np.int32)
    assert bf1.route_depth(rp, ci) == -1
    out = ctypes.c_int32(7)
    vp = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    # a future block in row 1, a decreasing row_ptr, too many blocks
    bad = np.array([0, 2, 3], dtype=np.int32)
    assert lib.bf1_route_depth(vp(np.array([0, 1, 3], dtype=np.int32)), vp(bad), 2, ctypes.byref(out)) == \
        bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_route_depth(vp(np.array([0, 2, 1], dtype=np.int32)), vp(ci), 2, ctypes.byref(out)) == \
        bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_route_depth(vp(rp), vp(ci), 16385, ctypes.byref(out)) == bf1.BF1_ERR_INVALID_ARG
    assert out.value == 7
    # unknown kind, capacity
    r = np.zeros(70, dtype=np.int32)
    c = np.zeros(500, dtype=np.int32)
    assert lib.bf1_plan_variant(3, 4096, 64, 2, 17, vp(r), vp(c), 500) == bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_plan_variant(1, 4096, 64, 2, 17, vp(r), vp(c), 441) == bf1.BF1_ERR_BUFFER_TOO_SMALL
    with pytest.raises(ValueError):
        bf1.plan_variant("dilated", 4096)


# ---- decode (host-side checks) ------------------------------------------------

def test_header_declares_the_decode():
    names = declared_functions()
    for want in ["bf1_decode_plan_stride", "bf1_decode_plan", "bf1_decode_workspace_size",
                 "bf1_decode_attn"]:
        assert want in names


@pytest.mark.parametrize("n,B,L", [(1, 64, 2), (64, 64, 2), (65, 64, 2), (32768, 64, 2), (65536, 64, 2),
                                   (30001, 64, 1), (5000, 128, 3), (1 << 20, 64, 0)])
def test_decode_plan_stride_is_the_largest_route(lib, n, B, L):
    NB = -(-n // B)
    cap = max(len(orc.route(j, L)) - 1 for j in range(NB))
    assert bf1.decode_plan_stride(n, B, L) == 3 + cap
    assert bf1.decode_plan_stride(n, B, L, dense=True) == 3 + (NB - 1)


def test_decode_workspace_size(lib):
    # 32K, batch 1, Qwen geometry: P = 11 pages -> 11 splits of one page;
    # record = G * (d + 2) floats per split
    st = bf1.decode_plan_stride(32768, 64, 2)
    assert st == 3 + 10
    assert bf1.decode_workspace_size(1, 16, 8, 128, st) == (8 * 11 * 2 * 130 * 4 + 255) // 256 * 256
    # batch 32: 1024 / 256 = 4 splits wanted -> 3 pages per split -> 4 splits
    assert bf1.decode_workspace_size(32, 16, 8, 128, st) == (32 * 8 * 4 * 2 * 130 * 4 + 255) // 256 * 256


def test_decode_invalid_arguments_rejected_without_device(lib):
    fake = ctypes.c_void_p(1 << 20)
    out = ctypes.c_int32(0)
    assert lib.bf1_decode_plan_stride(0, 64, 2, 0, ctypes.byref(out)) == bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_decode_plan_stride(100, 32, 2, 0, ctypes.byref(out)) == bf1.BF1_ERR_UNSUPPORTED
    assert lib.bf1_decode_plan_stride(100, 64, 33, 0, ctypes.byref(out)) == bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_decode_plan_stride(100, 64, 2, 2, ctypes.byref(out)) == bf1.BF1_ERR_INVALID_ARG
    # plan: stride below 2, null pointers, batch 0 is a no-op
    assert lib.bf1_decode_plan(1, fake, fake, 4, 4, 64, 2, 0, fake, 2, None) == bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_decode_plan(1, None, fake, 4, 4, 64, 2, 0, fake, 20, None) == bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_decode_plan(0, None, None, 4, 4, 64, 2, 0, None, 20, None) == bf1.BF1_OK
    args = [fake] * 4
    def attn(*tail, ws=fake, wsb=1 << 40, Hq=16, Hkv=8, d=128, B=64, stride=13):
        return lib.bf1_decode_attn(*args, 100, fake, stride, fake, None, 1, Hq, Hkv, d, B, ws, wsb, None)
    assert attn(d=96) == bf1.BF1_ERR_UNSUPPORTED
    assert attn(B=32) == bf1.BF1_ERR_UNSUPPORTED
    assert attn(Hq=12, Hkv=8) == bf1.BF1_ERR_INVALID_ARG
    assert attn(Hq=48, Hkv=3) == bf1.BF1_ERR_UNSUPPORTED
    assert attn(stride=2) == bf1.BF1_ERR_INVALID_ARG
    assert attn(ws=None) == bf1.BF1_ERR_INVALID_ARG
    assert attn(ws=ctypes.c_void_p((1 << 20) + 8)) == bf1.BF1_ERR_INVALID_ARG
    assert attn(wsb=1024) == bf1.BF1_ERR_BUFFER_TOO_SMALL


def test_key_split_mode_checked(lib):
    assert lib.bf1_set_forward_key_split(3) == bf1.BF1_ERR_INVALID_ARG
    assert lib.bf1_set_forward_key_split(-1) == bf1.BF1_ERR_INVALID_ARG
    for mode in (1, 2, 0):
        assert lib.bf1_set_forward_key_split(mode) == bf1.BF1_OK
