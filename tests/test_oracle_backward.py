"""Pins of the oracle's backward (CPU only): the gradients of the BF1
attention (§3.1 mask, softmax without bias) with respect to Q, K and V.

Independent checks, each able to catch a slip in the analytic formulas:
* central finite differences of the oracle's forward (the definition) for
  the loss sum(O * W), whose upstream gradient is dO = W;
* PyTorch autograd in float64 through a separately written masked-softmax
  forward (a library differentiating the definition);
* invariants that follow from the rows of P summing to one: the dV rows of a
  kv-head sum to the dO rows of its q-heads, and its dK rows sum to zero;
* the zero-keys closed form: with K = 0 every visible key has weight
  1/|S(t)|, so dQ = 0 and dV_s = sum over visible t of dO_t / |S(t)|;
* the transposed route against the closed form of who selects block i.
"""

import math

import numpy as np
import pytest
import torch

from oracle import bf1_oracle as orc


def _rand(seed, batch, Hq, Hkv, n, d):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((batch, Hq, n, d))
    k = rng.standard_normal((batch, Hkv, n, d))
    v = rng.standard_normal((batch, Hkv, n, d))
    w = rng.standard_normal((batch, Hq, n, d))
    return q, k, v, w


@pytest.mark.parametrize("n,b,L,Hq,Hkv", [(23, 4, 1, 2, 1), (17, 8, 2, 1, 1), (19, 4, 0, 4, 2)])
def test_backward_matches_finite_differences(n, b, L, Hq, Hkv):
    q, k, v, w = _rand(11 + n, 1, Hq, Hkv, n, 3)
    dq, dk, dv = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)

    def loss(q_, k_, v_):
        o, _ = orc.attn_full_mask_fp64(q_, k_, v_, b, L)
        return float(np.sum(o * w))

    eps = 1e-6
    rng = np.random.default_rng(5)
    for name, arr, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(12):  # random coordinates
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            plus, minus = arr.copy(), arr.copy()
            plus[idx] += eps
            minus[idx] -= eps
            args_p = {"q": (plus, k, v), "k": (q, plus, v), "v": (q, k, plus)}[name]
            args_m = {"q": (minus, k, v), "k": (q, minus, v), "v": (q, k, minus)}[name]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (name, idx, fd, grad[idx])


@pytest.mark.parametrize("n,b,L", [(70, 8, 2), (45, 16, 1)])
def test_backward_matches_torch_autograd(n, b, L):
    batch, Hq, Hkv, d = 2, 4, 2, 5
    q, k, v, w = _rand(3 + n, batch, Hq, Hkv, n, d)
    dq, dk, dv = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    mask = torch.tensor(orc.token_mask(n, b, L))
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    tv = torch.tensor(v, requires_grad=True)
    G = Hq // Hkv
    kk = tk.repeat_interleave(G, dim=1)
    vv = tv.repeat_interleave(G, dim=1)
    x = (tq @ kk.transpose(-1, -2)) / math.sqrt(d)
    x = x.masked_fill(~mask, float("-inf"))
    o = torch.softmax(x, dim=-1) @ vv
    (o * torch.tensor(w)).sum().backward()
    np.testing.assert_allclose(dq, tq.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk, tk.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv, tv.grad.numpy(), rtol=0, atol=1e-12)


def test_backward_row_sum_invariants():
    n, b, L = 300, 16, 2
    q, k, v, w = _rand(7, 1, 4, 2, n, 8)
    dq, dk, dv = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    # sum_s dK_s = c sum_t (sum_s dS_ts) q_t = 0, per kv-head
    assert np.abs(dk.sum(axis=2)).max() < 1e-10
    # sum_s dV_s = sum_t (sum_s P_ts) dO_t = sum of dO over the group's q-heads
    dsum = w.reshape(1, 2, 2, n, 8).sum(axis=(2, 3))
    np.testing.assert_allclose(dv.sum(axis=2), dsum, rtol=0, atol=1e-9)


def test_backward_zero_keys_closed_form():
    n, b, L = 130, 16, 2
    q, _, v, w = _rand(9, 1, 2, 1, n, 4)
    k = np.zeros((1, 1, n, 4))
    dq, dk, dv = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    assert np.abs(dq).max() < 1e-12
    mask = orc.token_mask(n, b, L).astype(np.float64)
    per_row = mask / mask.sum(axis=1, keepdims=True)  # uniform weights
    expect = sum(per_row.T @ w[0, h] for h in range(2))
    np.testing.assert_allclose(dv[0, 0], expect, rtol=0, atol=1e-12)


def test_backward_subsets_equal_full_rows():
    n, b, L = 200, 16, 2
    q, k, v, w = _rand(13, 1, 2, 1, n, 4)
    full = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    part = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L, q_blocks=[0, 5, 12], kv_blocks=[0, 3, 12])
    for jb in (0, 5, 12):
        sl = slice(jb * b, min((jb + 1) * b, n))
        np.testing.assert_allclose(part[0][:, :, sl], full[0][:, :, sl], rtol=0, atol=1e-12)
    for ib in (0, 3, 12):
        sl = slice(ib * b, min((ib + 1) * b, n))
        np.testing.assert_allclose(part[1][:, :, sl], full[1][:, :, sl], rtol=0, atol=1e-12)
        np.testing.assert_allclose(part[2][:, :, sl], full[2][:, :, sl], rtol=0, atol=1e-12)
    assert np.isnan(part[0][:, :, b:2 * b]).all() and np.isnan(part[1][:, :, b:2 * b]).all()


@pytest.mark.parametrize("NB,L", [(1, 2), (9, 1), (40, 2), (130, 3), (512, 2)])
def test_transposed_route_closed_form(NB, L):
    # Block i is selected by itself, its L local successors, the blocks 2^r
    # (r >= 2) past it, and -- block 0 only -- by every query block.
    b = 4
    row_ptr, col_idx = orc.csr_transposed(NB * b, b, L)
    for i in range(NB):
        got = col_idx[row_ptr[i]:row_ptr[i + 1]].tolist()
        if i == 0:
            expect = list(range(NB))
        else:
            cand = {i + ell for ell in range(0, L + 1)}
            r = 2
            while i + (1 << r) < NB:
                cand.add(i + (1 << r))
                r += 1
            expect = sorted(j for j in cand if j < NB)
        assert got == expect, (i, got, expect)


def test_backward_with_exact_output_equals_exact_delta():
    # D = rowsum(dO * O) for the exact O is the same number as rowsum(P * dP).
    n, b, L = 150, 16, 2
    q, k, v, w = _rand(17, 1, 4, 2, n, 6)
    o, _ = orc.attn_gathered_fp64(q, k, v, b, L)
    a = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    c = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L, o=o)
    for x, y in zip(a, c):
        np.testing.assert_allclose(x, y, rtol=0, atol=1e-12)


def test_abs_terms_bound_the_gradients():
    # |sum of terms| <= sum of |terms|, element by element.
    n, b, L = 120, 16, 2
    q, k, v, w = _rand(19, 1, 2, 1, n, 6)
    g = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    t = orc.attn_bwd_abs_terms_fp64(q, k, v, w, b, L)
    for x, y in zip(g, t):
        assert (np.abs(x) <= y + 1e-12).all()


# ---------------------------------------------------------------------------
# Tightness of the term-magnitude sums (the backward's element-wise error
# scale): they must equal the hand-worked values, and they must be attained
# exactly when every term of a gradient element has the same sign.
# ---------------------------------------------------------------------------

def _hand_case(case):
    V = np.array([[1, 0], [0, 1], [1, 1.0]])
    dO = np.array([[1, 0], [0, 2], [1, -1.0]])
    K = np.array([[1, 2], [3, -1], [-2, 1.0]])
    Q = np.array([[2, 1], [1, -1], [0, 3.0]])
    q, k = (np.zeros((3, 2)), K) if case == "A" else (Q, np.zeros((3, 2)))
    return [x[None, None] for x in (q, k, V, dO)]


def test_abs_terms_hand_worked(golden):
    from fractions import Fraction
    rows = golden("bwd_abs_terms_hand.txt")
    assert len(rows) == 16
    c = 1 / math.sqrt(2)
    for case, kind, grad, row, a, b, times in rows:
        q, k, v, do = _hand_case(case)
        got = orc.attn_bwd_abs_terms_fp64(q, k, v, do, 4, 2, kind=kind)
        g = {"dQ": got[0], "dK": got[1], "dV": got[2]}[grad][0, 0, int(row)]
        want = np.array([float(Fraction(a)), float(Fraction(b))]) * (c if times == "c" else 1.0)
        np.testing.assert_allclose(g, want, rtol=0, atol=1e-14, err_msg=f"{case} {kind} {grad} {row}")


def test_abs_terms_dv_attained_for_nonnegative_upstream():
    # With dO >= 0 every term P_ts dO_t of dV_s is non-negative, so the sum of
    # magnitudes is the gradient itself.
    n, b, L = 90, 8, 2
    q, k, v, w = _rand(23, 1, 4, 2, n, 5)
    w = np.abs(w)
    _, _, dv = orc.attn_bwd_gathered_fp64(q, k, v, w, b, L)
    _, _, tv = orc.attn_bwd_abs_terms_fp64(q, k, v, w, b, L)
    np.testing.assert_allclose(tv, np.abs(dv), rtol=1e-12, atol=1e-14)


def test_abs_terms_dq_attained_for_one_sign_per_row():
    # Two keys per query row (block width 1, route {0, j} at L = 0 only for
    # j = 1): dS of row 1 is (-x, +x).  With K_0 <= 0 <= K_1 both terms of
    # dQ_1 = c (dS_10 K_0 + dS_11 K_1) share a sign in every column, so the
    # sum of magnitudes equals |dQ_1|.
    rng = np.random.default_rng(29)
    q = rng.standard_normal((1, 1, 2, 4))
    k = np.stack([-np.abs(rng.standard_normal(4)), np.abs(rng.standard_normal(4))])[None, None]
    v = rng.standard_normal((1, 1, 2, 4))
    do = rng.standard_normal((1, 1, 2, 4))
    dq, _, _ = orc.attn_bwd_gathered_fp64(q, k, v, do, 1, 0)
    tq, _, _ = orc.attn_bwd_abs_terms_fp64(q, k, v, do, 1, 0)
    p_ds = np.sign(dq[0, 0, 1])
    assert np.all(p_ds != 0)
    np.testing.assert_allclose(tq[0, 0, 1], np.abs(dq[0, 0, 1]), rtol=1e-12)
