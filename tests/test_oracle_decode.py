"""Pins of the oracle's one-token decode (CPU only), §3.2 (a decoded token
reads O(log NB) blocks), §4.2 ("cached one-token decode" agrees with the
blockwise reference) and §5.4:

* the decode row equals the last row of the prefill forward computed from
  the full n x n mask (form (i), the definition) on the same keys, values
  and query -- the decode path is the forward at the last position;
* a route that covers every block reduces it to a dense causal row;
* K = 0 closed form: every visible key has weight 1/|S(t)|, with
  |S(t)| = (t mod b) + 1 + b c(j) from the closed route count;
* keys at positions >= seq_len are never read (NaN there changes nothing);
* the decode plan: c(j) earlier pages, mapped through the page table.
"""

import math

import numpy as np
import pytest

import test_oracle_route as TR
from oracle import bf1_oracle as orc


def _cache(seed, batch, Hq, Hkv, n, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((batch, Hq, d)), rng.standard_normal((batch, Hkv, n, d)),
            rng.standard_normal((batch, Hkv, n, d)))


@pytest.mark.parametrize("b,L", [(16, 2), (8, 1), (16, 3), (32, 0)])
def test_decode_equals_last_row_of_full_mask_forward(b, L):
    batch, Hq, Hkv, d, n_max = 3, 4, 2, 8, 300
    q, k, v = _cache(7 + b + L, batch, Hq, Hkv, n_max, d)
    seq_lens = [1, 5 * b, 257] if b < 32 else [1, 64, 300]
    o, l = orc.attn_decode_fp64(q, k, v, seq_lens, b, L)
    for beta, n in enumerate(seq_lens):
        t = n - 1
        rng = np.random.default_rng(n)
        qf = rng.standard_normal((1, Hq, n, d))     # earlier queries do not matter
        qf[0, :, t] = q[beta]
        of, lf = orc.attn_full_mask_fp64(qf, k[beta:beta + 1, :, :n], v[beta:beta + 1, :, :n], b, L)
        assert np.max(np.abs(o[beta] - of[0, :, t])) < 1e-12
        assert np.max(np.abs(l[beta] - lf[0, :, t])) < 1e-12


def test_decode_covering_route_is_dense_causal_row():
    b, L = 16, 2
    n = 4 * b                      # NB = 4 <= L + 2: every block selected
    q, k, v = _cache(3, 1, 2, 1, n, 8)
    o, l = orc.attn_decode_fp64(q, k, v, [n], b, L)
    qf = np.zeros((1, 2, n, 8))
    qf[0, :, n - 1] = q[0]
    od, ld = orc.dense_causal_fp64(qf, k, v, rows=[n - 1])
    assert np.max(np.abs(o[0] - od[0, :, n - 1])) < 1e-12
    assert np.max(np.abs(l[0] - ld[0, :, n - 1])) < 1e-12


@pytest.mark.parametrize("n", [1, 17, 64, 65, 1000, 4097])
def test_decode_zero_keys_closed_form(n):
    b, L = 64, 2
    rng = np.random.default_rng(n)
    q = rng.standard_normal((1, 2, 16))
    k = np.zeros((1, 1, n, 16))
    v = rng.standard_normal((1, 1, n, 16))
    o, l = orc.attn_decode_fp64(q, k, v, [n], b, L)
    t = n - 1
    j = t // b
    size = (t % b) + 1 + b * TR.pred_count(j, L)
    assert np.allclose(l, math.log(size), atol=1e-12, rtol=0)
    keys = [s for s in range(n) if s // b == j or s // b in orc.route(j, L)]
    assert len(keys) == size
    assert np.max(np.abs(o[0] - v[0, 0, keys].mean(axis=0))) < 1e-12


def test_decode_reads_nothing_past_the_sequence():
    b, L = 16, 2
    q, k, v = _cache(5, 2, 2, 1, 200, 8)
    seq_lens = [150, 33]
    o1, l1 = orc.attn_decode_fp64(q, k, v, seq_lens, b, L)
    k2, v2 = k.copy(), v.copy()
    for beta, n in enumerate(seq_lens):
        k2[beta, :, n:] = np.nan
        v2[beta, :, n:] = np.nan
    o2, l2 = orc.attn_decode_fp64(q, k2, v2, seq_lens, b, L)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


@pytest.mark.parametrize("L", [0, 1, 2, 3])
def test_decode_plan_counts_and_mapping(L):
    b = 64
    rng = np.random.default_rng(L)
    page_row = rng.permutation(1000)
    for n in [1, 64, 65, 128, 129, 4096, 32768, 30001, 64000]:
        j, earlier = orc.decode_plan(n, page_row, b, L)
        assert j == (n - 1) // b
        assert len(earlier) == TR.pred_count(j, L)
        inv = {int(p): i for i, p in enumerate(page_row)}
        blocks = [inv[p] for p in earlier]
        assert blocks == sorted(blocks) and all(i < j for i in blocks)
        assert set(blocks) | {j} == set(orc.route(j, L))
        jd, dense = orc.decode_plan(n, page_row, b, L, dense=True)
        assert jd == j and dense == [int(page_row[i]) for i in range(j)]
