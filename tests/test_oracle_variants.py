"""Pins of the oracle's route variants and graph depth (CPU only).

The paper's topology controls (§4.3, §5.1, §5.2, Table 1) are an
equal-pair-count local sliding route and a static random nonlocal route
(graph seed 17).  What pins them:

* matched sliding: its maximum shortest path at 512 blocks is 59, the value
  §5.2 reports (golden fixture), and its pair count equals BF1's;
* static random: the SplitMix64 outputs its draws come from match the
  published generator (golden fixture); every row keeps the self block and
  the locals, is causal and duplicate-free and has BF1's size; the draw is
  uniform over the candidate blocks (frequency test over many seeds).  The
  construction itself is a reading (parity unpinned beyond these);
* the depth search: breadth-first search against an all-pairs shortest path
  computed by min-plus matrix products, and BF1's 8 layers at 512 blocks;
* attention over a variant table: the gathered form against the full-mask
  softmax over the same table's token mask, and pair counts against the
  mask's popcount.
"""

import numpy as np
import pytest

from conftest import read_golden
from oracle import bf1_oracle as orc

KINDS = ("bf1", "sliding", "static_random")


def test_splitmix64_published_outputs():
    for seed, c, out in read_golden("splitmix64.txt"):
        assert orc.splitmix64(int(seed), int(c)) == int(out)


@pytest.mark.parametrize("route_kind,NB,L,depth", [tuple(r) for r in read_golden("route_variant_depth.txt")])
def test_depth_golden(route_kind, NB, L, depth):
    rp, ci = orc.variant_csr(route_kind, int(NB) * 64, 64, int(L))
    assert orc.max_shortest_path_csr(rp, ci) == int(depth)


def apsp_minplus(rp, ci):
    """All-pairs shortest path lengths by repeated min-plus products of the
    one-hop distance matrix (an independent check of the breadth-first
    search): D[i, j] = hops from block i to block j."""
    NB = len(rp) - 1
    inf = 10 ** 6
    A = np.full((NB, NB), inf, dtype=np.int64)
    np.fill_diagonal(A, 0)
    for j in range(NB):
        for i in ci[rp[j]:rp[j + 1]]:
            if int(i) != j:
                A[int(i), j] = 1
    D = A.copy()
    while True:
        nxt = np.min(D[:, :, None] + A[None, :, :], axis=1)
        if np.array_equal(nxt, D):
            return D
        D = nxt


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("NB,L", [(1, 2), (7, 2), (40, 2), (33, 1), (29, 3)])
def test_depth_bfs_matches_minplus(kind, NB, L):
    rp, ci = orc.variant_csr(kind, NB * 16, 16, L, seed=5)
    D = apsp_minplus(rp, ci)
    upper = [D[i, j] for j in range(NB) for i in range(j)]
    assert max(upper, default=0) < 10 ** 6
    assert orc.max_shortest_path_csr(rp, ci) == max(upper, default=0)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("n,b,L", [(1, 64, 2), (63, 64, 2), (257, 64, 2), (777, 16, 2), (1000, 8, 1),
                                   (1300, 16, 3), (2050, 32, 2), (512, 64, 0)])
def test_variant_pairs_equal_bf1_and_mask(kind, n, b, L):
    rp, ci = orc.variant_csr(kind, n, b, L, seed=17)
    bf1 = orc.selected_pairs(n, b, L)
    assert orc.csr_pairs(n, b, rp, ci) == bf1
    assert int(orc.token_mask_csr(n, b, rp, ci).sum()) == bf1


@pytest.mark.parametrize("L", [0, 1, 2, 3, 5])
def test_variant_rows_valid(L):
    NB = 300
    for kind in ("sliding", "static_random"):
        rp, ci = orc.variant_csr(kind, NB * 4, 4, L, seed=17)
        for j in range(NB):
            row = [int(i) for i in ci[rp[j]:rp[j + 1]]]
            assert row == sorted(set(row)), (kind, j)
            assert len(row) == len(orc.route(j, L)), (kind, j)
            assert 0 <= row[0] and row[-1] == j, (kind, j)
            assert set(range(max(0, j - L), j + 1)) <= set(row), (kind, j)
            if kind == "sliding":
                assert row == list(range(j - len(row) + 1, j + 1))


def test_sliding_hand_rows():
    # |P(j)| at L = 2 for j = 0..9 is 1, 2, 3, 4, 4, 5, 5, 5, 5, 6 (Eq. 1), so
    # the sliding windows are the most recent that many blocks.
    want = [[0], [0, 1], [0, 1, 2], [0, 1, 2, 3], [1, 2, 3, 4], [1, 2, 3, 4, 5], [2, 3, 4, 5, 6],
            [3, 4, 5, 6, 7], [4, 5, 6, 7, 8], [4, 5, 6, 7, 8, 9]]
    assert [orc.route_sliding(j, 2) for j in range(10)] == want


def test_static_random_is_uniform_over_candidates():
    # Row j = 40 at L = 2: BF1 selects {0, 8, 24, 32, 36, 38, 39, 40}, so the
    # random row keeps {38, 39, 40} and draws k = 5 of the m = 38 blocks
    # 0..37.  Over S seeds every candidate is drawn with probability k / m.
    j, L, S = 40, 2, 6000
    k, m = 5, 38
    counts = np.zeros(m, dtype=np.int64)
    for seed in range(S):
        row = orc.route_static_random(j, L, seed)
        far = [i for i in row if i < j - L]
        assert len(far) == k and len(set(far)) == k
        counts[far] += 1
    p = k / m
    mean, sd = S * p, np.sqrt(S * p * (1 - p))
    assert np.all(np.abs(counts - mean) < 5 * sd), counts
    chi2 = float(np.sum((counts - mean) ** 2 / mean))
    assert chi2 < 80.0, chi2      # 37 degrees of freedom: mean 37, sd ~8.6


def test_static_random_depends_on_seed_only_through_draws():
    a = orc.variant_csr("static_random", 64 * 200, 64, 2, seed=17)
    b = orc.variant_csr("static_random", 64 * 200, 64, 2, seed=17)
    c = orc.variant_csr("static_random", 64 * 200, 64, 2, seed=18)
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[0], c[0])
    assert not np.array_equal(a[1], c[1])


@pytest.mark.parametrize("kind", ("sliding", "static_random"))
@pytest.mark.parametrize("n,b,L", [(200, 16, 2), (257, 32, 1)])
def test_variant_attention_gathered_equals_full_mask(kind, n, b, L):
    rng = np.random.default_rng(11)
    q = rng.standard_normal((1, 2, n, 16))
    k = rng.standard_normal((1, 1, n, 16))
    v = rng.standard_normal((1, 1, n, 16))
    rp, ci = orc.variant_csr(kind, n, b, L, seed=17)
    o1, l1 = orc.attn_csr_fp64(q, k, v, b, rp, ci)
    o2, l2 = orc.attn_full_mask_fp64(q, k, v, b, mask=orc.token_mask_csr(n, b, rp, ci))
    assert np.max(np.abs(o1 - o2)) < 1e-12 and np.max(np.abs(l1 - l2)) < 1e-12


def test_sliding_covering_every_block_is_dense_causal():
    # At L = NB - 2 every BF1 row holds all of 0..j, so the sliding window is
    # the whole causal prefix: attention equals dense causal attention.
    n, b = 96, 16
    NB = n // b
    rp, ci = orc.variant_csr("sliding", n, b, NB - 2)
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((1, 1, n, 8)) for _ in range(3))
    o1, l1 = orc.attn_csr_fp64(q, k, v, b, rp, ci)
    o2, l2 = orc.dense_causal_fp64(q, k, v)
    assert np.max(np.abs(o1 - o2)) < 1e-12 and np.max(np.abs(l1 - l2)) < 1e-12
