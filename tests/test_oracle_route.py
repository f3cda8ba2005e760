"""Pins of the oracle's route, CSR and pair accounting against what the paper
and the mathematics fix (CPU only).

* hand-derived routes from §3.1 Eq. 1 (golden fixture);
* Proposition 1's bound |P(j)| <= 4 + floor(log2 j) (§3.2);
* the closed O(n log n) pair law, derived independently below, against
  brute-force enumeration of the token mask;
* the 26.98x selected-interaction reduction at 32K (§5.1, Table 2);
* the maximum shortest path of 8 layers at 512 blocks (§3.3, Prop. 2).
"""

import math

import numpy as np
import pytest

from conftest import read_golden
from oracle import bf1_oracle as orc


# ---------------------------------------------------------------------------
# Closed forms, derived from the definition by counting (not by enumeration)
# ---------------------------------------------------------------------------

def dyadic_new(j, L):
    """Dyadic offsets 2^r (r >= 2) that reach a block not already local."""
    return [1 << r for r in range(2, 40) if L < (1 << r) <= j]


def pred_count(j, L):
    """Number of selected blocks of query block j other than j itself:
    min(j, L) locals, the new dyadic ones, and the global block 0 when it is
    neither local nor dyadic."""
    D = dyadic_new(j, L)
    return min(j, L) + len(D) + (1 if (j > L and j not in D) else 0)


def pairs_closed(n, b, L):
    """Selected token pairs per (batch, head): every earlier selected block
    contributes b x (rows of block j) pairs, the self block a triangle with
    its diagonal; only the last block can be partial (m rows and keys)."""
    if n == 0:
        return 0
    NB = -(-n // b)
    m = n - (NB - 1) * b
    full = sum(pred_count(j, L) for j in range(NB - 1))
    return b * b * full + (NB - 1) * b * (b + 1) // 2 + m * b * pred_count(NB - 1, L) + m * (m + 1) // 2


def row_ptr_closed(j, L):
    """Start of row j in the CSR: sum over i < j of |P(i)| = 1 + pred_count(i),
    summed term by term in closed form."""
    selfs = j
    locs = j * (j - 1) // 2 if j <= L else L * (L - 1) // 2 + L * (j - L)
    dy = sum(j - (1 << r) for r in range(2, 40) if L < (1 << r) < j)
    glob = max(0, j - L - 1) - sum(1 for r in range(2, 40) if L < (1 << r) < j)
    return selfs + locs + dy + glob


# ---------------------------------------------------------------------------
# Route
# ---------------------------------------------------------------------------

def test_route_matches_hand_derived_eq1():
    rows = read_golden("routes_hand.txt")
    assert len(rows) >= 25
    for row in rows:
        L, j = int(row[0]), int(row[1])
        assert row[2] == ":"
        want = [int(x) for x in row[3:]]
        assert orc.route(j, L) == want, (L, j)


@pytest.mark.parametrize("L", [0, 1, 2])
def test_prop1_bound(L):
    # §3.2, Proposition 1: each block selects at most 4 + floor(log2 j)
    # predecessor blocks (stated for the paper's route; holds for L <= 2).
    for j in range(1, 5000):
        assert len(orc.route(j, L)) <= 4 + int(math.floor(math.log2(j)))


@pytest.mark.parametrize("L", [0, 1, 2, 3, 5, 8])
def test_route_sizes_match_closed_count(L):
    for j in range(0, 3000):
        r = orc.route(j, L)
        assert len(r) == 1 + pred_count(j, L)
        assert r == sorted(set(r)) and r[0] == 0 and r[-1] == j


@pytest.mark.parametrize("L", [0, 1, 2, 3, 7])
def test_csr_row_ptr_closed_form(L):
    row_ptr, col_idx = orc.csr(300 * 64 + 17, 64, L)
    NB = len(row_ptr) - 1
    assert NB == 301
    for j in range(NB + 1):
        assert row_ptr[j] == row_ptr_closed(j, L), (L, j)
    assert len(col_idx) == row_ptr[-1]


# ---------------------------------------------------------------------------
# Pair law: brute force over the token mask == enumeration == closed law
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 5, 63, 64, 65, 128, 257, 512, 777, 1000, 1300])
@pytest.mark.parametrize("L", [1, 2, 3])
def test_pairs_brute_force(n, L):
    b = 64
    brute = int(orc.token_mask(n, b, L).sum())
    assert brute == orc.selected_pairs(n, b, L) == pairs_closed(n, b, L)


@pytest.mark.parametrize("b", [4, 8, 16])
def test_pairs_brute_force_small_blocks(b):
    for n in [1, 3, b, b + 1, 5 * b - 1, 23 * b + 3]:
        for L in [0, 1, 2, 4]:
            brute = int(orc.token_mask(n, b, L).sum())
            assert brute == orc.selected_pairs(n, b, L) == pairs_closed(n, b, L)


def test_mask_is_causal_and_keeps_diagonal():
    m = orc.token_mask(777, 16, 2)
    assert not np.triu(m, 1).any()          # nothing above the diagonal
    assert m.diagonal().all()                # every row sees itself


def test_pair_law_is_n_log_n():
    # Proposition 1: pairs <= b^2 * sum_j (1 + |P(j)| bound) = O(n b log(n/b)).
    b = 64
    for n in [1 << k for k in range(10, 18)]:
        NB = n // b
        bound = b * b * sum(5 + int(math.log2(j)) if j else 1 for j in range(NB))
        assert orc.selected_pairs(n, b, 2) <= bound


def test_interaction_reduction_32k():
    rows = read_golden("interaction_reduction.txt")
    for n, b, L, printed, dec in rows:
        n, b, L, dec = int(n), int(b), int(L), int(dec)
        red = orc.dense_pairs(n) / orc.selected_pairs(n, b, L)
        assert round(red, dec) == float(printed), red


def test_communication_depth_512():
    rows = read_golden("communication_depth.txt")
    for NB, L, depth in rows:
        assert orc.max_shortest_path(int(NB), int(L)) == int(depth)


def test_communication_depth_popcount_bound():
    # §3.3: a path from i to j needs at most popcount(j - i) layers.
    NB = 200
    succ = {j: [i for i in orc.route(j, 2) if i != j] for j in range(NB)}
    # shortest path lengths by dynamic programming over the DAG
    dist = np.full((NB, NB), 10**9, dtype=np.int64)
    for i in range(NB):
        dist[i, i] = 0
    for j in range(NB):
        for p in succ[j]:
            dist[:, j] = np.minimum(dist[:, j], dist[:, p] + 1)
    for i in range(NB):
        for j in range(i + 1, NB):
            assert dist[i, j] <= bin(j - i).count("1") or i == 0
            if i == 0:
                assert dist[i, j] == 1
