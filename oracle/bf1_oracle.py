"""CPU oracle for BF1 causal dyadic block-sparse attention (prefill forward).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path
(the HIP library and its Python binding) never imports, calls or links it,
and this module imports nothing from the product path.

Everything here is written for clarity, not speed: the route is enumerated
as a set straight from its definition, the attention is an explicit masked
softmax in float64, and no blocking, fusion or reordering is done beyond
what the definition states.

Notation (paper §3.1): a sequence of n tokens is cut into NB = ceil(n/b)
blocks of width b, indexed 0..NB-1 (the paper calls the block count B; the
C interface of the library uses B for the *width*, so this module writes
b for the width and NB for the count to avoid the clash).

Route (§3.1, Eq. 1): query block j selects
    P(j) = {j, j-1, j-2, 0} ∪ {j - 2^r : r >= 2},
with invalid (negative) and duplicate indices removed.  The paper's reported
configuration has two local predecessor blocks; this oracle generalises the
local part to {j-1, ..., j-L} for a local width L >= 0 and keeps the dyadic
offsets at r >= 2 (offsets starting at four blocks, §3.1), so L = 2 is
exactly Eq. 1.

Mask (§3.1): the self block j uses a token-level causal triangle (key s is
visible to query t in the same block iff s <= t); every other selected block
is strictly earlier and fully visible.  Keys at positions >= n do not exist.

Backward: the gradients of O with respect to Q, K and V for an upstream
gradient dO, on the same route (the operator the paper trains through,
§2/§4.1).  With P the masked softmax weights, D_t = sum_s P_ts dP_ts and the
scale c = 1/sqrt(head_dim), these are the textbook softmax-attention
gradients: dV = P^T dO, dP = dO V^T, dS = P * (dP - D), dQ = c dS K,
dK = c dS^T Q, summed over the q-heads of a GQA group for dK and dV.

Route variants (§4.3, §5.1, §5.2, Table 1): the paper's two topology
controls at the same selected-pair budget as BF1 -- a contiguous local
sliding window and a fixed ("static") random nonlocal graph -- plus the
maximum shortest-path depth of any block route.  The paper names these
controls but does not spell out their construction; the readings taken here
are stated at route_sliding and route_static_random.  The random graph is
parity-unpinned beyond its invariants (exact row sizes, locals kept,
causality) and the published SplitMix64 outputs its draws come from.

Decode (§3.2, last paragraph; §4.2 "cached one-token decode"; §5.4): the
token at position t = seq_len - 1 of a sequence attends to the same keys as
row t of the prefill mask -- the earlier selected blocks of its block
j = t // b in full, and its own block up to t -- read from a cache of
earlier keys and values.  decode_plan lists the physical pages (blocks)
such a token reads through a page table; attn_decode_fp64 is the attention
row itself.

Attention: softmax with scale 1/sqrt(head_dim) and no score bias (§3.1,
"no scale-dependent score bias"), restricted to the mask above.  q-head h
reads kv-head h // (Hq / Hkv) (contiguous GQA groups).  Outputs are O
(same layout as Q) and the natural-log log-sum-exp LSE per query row.
"""

import math
from collections import deque

import numpy as np

__all__ = [
    "num_blocks",
    "route",
    "route_table",
    "csr",
    "token_mask",
    "token_mask_csr",
    "selected_pairs",
    "dense_pairs",
    "max_shortest_path",
    "route_sliding",
    "route_static_random",
    "splitmix64",
    "variant_csr",
    "csr_pairs",
    "max_shortest_path_csr",
    "attn_full_mask_fp64",
    "attn_gathered_fp64",
    "attn_csr_fp64",
    "dense_causal_fp64",
    "csr_transposed",
    "decode_plan",
    "attn_decode_fp64",
    "attn_bwd_csr_fp64",
    "attn_bwd_gathered_fp64",
    "attn_bwd_abs_terms_fp64",
]


# ---------------------------------------------------------------------------
# Route (§3.1, Eq. 1)
# ---------------------------------------------------------------------------

def num_blocks(n, b):
    """NB = ceil(n / b) blocks of width b (§3.1)."""
    if b <= 0:
        raise ValueError("block width must be positive")
    if n < 0:
        raise ValueError("sequence length must be non-negative")
    return (n + b - 1) // b


def route(j, L=2):
    """Selected key blocks of query block j, ascending (§3.1, Eq. 1).

    The union of the self block, L local predecessors, the global first
    block and the dyadic predecessors j - 2^r for r >= 2, with indices
    outside [0, j] and duplicates removed.
    """
    if j < 0:
        raise ValueError("block index must be non-negative")
    if L < 0:
        raise ValueError("local width must be non-negative")
    chosen = {j, 0}
    for ell in range(1, L + 1):
        chosen.add(j - ell)
    r = 2
    while (1 << r) <= j:
        chosen.add(j - (1 << r))
        r += 1
    return sorted(i for i in chosen if 0 <= i <= j)


def route_table(n, b, L=2):
    """List of routes, one per query block."""
    return [route(j, L) for j in range(num_blocks(n, b))]


def csr(n, b, L=2):
    """Route as a CSR table: row_ptr[NB+1], col_idx[nnz] (int32, ascending)."""
    rows = route_table(n, b, L)
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int64)
    for j, r in enumerate(rows):
        row_ptr[j + 1] = row_ptr[j] + len(r)
    col_idx = np.array([i for r in rows for i in r], dtype=np.int64)
    return row_ptr.astype(np.int32), col_idx.astype(np.int32)


def token_mask(n, b, L=2, rows=None):
    """Boolean token mask allowed[t, s] of shape [len(rows), n] (§3.1).

    allowed(t, s) holds iff block(s) is in P(block(t)) and either block(s)
    is strictly earlier than block(t) or s <= t inside the self block.
    """
    if rows is None:
        rows = np.arange(n)
    rows = np.asarray(rows)
    allowed = np.zeros((len(rows), n), dtype=bool)
    s = np.arange(n)
    for a, t in enumerate(rows):
        j = t // b
        for i in route(j, L):
            lo, hi = i * b, min((i + 1) * b, n)
            if i < j:
                allowed[a, lo:hi] = True
            else:  # self block: token-level causal triangle, diagonal kept
                allowed[a, lo:hi] = s[lo:hi] <= t
    return allowed


def token_mask_csr(n, b, row_ptr, col_idx):
    """[n, n] boolean token mask of any causal block route in CSR form, by
    the same rule as token_mask: earlier selected blocks fully visible, the
    self block as a causal triangle with its diagonal."""
    allowed = np.zeros((n, n), dtype=bool)
    s = np.arange(n)
    for t in range(n):
        j = t // b
        for i in col_idx[row_ptr[j]:row_ptr[j + 1]]:
            i = int(i)
            lo, hi = i * b, min((i + 1) * b, n)
            if i < j:
                allowed[t, lo:hi] = True
            elif i == j:
                allowed[t, lo:hi] = s[lo:hi] <= t
    return allowed


def selected_pairs(n, b, L=2):
    """Selected (query, key) token pairs per (batch, head), by enumeration.

    Walks every query block and every selected key block and counts the
    visible pairs of that block pair: a full rectangle for an earlier block,
    the causal triangle (diagonal included) for the self block.
    """
    total = 0
    for j, sel in enumerate(route_table(n, b, L)):
        rows_j = min((j + 1) * b, n) - j * b
        for i in sel:
            if i < j:
                total += rows_j * (min((i + 1) * b, n) - i * b)
            else:
                total += rows_j * (rows_j + 1) // 2
    return total


def dense_pairs(n):
    """Token pairs of dense causal attention, diagonal included."""
    return n * (n + 1) // 2


def max_shortest_path(NB, L=2):
    """Largest shortest-path length, in layers, from any block to any later
    block of the block graph whose edges are i -> j for i in P(j), i != j
    (the communication depth of §3.3, Proposition 2).  Breadth-first search
    from every source block."""
    return _max_shortest_path_rows([route(j, L) for j in range(NB)])


def _max_shortest_path_rows(rows):
    """Breadth-first search from every source block over the edges i -> j
    for i in rows[j], i != j; the largest distance to a later block.  Raises
    if some later block cannot be reached at all."""
    NB = len(rows)
    succ = [[] for _ in range(NB)]
    for j in range(NB):
        for i in rows[j]:
            if i != j:
                succ[i].append(j)
    worst = 0
    for src in range(NB):
        dist = [-1] * NB
        dist[src] = 0
        queue = deque([src])
        while queue:
            u = queue.popleft()
            for w in succ[u]:
                if dist[w] < 0:
                    dist[w] = dist[u] + 1
                    queue.append(w)
        for j in range(src + 1, NB):
            if dist[j] < 0:
                raise AssertionError(f"block {j} unreachable from {src}")
            worst = max(worst, dist[j])
    return worst


# ---------------------------------------------------------------------------
# Route variants at BF1's selected-pair budget (§4.3, §5.1, §5.2, Table 1)
# ---------------------------------------------------------------------------

_MASK64 = (1 << 64) - 1


def splitmix64(seed, c):
    """Output number c (c = 0, 1, ...) of the SplitMix64 generator seeded with
    ``seed`` (Steele, Lea and Flood, "Fast splittable pseudorandom number
    generators", OOPSLA 2014; the 64-bit finaliser constants of Vigna's
    public-domain splitmix64).  The state after c + 1 steps is
    seed + (c + 1) * 0x9E3779B97F4A7C15 mod 2^64, so any output can be
    evaluated directly from its counter."""
    z = (seed + (c + 1) * 0x9E3779B97F4A7C15) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def route_sliding(j, L=2):
    """Matched local sliding route of query block j: the |P(j)| most recent
    blocks, j - |P(j)| + 1 .. j, ascending.

    Reading: "equal-pair-count local sliding" (§4.3, §5.1; "contiguous
    local", Table 1) keeps BF1's block count per query block, so every row
    sees exactly as many key tokens as under Eq. 1 and the totals match.
    This reading gives a maximum shortest path of 59 at 512 blocks, the
    number §5.2 reports for matched sliding at 32K.
    """
    size = len(route(j, L))
    return list(range(j - size + 1, j + 1))


def route_static_random(j, L=2, seed=17):
    """Matched static-random nonlocal route of query block j.

    Reading (the paper fixes the seed, 17, and the budget but not the
    construction, §4.4 and Table 1): the self block and its L local
    predecessors are kept as in Eq. 1; BF1's nonlocal blocks (the global
    block 0 and the dyadic ones, all earlier than j - L) are replaced by as
    many distinct blocks drawn uniformly from 0 .. j - L - 1.  Row sizes, and
    therefore the selected pairs, equal BF1's.

    The draw is Floyd's sampling of k out of m = j - L candidates (Bentley
    and Floyd, "A sample of brilliance", CACM 30(9), 1987): for t = 0..k-1
    with r = m - k + t, take x uniform in [0, r]; add r if x was taken
    before, else x.  Draw t of row j uses the SplitMix64 output with counter
    j * 2^20 + t, mapped to [0, r] as (high 32 bits * (r + 1)) >> 32.
    """
    local = [i for i in range(j - L, j + 1) if i >= 0]
    k = len(route(j, L)) - len(local)
    m = j - L
    taken = set()
    for t in range(k):
        r = m - k + t
        x = ((splitmix64(seed, (j << 20) + t) >> 32) * (r + 1)) >> 32
        taken.add(r if x in taken else x)
    return sorted(taken | set(local))


def variant_csr(kind, n, b, L=2, seed=17):
    """CSR table (row_ptr[NB+1], col_idx) of a route: kind "bf1" (Eq. 1),
    "sliding" or "static_random" (see route_sliding, route_static_random)."""
    NB = num_blocks(n, b)
    if kind == "bf1":
        rows = [route(j, L) for j in range(NB)]
    elif kind == "sliding":
        rows = [route_sliding(j, L) for j in range(NB)]
    elif kind == "static_random":
        rows = [route_static_random(j, L, seed) for j in range(NB)]
    else:
        raise ValueError(f"unknown route kind {kind!r}")
    row_ptr = np.zeros(NB + 1, dtype=np.int64)
    for j, r in enumerate(rows):
        row_ptr[j + 1] = row_ptr[j] + len(r)
    col_idx = np.array([i for r in rows for i in r], dtype=np.int64)
    return row_ptr.astype(np.int32), col_idx.astype(np.int32)


def csr_pairs(n, b, row_ptr, col_idx):
    """Selected (query, key) token pairs per (batch, head) of any causal
    block route in CSR form, counted block pair by block pair as in
    selected_pairs."""
    total = 0
    for j in range(len(row_ptr) - 1):
        rows_j = min((j + 1) * b, n) - j * b
        for i in col_idx[row_ptr[j]:row_ptr[j + 1]]:
            i = int(i)
            if i < j:
                total += rows_j * (min((i + 1) * b, n) - i * b)
            elif i == j:
                total += rows_j * (rows_j + 1) // 2
    return total


def max_shortest_path_csr(row_ptr, col_idx):
    """Communication depth (§3.3, §5.2) of any block route in CSR form: the
    largest shortest-path length from a block to a later block."""
    NB = len(row_ptr) - 1
    return _max_shortest_path_rows(
        [[int(i) for i in col_idx[row_ptr[j]:row_ptr[j + 1]]] for j in range(NB)])


# ---------------------------------------------------------------------------
# Attention (§3.1 mask; softmax attention without bias)
# ---------------------------------------------------------------------------

def _check_shapes(q, k, v):
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("expected [batch, heads, n, head_dim] arrays")
    batch, Hq, n, d = q.shape
    if k.shape != v.shape or k.shape[0] != batch or k.shape[2] != n or k.shape[3] != d:
        raise ValueError("K and V must be [batch, Hkv, n, head_dim] matching Q")
    Hkv = k.shape[1]
    if Hkv == 0 or Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    return batch, Hq, Hkv, n, d


def _softmax_rows(x, vals):
    """Explicit softmax over the last axis of x (rows with -inf entries are
    masked keys), returning (weights @ vals, log-sum-exp)."""
    m = np.max(x, axis=-1, keepdims=True)
    lse = m + np.log(np.sum(np.exp(x - m), axis=-1, keepdims=True))
    w = np.exp(x - lse)
    return w @ vals, lse[..., 0]


def attn_full_mask_fp64(q, k, v, b, L=2, scale=None, mask=None):
    """Form (i): materialise the n x n token mask and run a masked softmax.

    For small n only (memory is n^2 per head).  Inputs are float arrays in
    [batch, H, n, d] layout; returns (O float64 [batch, Hq, n, d],
    LSE float64 [batch, Hq, n], natural log).  ``mask`` replaces the BF1
    mask by another [n, n] boolean token mask (e.g. token_mask_csr).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    batch, Hq, Hkv, n, d = _check_shapes(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    G = Hq // Hkv
    if mask is None:
        mask = token_mask(n, b, L)
    out = np.zeros((batch, Hq, n, d))
    lse = np.zeros((batch, Hq, n))
    for beta in range(batch):
        for h in range(Hq):
            g = h // G
            x = scale * (q[beta, h] @ k[beta, g].T)
            x = np.where(mask, x, -np.inf)
            out[beta, h], lse[beta, h] = _softmax_rows(x, v[beta, g])
    return out, lse


def attn_csr_fp64(q, k, v, b, row_ptr, col_idx, scale=None, blocks=None):
    """Form (ii): gathered attention over an explicit block route given as
    a CSR table (row j selects key blocks col_idx[row_ptr[j]:row_ptr[j+1]]).

    Per query block, the selected key ranges are concatenated, the self
    block gets its causal triangle, and one explicit softmax runs over the
    gathered keys.  ``blocks`` restricts the computation to some query
    blocks (the other rows of the outputs are left as NaN).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    batch, Hq, Hkv, n, d = _check_shapes(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    G = Hq // Hkv
    NB = num_blocks(n, b)
    out = np.full((batch, Hq, n, d), np.nan)
    lse = np.full((batch, Hq, n), np.nan)
    todo = range(NB) if blocks is None else blocks
    for j in todo:
        t0, t1 = j * b, min((j + 1) * b, n)
        sel = [int(i) for i in col_idx[row_ptr[j]:row_ptr[j + 1]]]
        keys = np.concatenate([np.arange(i * b, min((i + 1) * b, n)) for i in sel])
        t = np.arange(t0, t1)[:, None]
        s = keys[None, :]
        allowed = (s // b < j) | (s <= t)
        for beta in range(batch):
            for h in range(Hq):
                g = h // G
                x = scale * (q[beta, h, t0:t1] @ k[beta, g, keys].T)
                x = np.where(allowed, x, -np.inf)
                out[beta, h, t0:t1], lse[beta, h, t0:t1] = _softmax_rows(x, v[beta, g, keys])
    return out, lse


def attn_gathered_fp64(q, k, v, b, L=2, scale=None, blocks=None):
    """Form (ii) over the BF1 route of Eq. 1 (O(n log n) work)."""
    n = np.shape(q)[2]
    row_ptr, col_idx = csr(n, b, L)
    return attn_csr_fp64(q, k, v, b, row_ptr, col_idx, scale=scale, blocks=blocks)


def dense_causal_fp64(q, k, v, scale=None, rows=None):
    """Plain dense causal softmax attention in float64 (every key s <= t).

    ``rows`` optionally restricts the query positions computed (others NaN).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    batch, Hq, Hkv, n, d = _check_shapes(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    G = Hq // Hkv
    rows = np.arange(n) if rows is None else np.asarray(rows)
    out = np.full((batch, Hq, n, d), np.nan)
    lse = np.full((batch, Hq, n), np.nan)
    for beta in range(batch):
        for h in range(Hq):
            g = h // G
            for t in rows:
                x = scale * (k[beta, g, : t + 1] @ q[beta, h, t])
                m = np.max(x)
                z = np.sum(np.exp(x - m))
                lse[beta, h, t] = m + np.log(z)
                out[beta, h, t] = np.exp(x - lse[beta, h, t]) @ v[beta, g, : t + 1]
    return out, lse


# ---------------------------------------------------------------------------
# Backward (gradients of the §3.1 attention with respect to Q, K, V)
# ---------------------------------------------------------------------------

def csr_transposed(n, b, L=2):
    """Transposed route: for every key block i, the ascending query blocks j
    that select it (i in P(j), Eq. 1), as CSR (row_ptr[NB+1], col_idx).
    Built by inverting the enumerated route table."""
    NB = num_blocks(n, b)
    users = [[] for _ in range(NB)]
    for j, sel in enumerate(route_table(n, b, L)):
        for i in sel:
            users[i].append(j)
    row_ptr = np.zeros(NB + 1, dtype=np.int64)
    for i in range(NB):
        row_ptr[i + 1] = row_ptr[i] + len(users[i])
    col_idx = np.array([j for u in users for j in sorted(u)], dtype=np.int64)
    return row_ptr.astype(np.int32), col_idx.astype(np.int32)


def attn_bwd_csr_fp64(q, k, v, do, b, row_ptr, col_idx, scale=None, q_blocks=None,
                      kv_blocks=None, o=None, _core=None):
    """Gradients (dQ, dK, dV) of the attention over a CSR block route, in
    float64, for the upstream gradient dO (same layout as O).

    For every query block j the selected key ranges are gathered exactly as
    in the forward (form ii), the masked softmax weights P are formed, and
    with D = rowsum(P * dP):
        dP = dO V^T,  dS = P * (dP - D),
        dV += P^T dO,  dQ = c dS K,  dK += c dS^T Q.
    ``q_blocks`` restricts which query blocks' dQ rows are computed and
    ``kv_blocks`` which key blocks' dK/dV rows are accumulated (all by
    default); rows not computed are NaN.  Only the query blocks needed for
    the requested rows are visited.  ``o`` (the forward output, same layout as
    Q) makes D = rowsum(dO * o) instead of the exact rowsum(P * dP): the two
    agree for the exact o; a given o is what a backward that takes O as an
    input computes with.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    batch, Hq, Hkv, n, d = _check_shapes(q, k, v)
    if do.shape != q.shape:
        raise ValueError("dO must have the shape of Q")
    if o is not None:
        o = np.asarray(o, dtype=np.float64)
        if o.shape != q.shape:
            raise ValueError("o must have the shape of Q")
    core = _core if _core is not None else _bwd_gathered
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    G = Hq // Hkv
    NB = num_blocks(n, b)
    qset = set(range(NB)) if q_blocks is None else {int(x) for x in q_blocks}
    kvset = set(range(NB)) if kv_blocks is None else {int(x) for x in kv_blocks}
    dq = np.full(q.shape, np.nan)
    dk = np.full(k.shape, np.nan)
    dv = np.full(v.shape, np.nan)
    for j in qset:
        dq[:, :, j * b:min((j + 1) * b, n)] = 0.0
    for i in kvset:
        dk[:, :, i * b:min((i + 1) * b, n)] = 0.0
        dv[:, :, i * b:min((i + 1) * b, n)] = 0.0
    for j in range(NB):
        sel = [int(i) for i in col_idx[row_ptr[j]:row_ptr[j + 1]]]
        if j not in qset and not kvset.intersection(sel):
            continue
        t0, t1 = j * b, min((j + 1) * b, n)
        keys = np.concatenate([np.arange(i * b, min((i + 1) * b, n)) for i in sel])
        t = np.arange(t0, t1)[:, None]
        s = keys[None, :]
        allowed = (s // b < j) | (s <= t)
        keep = np.isin(keys // b, list(kvset))  # key rows whose dK/dV are requested
        for beta in range(batch):
            for h in range(Hq):
                g = h // G
                delta = None if o is None else np.sum(do[beta, h, t0:t1] * o[beta, h, t0:t1], axis=1)
                gq, gk, gv = core(q[beta, h, t0:t1], k[beta, g, keys], v[beta, g, keys],
                                  do[beta, h, t0:t1], allowed, scale, delta)
                if j in qset:
                    dq[beta, h, t0:t1] = gq
                if keep.any():
                    kk = keys[keep]
                    dv[beta, g, kk] += gv[keep]
                    dk[beta, g, kk] += gk[keep]
    return dq, dk, dv


def _bwd_weights(qr, kr, vr, dor, allowed, scale, delta):
    """Masked softmax weights P, dP = dO V^T and dS = P (dP - D) of one set of
    query rows over gathered keys (D = rowsum(P dP) unless given)."""
    x = scale * (qr @ kr.T)
    x = np.where(allowed, x, -np.inf)
    m = np.max(x, axis=1, keepdims=True)
    p = np.exp(x - m)
    p /= np.sum(p, axis=1, keepdims=True)
    dp = dor @ vr.T
    if delta is None:
        delta = np.sum(p * dp, axis=1)
    ds = p * (dp - delta[:, None])
    return p, ds


def _bwd_gathered(qr, kr, vr, dor, allowed, scale, delta=None):
    """Softmax-attention gradients for one set of query rows qr over gathered
    keys kr / values vr with a boolean mask: returns (dQ rows, dK rows,
    dV rows) of this row set's contribution."""
    p, ds = _bwd_weights(qr, kr, vr, dor, allowed, scale, delta)
    return scale * (ds @ kr), scale * (ds.T @ qr), p.T @ dor


def _bwd_abs_terms(qr, kr, vr, dor, allowed, scale, delta=None):
    """Sums of the magnitudes of the terms of each gradient element:
    c sum_s |dS||K|, c sum_t |dS||Q|, sum_t P |dO| (same shapes)."""
    p, ds = _bwd_weights(qr, kr, vr, dor, allowed, scale, delta)
    a = np.abs(ds)
    return scale * (a @ np.abs(kr)), scale * (a.T @ np.abs(qr)), p.T @ np.abs(dor)


def _bwd_abs_terms_pdp(qr, kr, vr, dor, allowed, scale, delta=None):
    """As _bwd_abs_terms with |dS| = P |dP - D| replaced by P (|dP| + |D|):
    the scale of the cancellation in dP - D (dV has no such term: zeros)."""
    p, _ = _bwd_weights(qr, kr, vr, dor, allowed, scale, delta)
    dp = dor @ vr.T
    if delta is None:
        delta = np.sum(p * dp, axis=1)
    a = p * (np.abs(dp) + np.abs(delta)[:, None])
    return scale * (a @ np.abs(kr)), scale * (a.T @ np.abs(qr)), np.zeros((kr.shape[0], dor.shape[1]))


def attn_bwd_gathered_fp64(q, k, v, do, b, L=2, scale=None, q_blocks=None, kv_blocks=None,
                           o=None):
    """Backward over the BF1 route of Eq. 1."""
    n = np.shape(q)[2]
    row_ptr, col_idx = csr(n, b, L)
    return attn_bwd_csr_fp64(q, k, v, do, b, row_ptr, col_idx, scale=scale,
                             q_blocks=q_blocks, kv_blocks=kv_blocks, o=o)


def attn_bwd_abs_terms_fp64(q, k, v, do, b, L=2, scale=None, q_blocks=None, kv_blocks=None,
                            o=None, kind="ds"):
    """Term-magnitude sums of the backward over the BF1 route, laid out like
    (dQ, dK, dV).  kind "ds": c sum_s |dS_ts| |K_s|, c sum_t |dS_ts| |Q_t|,
    sum_t P_ts |dO_t| -- an implementation that rounds P and dS to bf16
    (relative error <= 2^-8, 8 significant bits) before the products has
    element errors bounded by 2^-8 times these.  kind "pdp": the same with |dS| replaced by
    P (|dP| + |D|), the scale of the fp32 cancellation in dS = P (dP - D)."""
    n = np.shape(q)[2]
    row_ptr, col_idx = csr(n, b, L)
    core = {"ds": _bwd_abs_terms, "pdp": _bwd_abs_terms_pdp}[kind]
    return attn_bwd_csr_fp64(q, k, v, do, b, row_ptr, col_idx, scale=scale, q_blocks=q_blocks,
                             kv_blocks=kv_blocks, o=o, _core=core)


# ---------------------------------------------------------------------------
# One-token decode (§3.2, §4.2, §5.4)
# ---------------------------------------------------------------------------

def decode_plan(seq_len, page_row, b, L=2, dense=False):
    """Pages read by the newest token of a sequence of seq_len tokens whose
    logical block i lives in physical page page_row[i]: returns (j, earlier)
    with j = (seq_len - 1) // b the token's block and ``earlier`` the physical
    pages of the selected blocks before j (P(j) without j, ascending by
    logical block; every earlier block for ``dense``).  The self page is
    page_row[j]."""
    if seq_len < 1:
        raise ValueError("a decode step needs at least one token")
    j = (seq_len - 1) // b
    blocks = range(j) if dense else [i for i in route(j, L) if i < j]
    return j, [int(page_row[i]) for i in blocks]


def attn_decode_fp64(q, k, v, seq_lens, b, L=2, scale=None):
    """Attention of each sequence's newest token (position t = seq_len - 1).

    q: [batch, Hq, d] (the newest token's query per q-head); k, v:
    [batch, Hkv, n_max, d] logical key/value caches (positions >= seq_len are
    ignored).  Row t of the §3.1 token mask over seq_len tokens decides which
    keys are visible; returns (O [batch, Hq, d], LSE [batch, Hq]) in float64.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    batch, Hq, d = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    G = Hq // Hkv
    out = np.zeros((batch, Hq, d))
    lse = np.zeros((batch, Hq))
    for beta in range(batch):
        n = int(seq_lens[beta])
        t = n - 1
        keys = np.nonzero(token_mask(n, b, L, rows=[t])[0])[0]
        for h in range(Hq):
            g = h // G
            x = scale * (k[beta, g, keys] @ q[beta, h])
            o, l = _softmax_rows(x[None, :], v[beta, g, keys])
            out[beta, h], lse[beta, h] = o[0], l[0]
    return out, lse
