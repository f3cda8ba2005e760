"""Sizes at the interface's limits.

The longest sequence the interface accepts, n = 2^24 - 1 tokens (every
per-head byte offset of a head_dim 128 row then stays below 2^32), through
the BF1 forward at head_dim 128, B = 64, L = 2, with one GQA group of two
q-heads; the fp64 oracle checks sampled query blocks, the partial last block
(63 tokens) among them.  The inputs (26 GB on the device) are drawn there by
a seeded generator; the oracle gets the device's bits of the rows it needs.

Each sampled block j is checked as a compact problem holding only its route:
the selected blocks P(j) (§3.1, Eq. 1, ascending, the self block last) laid
side by side, with query block j as the last block.  The mask of §3.1 only
distinguishes earlier blocks (fully visible) from the self block (causal by
position inside the block), and both are preserved by that relabelling.
Bars: the forward's (O max-abs 2e-2, mean-abs 2e-3, LSE max-abs 1e-3).

The backward at 2^20 tokens, where its dS workspace (one 8 KB unit per
selected block pair and q-head) passes 2^31 bytes and key block 0's list of
16384 query blocks is cut into 1024 partial slots; sampled dQ rows and
dK / dV rows (block 0 among them) against the oracle, with the backward's
element-wise bound (test_gpu_backward.py).
"""

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
import test_gpu_backward as TB
import test_gpu_parity as TP
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu

N_MAX = (1 << 24) - 1


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()
    yield
    torch.cuda.synchronize()


def test_forward_longest_supported_sequence():
    b, L = 64, 2
    w = synth.Workload("longest", 1, N_MAX, 2, 1, 128, b, L, seed=24)
    TP.say(f"longest sequence: n = {w.n}, drawing inputs on the device")
    q, k, v = synth.make_qkv_device(w)
    o, lse = bf1.attn_fwd(q, k, v, B=b, L=L)
    torch.cuda.synchronize()
    NB = orc.num_blocks(w.n, b)
    assert NB == 1 << 18 and w.n - (NB - 1) * b == 63
    for j in (0, 1, 5, 1000, NB // 2 + 3, NB - 2, NB - 1):
        blocks = orc.route(j, L)
        m = len(blocks)
        t0, t1 = j * b, min((j + 1) * b, w.n)
        nc = (m - 1) * b + (t1 - t0)
        qc = np.zeros((1, w.Hq, nc, w.d))
        kc = np.zeros((1, w.Hkv, nc, w.d))
        vc = np.zeros((1, w.Hkv, nc, w.d))
        qc[:, :, (m - 1) * b:] = synth.to_f64(q[:, :, t0:t1].cpu())
        for c, i in enumerate(blocks):
            s0, s1 = i * b, min((i + 1) * b, w.n)
            kc[:, :, c * b:c * b + (s1 - s0)] = synth.to_f64(k[:, :, s0:s1].cpu())
            vc[:, :, c * b:c * b + (s1 - s0)] = synth.to_f64(v[:, :, s0:s1].cpu())
        # compact route: block c < m-1 selects itself only (not checked);
        # the last block selects every block of the compact sequence
        row_ptr = np.array(list(range(m)) + [2 * m - 1], dtype=np.int64)
        col_idx = np.array(list(range(m - 1)) + list(range(m)), dtype=np.int64)
        o_ref, l_ref = orc.attn_csr_fp64(qc, kc, vc, b, row_ptr, col_idx, blocks=[m - 1])
        TP.compare(o[:, :, t0:t1], lse[:, :, t0:t1], o_ref[:, :, (m - 1) * b:], l_ref[:, :, (m - 1) * b:],
                   tag=f"longest sequence, query block {j} ({m} blocks)")
    # every output row written and finite (one q-head at a time)
    for h in range(w.Hq):
        assert torch.isfinite(o[:, h]).all() and torch.isfinite(lse[:, h]).all(), h


def test_backward_million_tokens():
    b, L = 64, 2
    w = synth.Workload("bwd_1m", 1, 1 << 20, 2, 1, 64, b, L, seed=20)
    NB = orc.num_blocks(w.n, b)
    assert bf1.bwd_workspace_size(w.batch, w.n, w.Hq, w.Hkv, w.d, b, L) > 1 << 31
    q_blocks = [0, 1, 4097, NB - 1]
    kv_blocks = [0, 2, 8191, NB - 1]
    TP.say(f"backward n = {w.n}: q blocks {q_blocks}, kv blocks {kv_blocks}")
    (dq, dk, dv), ref, terms = TB.run_case(w, q_blocks=q_blocks, kv_blocks=kv_blocks)
    for t in (dq, dk, dv):
        assert torch.isfinite(t).all()
    qrows, kvrows = TB._rows(q_blocks, b, w.n), TB._rows(kv_blocks, b, w.n)
    for name, got, r, t, rows in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref, terms, (qrows, kvrows, kvrows)):
        TB.check_bound(got, r, t, rows=rows, tag=f"n = {w.n} {name}")
