"""The longest sequence the interface accepts, n = 2^24 - 1 tokens (every
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
"""

import numpy as np
import pytest
import torch

import paper_2608_20427_amd as bf1
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
