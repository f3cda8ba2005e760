"""GPU checks of the whole-model prefill stack of the timing study (§4.3,
§5.3): the stack with its attention on this library's kernels against the
fp64 oracle stack, on a small configuration with the same seeded weights.

Bar (derived from the arithmetic): the GPU stack keeps activations in bf16
(8 significant bits) and rounds after every operator, so the last-position
logits carry a relative error of order 2^-8 per operator and layer; three
layers stay well inside 5e-2 of the largest logit, while a wiring mistake
(head order, rotary phase, norm, route) moves logits by order one.  With a
route that covers every block the BF1 and dense layers give bitwise equal
logits (the kernels are bitwise equal there).
"""

import sys

import numpy as np
import pytest
import torch

from oracle import model_oracle as mo
from paper_2608_20427_amd import synth
from paper_2608_20427_amd.prefill_model import PrefillStack, middle_layers

pytestmark = pytest.mark.gpu

CFG = synth.ModelConfig(layers=3, hidden=256, heads=4, kv_heads=2, head_dim=64, intermediate=512, vocab=1000,
                        rope_theta=1.0e6, eps=1e-6)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def stack():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = synth.make_model_weights(CFG, 11)
    return PrefillStack(CFG, w, device="cuda"), {k: v.to(torch.float64).numpy() for k, v in w.items()}


@pytest.mark.parametrize("layers", ["dense", "middle", "all"])
@pytest.mark.parametrize("n", [700, 129])
def test_stack_matches_oracle(stack, layers, n):
    st, w64 = stack
    sel = {"dense": set(), "middle": middle_layers(CFG, 1), "all": set(range(CFG.layers))}[layers]
    ids = synth.make_tokens(CFG, n, 3 + n)
    got = st.last_logits(torch.from_numpy(ids).cuda(), sel).cpu().double().numpy()
    ref = mo.prefill_last_logits_fp64(ids, w64, CFG, sel, b=64, L=2)
    err = np.max(np.abs(got - ref))
    say(f"  stack {layers} n={n}: max |logit err| {err:.3e} (max |logit| {np.max(np.abs(ref)):.2f})")
    assert np.isfinite(got).all()
    assert err <= 5e-2 * np.max(np.abs(ref))


def test_covering_route_stack_is_bitwise_dense(stack):
    st, _ = stack
    ids = torch.from_numpy(synth.make_tokens(CFG, 256, 5)).cuda()   # 4 blocks of 64
    a = st.last_logits(ids, set())
    b = st.last_logits(ids, set(range(CFG.layers)))
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_bf1_layers_change_a_long_prefill(stack):
    st, _ = stack
    ids = torch.from_numpy(synth.make_tokens(CFG, 1500, 6)).cuda()
    a = st.last_logits(ids, set())
    b = st.last_logits(ids, set(range(CFG.layers)))
    torch.cuda.synchronize()
    assert not torch.equal(a, b)
