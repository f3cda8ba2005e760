"""Pins of the whole-model prefill oracle (CPU only): the decoder stack of the
timing study (§4.1, §4.3, §5.3).

* Dense configuration against an independent implementation of the same
  architecture: the transformers library's Qwen3 model in float64, loaded
  with the same weights (eager attention on the CPU).  A slip in a norm, the
  rotary embedding, the head grouping, the MLP or the tied output head makes
  the logits disagree.
* BF1 layers with a route that covers every block (n <= (L + 2) b) equal the
  dense configuration; with a longer sequence they differ (the route is used).
"""

import numpy as np
import pytest
import torch

from oracle import model_oracle as mo
from paper_2608_20427_amd import synth

TINY = synth.ModelConfig(layers=3, hidden=96, heads=4, kv_heads=2, head_dim=16, intermediate=160, vocab=300,
                         rope_theta=1.0e4, eps=1e-6)


def _weights(cfg, seed):
    return {k: v.to(torch.float64).numpy() for k, v in synth.make_model_weights(cfg, seed).items()}


def _hf_logits(cfg, w, ids):
    from transformers import Qwen3Config, Qwen3ForCausalLM
    hc = Qwen3Config(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.intermediate,
                     num_hidden_layers=cfg.layers, num_attention_heads=cfg.heads,
                     num_key_value_heads=cfg.kv_heads, head_dim=cfg.head_dim, rms_norm_eps=cfg.eps,
                     rope_parameters={"rope_type": "default", "rope_theta": cfg.rope_theta},
                     tie_word_embeddings=True, attention_bias=False, max_position_embeddings=4096,
                     attn_implementation="eager")
    m = Qwen3ForCausalLM(hc).to(torch.float64).eval()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(w["embed"]))
        m.model.norm.weight.copy_(t(w["final_norm"]))
        for l, layer in enumerate(m.model.layers):
            p = f"{l}."
            layer.input_layernorm.weight.copy_(t(w[p + "in_norm"]))
            layer.post_attention_layernorm.weight.copy_(t(w[p + "post_norm"]))
            at = layer.self_attn
            at.q_proj.weight.copy_(t(w[p + "wq"].T))
            at.k_proj.weight.copy_(t(w[p + "wk"].T))
            at.v_proj.weight.copy_(t(w[p + "wv"].T))
            at.o_proj.weight.copy_(t(w[p + "wo"].T))
            at.q_norm.weight.copy_(t(w[p + "q_norm"]))
            at.k_norm.weight.copy_(t(w[p + "k_norm"]))
            layer.mlp.gate_proj.weight.copy_(t(w[p + "wg"].T))
            layer.mlp.up_proj.weight.copy_(t(w[p + "wu"].T))
            layer.mlp.down_proj.weight.copy_(t(w[p + "wd"].T))
        assert m.lm_head.weight.data_ptr() == m.model.embed_tokens.weight.data_ptr()
        out = m(input_ids=torch.from_numpy(np.asarray(ids))[None]).logits
    return out[0, -1].numpy()


@pytest.mark.parametrize("n", [1, 37, 200])
def test_dense_stack_matches_transformers_qwen3(n):
    w = _weights(TINY, 3)
    ids = synth.make_tokens(TINY, n, 7)
    ours = mo.prefill_last_logits_fp64(ids, w, TINY, bf1_layers=set(), b=16, L=2)
    ref = _hf_logits(TINY, w, ids)
    # the library's RMSNorm computes in float32 even inside a float64 model
    # (about 1e-7 relative per norm); a wiring slip moves logits by O(1)
    assert np.max(np.abs(ours - ref)) < 2e-5 * np.max(np.abs(ref))


def test_bf1_layers_with_covering_route_equal_dense():
    w = _weights(TINY, 4)
    ids = synth.make_tokens(TINY, 64, 8)          # 4 blocks of 16: P(j) covers 0..j at L = 2
    dense = mo.prefill_last_logits_fp64(ids, w, TINY, set(), b=16, L=2)
    bf1 = mo.prefill_last_logits_fp64(ids, w, TINY, {0, 1, 2}, b=16, L=2)
    assert np.max(np.abs(dense - bf1)) < 1e-10 * np.max(np.abs(dense))


def test_bf1_layers_change_a_long_prefill():
    w = _weights(TINY, 5)
    ids = synth.make_tokens(TINY, 300, 9)
    dense = mo.prefill_last_logits_fp64(ids, w, TINY, set(), b=16, L=2)
    one = mo.prefill_last_logits_fp64(ids, w, TINY, {1}, b=16, L=2)
    assert np.max(np.abs(dense - one)) > 1e-6 * np.max(np.abs(dense))


def test_rope_is_a_rotation_with_relative_phase():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((50, 3, 16))
    y = mo.rope(x, 1.0e4)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    # <rope(q)_s, rope(k)_t> depends on t - s only
    q = np.repeat(rng.standard_normal((1, 1, 16)), 50, axis=0)
    k = np.repeat(rng.standard_normal((1, 1, 16)), 50, axis=0)
    rq, rk = mo.rope(q, 1.0e4), mo.rope(k, 1.0e4)
    d1 = np.sum(rq[10, 0] * rk[3, 0])
    d2 = np.sum(rq[30, 0] * rk[23, 0])
    assert abs(d1 - d2) < 1e-10
