"""Planted mistakes in the oracle (CPU only): each plausible slip -- a dropped
route term, a wrong offset, a strict diagonal, a wrong scale, a wrong GQA map,
a dropped log-sum-exp term -- must make at least one pin fail.  This checks
that the pins are sharp enough to trust the oracle."""

import numpy as np
import pytest

import test_oracle_attention as TA
import test_oracle_route as TR
import test_oracle_variants as TV
from oracle import bf1_oracle as orc

_route = orc.route


def route_no_global(j, L=2):
    return [i for i in _route(j, L) if i != 0 or j == 0]


def route_dyadic_from_8(j, L=2):
    out = set(_route(j, L))
    if j >= 4 and 4 > L:
        out.discard(j - 4)
    return sorted(out)


def route_extra_j3(j, L=2):
    out = set(_route(j, L))
    if j >= 3:
        out.add(j - 3)
    return sorted(out)


def run_pins(pins):
    """Return True if some pin fails under the current (mutated) oracle."""
    for fn, args in pins:
        try:
            fn(*args)
        except AssertionError:
            return True
    return False


ROUTE_PINS = [
    (TR.test_route_matches_hand_derived_eq1, ()),
    (TR.test_interaction_reduction_32k, ()),
    (TR.test_pairs_brute_force, (777, 2)),
]


@pytest.mark.parametrize("bad", [route_no_global, route_dyadic_from_8, route_extra_j3])
def test_route_mutations_are_caught(monkeypatch, bad):
    monkeypatch.setattr(orc, "route", bad)
    assert run_pins(ROUTE_PINS)


def softmax_no_max_shift_in_lse(x, vals):
    m = np.max(x, axis=-1, keepdims=True)
    lse = np.log(np.sum(np.exp(x - m), axis=-1, keepdims=True))   # forgot "+ m"
    w = np.exp(x - m - lse)
    return w @ vals, lse[..., 0]


def softmax_unnormalised(x, vals):
    m = np.max(x, axis=-1, keepdims=True)
    w = np.exp(x - m)
    return w @ vals, (m + np.log(np.sum(w, axis=-1, keepdims=True)))[..., 0]


ATTN_PINS = [
    (TA.test_oracle_equals_library_sdpa_on_hand_mask, (70, 4)),
    (TA.test_route_covering_every_block_is_dense_causal, (256, 64, 2)),
    (TA.test_zero_keys_closed_form, (777, 64, 2)),
    (TA.test_gqa_grouping_contiguous, ()),
]


@pytest.mark.parametrize("bad", [softmax_no_max_shift_in_lse, softmax_unnormalised])
def test_softmax_mutations_are_caught(monkeypatch, bad):
    monkeypatch.setattr(orc, "_softmax_rows", bad)
    assert run_pins(ATTN_PINS)


def test_strict_diagonal_is_caught(monkeypatch):
    real = orc.token_mask

    def strict(n, b, L=2, rows=None):
        m = real(n, b, L, rows)
        r = np.arange(n) if rows is None else np.asarray(rows)
        m[np.arange(len(r)), r] = False
        return m

    monkeypatch.setattr(orc, "token_mask", strict)
    assert run_pins([(TR.test_pairs_brute_force, (257, 2)), (TR.test_mask_is_causal_and_keeps_diagonal, ())])


def test_wrong_scale_is_caught(monkeypatch):
    real = orc.attn_csr_fp64
    monkeypatch.setattr(orc, "attn_csr_fp64",
                        lambda q, k, v, b, rp, ci, scale=None, blocks=None:
                        real(q, k, v, b, rp, ci, scale=1.0 / q.shape[-1], blocks=blocks))
    assert run_pins(ATTN_PINS)


def test_wrong_gqa_map_is_caught(monkeypatch):
    real = orc.attn_csr_fp64

    def interleaved(q, k, v, b, rp, ci, scale=None, blocks=None):
        # maps q-head h to kv-head h % Hkv instead of h // G
        Hq, Hkv = q.shape[1], k.shape[1]
        G = Hq // Hkv
        idx = [h % Hkv for h in range(Hq)]
        kk = np.repeat(k, 1, axis=1)[:, idx]
        vv = np.repeat(v, 1, axis=1)[:, idx]
        return real(q, kk, vv, b, rp, ci, scale=scale, blocks=blocks) if G > 1 else real(q, k, v, b, rp, ci, scale, blocks)

    monkeypatch.setattr(orc, "attn_csr_fp64", interleaved)
    assert run_pins([(TA.test_gqa_grouping_contiguous, ())])


# ---- backward: planted slips in the per-row-set gradient core -------------
import test_oracle_backward as TB  # noqa: E402

_bwd = orc._bwd_gathered


def _bwd_parts(qr, kr, vr, dor, allowed, scale):
    x = scale * (qr @ kr.T)
    x = np.where(allowed, x, -np.inf)
    p = np.exp(x - np.max(x, axis=1, keepdims=True))
    p /= np.sum(p, axis=1, keepdims=True)
    dp = dor @ vr.T
    delta = np.sum(p * dp, axis=1, keepdims=True)
    return p, dp, delta


def bwd_no_delta(qr, kr, vr, dor, allowed, scale, delta=None):
    p, dp, _ = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    ds = p * dp
    return scale * (ds @ kr), scale * (ds.T @ qr), p.T @ dor


def bwd_sign_flip(qr, kr, vr, dor, allowed, scale, delta=None):
    p, dp, delta = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    ds = p * (delta - dp)
    return scale * (ds @ kr), scale * (ds.T @ qr), p.T @ dor


def bwd_dk_unscaled(qr, kr, vr, dor, allowed, scale, delta=None):
    p, dp, delta = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    ds = p * (dp - delta)
    return scale * (ds @ kr), ds.T @ qr, p.T @ dor


def bwd_dv_transposed_weights(qr, kr, vr, dor, allowed, scale, delta=None):
    p, dp, delta = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    ds = p * (dp - delta)
    w = np.exp(np.where(allowed, scale * (qr @ kr.T), -np.inf))  # unnormalised weights
    return scale * (ds @ kr), scale * (ds.T @ qr), w.T @ dor


BWD_PINS = [
    (TB.test_backward_matches_finite_differences, (23, 4, 1, 2, 1)),
    (TB.test_backward_row_sum_invariants, ()),
    (TB.test_backward_zero_keys_closed_form, ()),
]


@pytest.mark.parametrize("bad", [bwd_no_delta, bwd_sign_flip, bwd_dk_unscaled,
                                 bwd_dv_transposed_weights])
def test_backward_mutations_are_caught(monkeypatch, bad):
    monkeypatch.setattr(orc, "_bwd_gathered", bad)
    assert run_pins(BWD_PINS)


# ---- backward error scale: planted slips in the term-magnitude sums --------
from conftest import read_golden  # noqa: E402


def terms_unscaled(qr, kr, vr, dor, allowed, scale, delta=None):
    # c dropped from the dQ and dK terms
    p, dp, delta = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    a = np.abs(p * (dp - delta))
    return a @ np.abs(kr), a.T @ np.abs(qr), p.T @ np.abs(dor)


def terms_p_for_ds(qr, kr, vr, dor, allowed, scale, delta=None):
    # |dS| replaced by P
    p, dp, delta = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    return scale * (p @ np.abs(kr)), scale * (p.T @ np.abs(qr)), p.T @ np.abs(dor)


def terms_pdp_without_p(qr, kr, vr, dor, allowed, scale, delta=None):
    # P dropped from the cancellation scale P (|dP| + |D|)
    p, dp, delta = _bwd_parts(qr, kr, vr, dor, allowed, scale)
    a = np.where(allowed, np.abs(dp) + np.abs(delta), 0.0)
    return scale * (a @ np.abs(kr)), scale * (a.T @ np.abs(qr)), np.zeros((kr.shape[0], dor.shape[1]))


TERM_PINS = [
    (TB.test_abs_terms_hand_worked, (read_golden,)),
    (TB.test_abs_terms_dv_attained_for_nonnegative_upstream, ()),
    (TB.test_abs_terms_dq_attained_for_one_sign_per_row, ()),
]


@pytest.mark.parametrize("name,bad", [("_bwd_abs_terms", terms_unscaled),
                                      ("_bwd_abs_terms", terms_p_for_ds),
                                      ("_bwd_abs_terms_pdp", terms_pdp_without_p)])
def test_backward_error_scale_mutations_are_caught(monkeypatch, name, bad):
    monkeypatch.setattr(orc, name, bad)
    assert run_pins(TERM_PINS)


# ---------------------------------------------------------------------------
# Route variants and the depth search
# ---------------------------------------------------------------------------

_splitmix = orc.splitmix64


def sliding_one_too_wide(j, L=2):
    size = len(_route(j, L)) + 1
    return list(range(max(0, j - size + 1), j + 1))


def sliding_skips_self(j, L=2):
    size = len(_route(j, L))
    return list(range(j - size, j)) if j >= size else list(range(j + 1))


def random_half_open_draw(j, L=2, seed=17):
    local = [i for i in range(j - L, j + 1) if i >= 0]
    k = len(_route(j, L)) - len(local)
    taken = set()
    for t in range(k):
        r = j - L - k + t
        x = ((_splitmix(seed, (j << 20) + t) >> 32) * r) >> 32     # [0, r) instead of [0, r]
        taken.add(r if x in taken else x)
    return sorted(taken | set(local))


def random_drops_locals(j, L=2, seed=17):
    row = _random(j, L, seed)
    return sorted(set(row) - {j - 1})


def splitmix_wrong_shift(seed, c):
    z = (seed + (c + 1) * 0x9E3779B97F4A7C15) & ((1 << 64) - 1)
    z = ((z ^ (z >> 31)) * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & ((1 << 64) - 1)
    return z ^ (z >> 31)


_random = orc.route_static_random

VARIANT_PINS = [
    (TV.test_splitmix64_published_outputs, ()),
    (TV.test_sliding_hand_rows, ()),
    (TV.test_depth_golden, ("sliding", "512", "2", "59")),
    (TV.test_variant_pairs_equal_bf1_and_mask, ("sliding", 777, 16, 2)),
    (TV.test_variant_pairs_equal_bf1_and_mask, ("static_random", 777, 16, 2)),
    (TV.test_variant_rows_valid, (2,)),
    (TV.test_static_random_is_uniform_over_candidates, ()),
]


@pytest.mark.parametrize("name,bad", [("route_sliding", sliding_one_too_wide),
                                      ("route_sliding", sliding_skips_self),
                                      ("route_static_random", random_half_open_draw),
                                      ("route_static_random", random_drops_locals),
                                      ("splitmix64", splitmix_wrong_shift)])
def test_variant_mutations_are_caught(monkeypatch, name, bad):
    monkeypatch.setattr(orc, name, bad)
    assert run_pins(VARIANT_PINS)


def bfs_off_by_one(rows):
    return _depth_rows(rows) + 1


_depth_rows = orc._max_shortest_path_rows


def test_depth_mutation_is_caught(monkeypatch):
    monkeypatch.setattr(orc, "_max_shortest_path_rows", bfs_off_by_one)
    assert run_pins([(TV.test_depth_bfs_matches_minplus, ("sliding", 40, 2)),
                     (TV.test_depth_golden, ("bf1", "512", "2", "8"))])


# ---------------------------------------------------------------------------
# Decode
# ---------------------------------------------------------------------------

import test_oracle_decode as TD

_decode = orc.attn_decode_fp64
_decode_plan = orc.decode_plan


def decode_previous_row(q, k, v, seq_lens, b, L=2, scale=None):
    # reads the keys of row t - 1 (a stale mask row) for sequences longer than one token
    return _decode(q, k, v, [max(1, int(n) - 1) for n in seq_lens], b, L, scale)


def decode_plan_with_self(seq_len, page_row, b, L=2, dense=False):
    j, earlier = _decode_plan(seq_len, page_row, b, L, dense)
    return j, earlier + [int(page_row[j])]


def decode_plan_next_block(seq_len, page_row, b, L=2, dense=False):
    return _decode_plan(seq_len + b, page_row, b, L, dense)


DECODE_PINS = [
    (TD.test_decode_equals_last_row_of_full_mask_forward, (16, 2)),
    (TD.test_decode_zero_keys_closed_form, (1000,)),
    (TD.test_decode_plan_counts_and_mapping, (2,)),
]


@pytest.mark.parametrize("name,bad", [("attn_decode_fp64", decode_previous_row),
                                      ("decode_plan", decode_plan_with_self),
                                      ("decode_plan", decode_plan_next_block)])
def test_decode_mutations_are_caught(monkeypatch, name, bad):
    monkeypatch.setattr(orc, name, bad)
    assert run_pins(DECODE_PINS)


# ---------------------------------------------------------------------------
# Whole-model prefill oracle
# ---------------------------------------------------------------------------

import test_oracle_model as TM
from oracle import model_oracle as mo

_rope = mo.rope
_rms = mo.rms_norm


def rope_sign_flip(x, theta):
    n, _, d = x.shape
    half = d // 2
    inv = theta ** (-np.arange(0, d, 2, dtype=np.float64) / d)
    ang = np.arange(n, dtype=np.float64)[:, None] * inv[None, :]
    cos = np.concatenate([np.cos(ang), np.cos(ang)], axis=-1)[:, None, :]
    sin = np.concatenate([np.sin(ang), np.sin(ang)], axis=-1)[:, None, :]
    rotated = np.concatenate([x[..., half:], -x[..., :half]], axis=-1)     # wrong sign
    return x * cos + rotated * sin


def rms_without_eps_gain(x, w, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)       # gain dropped


def relu_not_silu(x):
    return np.maximum(x, 0.0)


MODEL_PINS = [(TM.test_dense_stack_matches_transformers_qwen3, (37,))]


@pytest.mark.parametrize("name,bad", [("rope", rope_sign_flip), ("rms_norm", rms_without_eps_gain),
                                      ("silu", relu_not_silu)])
def test_model_mutations_are_caught(monkeypatch, name, bad):
    monkeypatch.setattr(mo, name, bad)
    assert run_pins(MODEL_PINS)
