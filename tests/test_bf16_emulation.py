"""Pins of the bf16 rounding emulation (tests/bf16_emulation.py), which sets the floor a
bf16 case is held to when it misses the 2e-2 target.  With no rounding point it must be
the oracle; its rounding must be round-to-nearest-even to bfloat16; every point must
change the result; and the decode-step form must agree with the oracle's decode step."""
import numpy as np
import pytest

import oracle
from paper_2608_14498_amd import configs, inputs
from tests import bf16_emulation as em

MODEL = configs.ModelShape(n_layers=2, d_model=128, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=256,
                           vocab=512, dtype="bf16")


def _case():
    w = configs.custom(MODEL, [40], [30], [9], index=501)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    return w, hw, bt


def test_round_bf16_is_nearest_even():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ties = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8)], np.float32)  # halfway cases
    x = np.concatenate([x, ties])
    want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(x))
    assert np.array_equal(em.round_bf16(x), want.astype(np.float64))
    assert em.round_bf16(ties).tolist() == [1.0, 1.0 + 2.0 ** -6, -1.0]


def test_no_rounding_point_is_the_oracle():
    w, hw, bt = _case()
    W = hw.as_f32()
    vis = inputs.to_f32(bt.visual).astype(np.float64)
    K, V, h, _ = oracle.prefix_forward_one(W, MODEL, bt.token_ids, vis)
    ref = oracle.suffix_logprob_one(W, MODEL, K, V, h, bt.response_ids)
    got = em.forward_logprobs(W, MODEL, bt.token_ids, vis, bt.response_ids, em.Rounder("bf16", ()))
    assert np.max(np.abs(got - ref)) <= 1e-10


@pytest.mark.parametrize("point", em.POINTS)
def test_every_rounding_point_moves_the_result(point):
    w, hw, bt = _case()
    W = hw.as_f32()
    vis = inputs.to_f32(bt.visual).astype(np.float64)
    exact = em.forward_logprobs(W, MODEL, bt.token_ids, vis, bt.response_ids, em.Rounder("bf16", ()))
    one = em.forward_logprobs(W, MODEL, bt.token_ids, vis, bt.response_ids, em.Rounder("bf16", (point,)))
    d = np.max(np.abs(one - exact))
    assert 1e-7 < d < 0.1, (point, d)
    f16 = em.forward_logprobs(W, MODEL, bt.token_ids, vis, bt.response_ids, em.Rounder("f16", (point,)))
    assert np.max(np.abs(f16 - exact)) < d  # fp16 keeps 3 more mantissa bits


def test_decode_form_matches_oracle_decode_step():
    w, hw, bt = _case()
    W = hw.as_f32()
    dec = inputs.make_decode(w, batch=3, kv_len=np.array([0, 17, 40], np.int32), cap=48)
    ck, cv = inputs.to_f32(dec.cache_k), inputs.to_f32(dec.cache_v)
    lo, _, _, _ = oracle.decode_step(W, MODEL, ck, cv, dec.kv_len, dec.token_ids)
    got = em.decode_logits(W, MODEL, ck, cv, dec.kv_len, dec.token_ids, em.Rounder("bf16", ()))
    assert np.max(np.abs(got - lo)) <= 1e-10
    rounded = em.decode_logits(W, MODEL, ck, cv, dec.kv_len, dec.token_ids, em.Rounder("bf16", em.POINTS))
    assert 1e-6 < np.max(np.abs(rounded - lo)) < 0.1
