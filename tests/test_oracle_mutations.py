"""Plant plausible mistakes in the oracle (on the CPU) and check that a pin catches each.

Every mutation replaces one oracle building block with a subtly wrong version
(a wrong pairing, sign, index, scale or position, a dropped term, a transposed
operand); the pins of test_oracle_pins.py must then fail.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import oracle.backbone as ob
from tests.pin_helpers import hf_qwen2
from tests.pin_helpers import hf_mrope
from tests.test_oracle_pins import HF_TOL, MROPE_SMALL, SMALL, _seq, _setup, video_positions


def _pins_hold() -> bool:
    """True iff every pin below still holds."""
    w, W, bt = _setup(P=(19,), Vis=(11,), S=(6,))
    ids, vis, resp = _seq(bt, 0)
    lp_hf, keys, _, _, logp = hf_qwen2(W, SMALL, ids, vis, resp, full_logp=True)
    K, V, h, _ = ob.prefix_forward_one(W, SMALL, ids, vis)
    lp = ob.suffix_logprob_one(W, SMALL, K, V, h, resp)
    lpu = ob.unsplit_logprob_one(W, SMALL, ids, vis, resp)
    ok = np.max(np.abs(lp - lp_hf)) < HF_TOL and np.max(np.abs(lpu - lp_hf)) < HF_TOL
    ok &= np.max(np.abs(K[0] - keys[0][:19])) < HF_TOL
    # constant-vector RMSNorm closed form
    c, eps, d = 1e-4, 1e-6, 8
    ok &= bool(np.allclose(ob.rmsnorm(np.full((1, d), c), np.ones(d), eps)[0], c / math.sqrt(c * c + eps)))
    # attention vs torch SDPA
    rng = np.random.default_rng(3)
    q, k, v = rng.standard_normal((5, 4, 8)), rng.standard_normal((5, 2, 8)), rng.standard_normal((5, 2, 8))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).transpose(0, 1)[None], torch.tensor(k).transpose(0, 1)[None],
        torch.tensor(v).transpose(0, 1)[None], is_causal=True, enable_gqa=True)[0].transpose(0, 1)
    got = ob.attention(q, k, v, np.arange(5), np.arange(5))
    ok &= bool(np.allclose(got, ref.numpy(), atol=1e-10))
    # multimodal RoPE vs transformers, and the split invariant with 3-D prefix positions
    pos3 = rng.integers(0, 300, (3, 7))
    qq, kk = rng.standard_normal((7, 4, 16)), rng.standard_normal((7, 2, 16))
    qh, _ = hf_mrope(qq, kk, pos3, MROPE_SMALL, 1e6)
    ok &= bool(np.max(np.abs(ob.apply_rope(qq, ob.rope_angles_mrope(pos3, 16, 1e6, MROPE_SMALL)) - qh)) < 1e-12)
    w2, W2, bt2 = _setup(P=(21,), Vis=(12,), S=(7,), index=9)
    ids2, vis2, resp2 = _seq(bt2, 0)
    p3, nxt = video_positions(12, 9, (2, 2, 3))
    K2, V2, h2, _ = ob.prefix_forward_one(W2, SMALL, ids2, vis2, mrope=(p3, MROPE_SMALL))
    lps = ob.suffix_logprob_one(W2, SMALL, K2, V2, h2, resp2, rope_start=nxt)
    lpu2 = ob.unsplit_logprob_one(W2, SMALL, ids2, vis2, resp2, mrope=(p3, MROPE_SMALL), rope_start=nxt)
    ok &= bool(np.max(np.abs(lps - lpu2)) < 1e-10)
    # prompt-token log-probabilities vs the library's teacher-forced log-softmax
    lpp = ob.prompt_logprob_one(W, SMALL, ids, vis)
    t = np.nonzero(ids >= 0)[0]
    t = t[t > 0]
    ok &= bool(np.max(np.abs(lpp[t] - logp[t - 1, ids[t]])) < HF_TOL)
    return bool(ok)


def _rope_interleaved(x, angles):
    c, s = np.cos(angles)[:, None, :], np.sin(angles)[:, None, :]
    out = x.copy()
    out[..., 0::2] = x[..., 0::2] * c - x[..., 1::2] * s
    out[..., 1::2] = x[..., 1::2] * c + x[..., 0::2] * s
    return out


def _rope_sign(x, angles):
    half = x.shape[-1] // 2
    c, s = np.cos(angles)[:, None, :], np.sin(angles)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)


def _rope_freq(positions, head_dim, theta):
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.asarray(positions, np.float64)[:, None] * np.power(theta, -i / head_dim)[None, :]


def _attention_mod(q, k, v, q_pos, k_pos, chunk=1024):
    Hq, Hkv = q.shape[1], k.shape[1]
    out = np.empty(q.shape)
    for h in range(Hq):
        g = h % Hkv
        s = (q[:, h] @ k[:, g].T) / math.sqrt(q.shape[2])
        s = np.where(np.asarray(k_pos)[None] <= np.asarray(q_pos)[:, None], s, -np.inf)
        p = np.exp(s - s.max(1, keepdims=True))
        out[:, h] = (p / p.sum(1, keepdims=True)) @ v[:, g]
    return out


def _attention_noscale(q, k, v, q_pos, k_pos, chunk=1024):
    return ORIG["attention"](q * math.sqrt(q.shape[2]), k, v, q_pos, k_pos)


def _attention_strict(q, k, v, q_pos, k_pos, chunk=1024):
    # excludes the key at the query's own position; first row falls back to itself
    qp = np.asarray(q_pos)
    out = ORIG["attention"](q, k, v, qp - 1, k_pos)
    first = qp == np.min(k_pos)
    if first.any():
        out[first] = ORIG["attention"](q[first], k, v, qp[first], k_pos)
    return out


def _rmsnorm_noeps(x, w, eps):
    return ORIG["rmsnorm"](x, w, 0.0)


def _silu_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def _layer_no_attn_residual(x, lw, cfg, positions, past_k=None, past_v=None, past_pos=None, angles=None):
    y, k, v = ORIG["decoder_layer"](x, lw, cfg, positions, past_k, past_v, past_pos, angles=angles)
    lw2 = dict(lw, w_down=np.zeros_like(lw["w_down"]))
    y_attn, _, _ = ORIG["decoder_layer"](x, lw2, cfg, positions, past_k, past_v, past_pos, angles=angles)
    return y - x, k, v  # residual input dropped


def _layer_wo_transposed(x, lw, cfg, positions, past_k=None, past_v=None, past_pos=None, angles=None):
    return ORIG["decoder_layer"](x, dict(lw, wo=np.ascontiguousarray(lw["wo"].T)), cfg, positions,
                                 past_k, past_v, past_pos, angles=angles)


def _suffix_shift(weights, cfg, K, V, h_last, response_ids, rope_start=None):
    S = len(response_ids)
    P = K.shape[1]
    y = np.asarray(weights.embed[np.asarray(response_ids)], np.float64)
    for l, lw in enumerate(weights.layers):
        y, _, _ = ob.decoder_layer(y, lw, cfg, P - 1 + np.arange(S), K[l], V[l], np.arange(P))
    z = np.concatenate([np.asarray(h_last)[None], y[:S - 1]])
    return ob.score_rows(weights, cfg, z, np.asarray(response_ids))


def _suffix_no_boundary(weights, cfg, K, V, h_last, response_ids, rope_start=None):
    S = len(response_ids)
    P = K.shape[1]
    y = np.asarray(weights.embed[np.asarray(response_ids)], np.float64)
    for l, lw in enumerate(weights.layers):
        y, _, _ = ob.decoder_layer(y, lw, cfg, P + np.arange(S), K[l], V[l], np.arange(P))
    return ob.score_rows(weights, cfg, y, np.asarray(response_ids))


def _mrope_sections_reversed(pos3, head_dim, theta, sections):
    return ORIG["rope_angles_mrope"](np.asarray(pos3)[::-1], head_dim, theta, tuple(sections)[::-1])


def _suffix_restarts_at_prefix_length(weights, cfg, K, V, h_last, response_ids, rope_start=None):
    return ORIG["suffix_logprob_one"](weights, cfg, K, V, h_last, response_ids)


def _prompt_from_own_row(weights, cfg, token_ids, visual, mrope=None):
    ids = np.asarray(token_ids)
    out = np.full(len(ids), np.nan)
    t = np.nonzero(ids[1:] >= 0)[0] + 1
    _, _, _, x = ob.prefix_forward_one(weights, cfg, ids, visual, mrope)
    out[t] = ob.score_rows(weights, cfg, x[t], ids[t])
    return out


ORIG = {n: getattr(ob, n) for n in ("attention", "rmsnorm", "decoder_layer", "apply_rope",
                                    "rope_angles", "rope_angles_mrope", "silu", "suffix_logprob_one")}

MUTATIONS = {
    "rope_interleaved_pairs": ("apply_rope", _rope_interleaved),
    "rope_wrong_sign": ("apply_rope", _rope_sign),
    "rope_wrong_frequency": ("rope_angles", _rope_freq),
    "gqa_head_modulo": ("attention", _attention_mod),
    "attention_unscaled": ("attention", _attention_noscale),
    "attention_excludes_self": ("attention", _attention_strict),
    "rmsnorm_without_eps": ("rmsnorm", _rmsnorm_noeps),
    "silu_is_sigmoid": ("silu", _silu_sigmoid),
    "residual_dropped": ("decoder_layer", _layer_no_attn_residual),
    "wo_transposed": ("decoder_layer", _layer_wo_transposed),
    "suffix_positions_off_by_one": ("suffix_logprob_one", _suffix_shift),
    "suffix_scores_from_own_row": ("suffix_logprob_one", _suffix_no_boundary),
    "mrope_sections_reversed": ("rope_angles_mrope", _mrope_sections_reversed),
    "mrope_suffix_restarts_at_prefix_length": ("suffix_logprob_one", _suffix_restarts_at_prefix_length),
    "prompt_scored_from_own_row": ("prompt_logprob_one", _prompt_from_own_row),
}


def test_pins_hold_unmutated():
    assert _pins_hold()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    fn, repl = MUTATIONS[name]
    monkeypatch.setattr(ob, fn, repl)
    assert not _pins_hold(), f"planted mistake {name} passed every pin"
