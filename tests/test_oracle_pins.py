"""Pins of the CPU oracle against references that do not share its code.

Each pin is chosen so that a plausible mistake in the oracle (a dropped term,
a wrong sign or index, a transposed operand, an off-by-one position) fails at
least one of them; tests/test_oracle_mutations.py plants such mistakes and
checks that they are caught.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_14498_amd import configs, inputs
from tests.pin_helpers import brute_force, hf_mrope, hf_qwen2

SMALL = configs.ModelShape(n_layers=2, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                           ffn_dim=96, vocab=97, dtype="f32")


def _setup(model=SMALL, P=(23,), Vis=(15,), S=(9,), index=7, norm="random", bias=True):
    w = configs.custom(model, P, Vis, S, index=index)
    W = inputs.make_weights(w, norm=norm, bias=bias).as_f32()
    bt = inputs.make_batch(w)
    return w, W, bt


def _seq(bt, b):
    cp, cs = bt.cu_prefix, bt.cu_suffix
    ids = bt.token_ids[cp[b]:cp[b + 1]]
    vo = sum(bt.visual_lens[:b])
    vis = inputs.to_f32(bt.visual[vo:vo + bt.visual_lens[b]])
    return ids, vis, bt.response_ids[cs[b]:cs[b + 1]]


# ----------------------------------------------------------------------------------------
# whole pipeline vs the transformers Qwen2 implementation (float64)
# ----------------------------------------------------------------------------------------
# The library forms RoPE angles in float32 (positions < 64 here: angle error ~1e-6 rad),
# so agreement is to ~1e-7 (observed: 2.4e-8 on log-probs, 1.1e-7 on keys), not to float64
# rounding.  Any of the mistakes planted in test_oracle_mutations.py moves results by >1e-3.
HF_TOL = 1e-6


@pytest.mark.parametrize("P,Vis,S", [((23,), (15,), (9,)), ((1,), (0,), (4,)), ((40,), (40,), (1,))])
def test_oracle_matches_hf_qwen2(P, Vis, S):
    w, W, bt = _setup(P=P, Vis=Vis, S=S)
    ids, vis, resp = _seq(bt, 0)
    lp_hf, keys, vals, h_hf = hf_qwen2(W, SMALL, ids, vis, resp)
    lp_unsplit = oracle.unsplit_logprob_one(W, SMALL, ids, vis, resp)
    K, V, h_last, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    lp_split = oracle.suffix_logprob_one(W, SMALL, K, V, h_last, resp)
    assert np.max(np.abs(lp_unsplit - lp_hf)) < HF_TOL
    assert np.max(np.abs(lp_split - lp_hf)) < HF_TOL
    for l in range(SMALL.n_layers):
        np.testing.assert_allclose(K[l], keys[l][:P[0]], atol=HF_TOL, rtol=0)
        np.testing.assert_allclose(V[l], vals[l][:P[0]], atol=HF_TOL, rtol=0)
    np.testing.assert_allclose(h_last, h_hf, atol=HF_TOL, rtol=0)


def test_oracle_matches_brute_force():
    tiny = configs.ModelShape(n_layers=2, d_model=8, n_q_heads=2, n_kv_heads=1, head_dim=4,
                              ffn_dim=6, vocab=11, dtype="f32")
    w, W, bt = _setup(model=tiny, P=(5,), Vis=(3,), S=(3,), index=3)
    ids, vis, resp = _seq(bt, 0)
    lp_bf = brute_force(W, tiny, ids, vis, resp)
    K, V, h, _ = oracle.prefix_forward_one(W, tiny, ids, vis)
    lp = oracle.suffix_logprob_one(W, tiny, K, V, h, resp)
    assert np.max(np.abs(lp - lp_bf)) < 1e-12


# ----------------------------------------------------------------------------------------
# split invariant: prefix + suffix == unsplit forward
# ----------------------------------------------------------------------------------------
@pytest.mark.parametrize("P,S", [(1, 0), (1, 1), (2, 2), (17, 5), (64, 16)])
def test_split_invariant(P, S):
    w, W, bt = _setup(P=(P,), Vis=(P // 2,), S=(S,), index=11)
    ids, vis, resp = _seq(bt, 0)
    K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    a = oracle.suffix_logprob_one(W, SMALL, K, V, h, resp)
    b = oracle.unsplit_logprob_one(W, SMALL, ids, vis, resp)
    assert a.shape == (S,)
    assert np.max(np.abs(a - b), initial=0.0) < 1e-10


# ----------------------------------------------------------------------------------------
# closed forms
# ----------------------------------------------------------------------------------------
def test_zero_lm_head_gives_uniform():
    w, W, bt = _setup(P=(7,), Vis=(3,), S=(5,))
    W.lm_head = np.zeros_like(W.lm_head)
    ids, vis, resp = _seq(bt, 0)
    K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    lp = oracle.suffix_logprob_one(W, SMALL, K, V, h, resp)
    assert np.all(lp == -math.log(SMALL.vocab))
    # the value quoted for the production vocabulary
    assert abs(-math.log(152064) - (-11.932056763842207)) < 1e-15
    assert abs(-math.log(2048) - (-7.6246189861593985)) < 1e-15


def test_scored_distribution_sums_to_one():
    # scoring every vocabulary id from the same boundary state gives a distribution
    w, W, bt = _setup(P=(9,), Vis=(4,), S=(1,))
    ids, vis, _ = _seq(bt, 0)
    _, _, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    z = np.repeat(np.asarray(h)[None, :], SMALL.vocab, axis=0)
    lp = oracle.score_rows(W, SMALL, z, np.arange(SMALL.vocab))
    assert abs(np.exp(lp).sum() - 1.0) < 1e-12
    assert np.all(lp < 0)


def test_identity_layers_reduce_to_log_softmax():
    """Wo = Wd = 0 make every layer the identity on the residual stream."""
    w, W, bt = _setup(P=(9,), Vis=(4,), S=(6,))
    for lw in W.layers:
        lw["wo"] = np.zeros_like(lw["wo"])
        lw["w_down"] = np.zeros_like(lw["w_down"])
    ids, vis, resp = _seq(bt, 0)
    K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    lp = oracle.suffix_logprob_one(W, SMALL, K, V, h, resp)
    E = torch.tensor(W.embed, dtype=torch.float64)
    last = torch.tensor(vis[-1], dtype=torch.float64) if ids[-1] < 0 else E[int(ids[-1])]
    rows = torch.cat([last[None], torch.nn.functional.embedding(torch.tensor(resp[:-1]).long(), E)])
    z = torch.nn.functional.rms_norm(rows, (SMALL.d_model,),
                                     torch.tensor(W.final_norm, dtype=torch.float64), SMALL.rms_eps)
    ref = torch.log_softmax(z @ torch.tensor(W.lm_head, dtype=torch.float64).T, dim=-1)
    ref = ref[torch.arange(len(resp)), torch.tensor(resp).long()].numpy()
    assert np.max(np.abs(lp - ref)) < 1e-12


def test_rmsnorm_constant_vector_and_library():
    d, eps = 64, 1e-6
    for c in (0.0, 1e-4, 0.5, -3.0):
        w = np.linspace(0.5, 1.5, d)
        got = oracle.rmsnorm(np.full((1, d), c), w, eps)[0]
        np.testing.assert_allclose(got, c / math.sqrt(c * c + eps) * w, rtol=1e-14, atol=0)
    x = np.random.default_rng(0).standard_normal((5, d))
    w = np.random.default_rng(1).standard_normal(d)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (d,), torch.tensor(w), eps).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, w, eps), ref, rtol=1e-13, atol=1e-14)


# ----------------------------------------------------------------------------------------
# RoPE
# ----------------------------------------------------------------------------------------
def test_rope_matches_complex_rotation():
    """Rotate-half RoPE is multiplication of (x_i + i x_{i+D/2}) by exp(i t f_i), f_i = theta^(-2i/D)."""
    rng = np.random.default_rng(5)
    D, theta = 16, 1e6
    x = rng.standard_normal((6, 3, D))
    pos = np.array([0, 1, 2, 100, 4095, 16383])
    got = oracle.apply_rope(x, oracle.rope_angles(pos, D, theta))
    for t in range(len(pos)):
        for h in range(3):
            for i in range(D // 2):
                f = theta ** (-(2 * i) / D)
                z = complex(x[t, h, i], x[t, h, i + D // 2]) * complex(math.cos(pos[t] * f),
                                                                      math.sin(pos[t] * f))
                assert abs(got[t, h, i] - z.real) < 1e-12
                assert abs(got[t, h, i + D // 2] - z.imag) < 1e-12


def test_rope_identities():
    rng = np.random.default_rng(6)
    D = 128
    q, k = rng.standard_normal((1, 1, D)), rng.standard_normal((1, 1, D))
    a0 = oracle.rope_angles([0], D, 1e6)
    np.testing.assert_array_equal(oracle.apply_rope(q, a0), q)          # position 0 = identity
    assert np.allclose(oracle.rope_angles([1], D, 1e6)[0, 0], 1.0)      # first pair turns 1 rad/step
    m, n, s = 37, 12, 1000
    r = lambda x, p: oracle.apply_rope(x, oracle.rope_angles([p], D, 1e6))
    for p in (m, n):                                                    # pair norms preserved
        x = r(q, p)[0, 0]
        half = D // 2
        np.testing.assert_allclose(x[:half] ** 2 + x[half:] ** 2,
                                   q[0, 0, :half] ** 2 + q[0, 0, half:] ** 2, rtol=1e-12)
    d1 = np.dot(r(q, m)[0, 0], r(k, n)[0, 0])                           # relative position
    d2 = np.dot(r(q, m + s)[0, 0], r(k, n + s)[0, 0])
    assert abs(d1 - d2) < 1e-10


# ----------------------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------------------
@pytest.mark.parametrize("nq,nk_past,Hq,Hkv", [(13, 0, 4, 2), (7, 21, 6, 2), (1, 0, 2, 2)])
def test_attention_matches_torch_sdpa(nq, nk_past, Hq, Hkv):
    rng = np.random.default_rng(nq + nk_past)
    D = 16
    q = rng.standard_normal((nq, Hq, D))
    k = rng.standard_normal((nk_past + nq, Hkv, D))
    v = rng.standard_normal((nk_past + nq, Hkv, D))
    qpos = nk_past + np.arange(nq)
    kpos = np.arange(nk_past + nq)
    got = oracle.attention(q, k, v, qpos, kpos)
    mask = torch.tensor(kpos[None, :] <= qpos[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).transpose(0, 1)[None], torch.tensor(k).transpose(0, 1)[None],
        torch.tensor(v).transpose(0, 1)[None], attn_mask=mask, enable_gqa=True)
    np.testing.assert_allclose(got, ref[0].transpose(0, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(9)
    v = rng.standard_normal((1, 1, 8))
    q = rng.standard_normal((1, 2, 8))
    out = oracle.attention(q, rng.standard_normal((1, 1, 8)), v, [0], [0])
    np.testing.assert_allclose(out[0, 0], v[0, 0])                      # one key: o = v0
    np.testing.assert_allclose(out[0, 1], v[0, 0])
    k = np.repeat(rng.standard_normal((1, 1, 8)), 6, axis=0)            # equal keys: mean of visible v
    v = rng.standard_normal((6, 1, 8))
    q = rng.standard_normal((6, 1, 8))
    out = oracle.attention(q, k, v, np.arange(6), np.arange(6))
    for t in range(6):
        np.testing.assert_allclose(out[t, 0], v[:t + 1, 0].mean(axis=0), rtol=1e-12)


def test_gqa_equals_replicated_mha():
    w, W, bt = _setup(P=(11,), Vis=(6,), S=(4,))
    ids, vis, resp = _seq(bt, 0)
    G = SMALL.group
    mha = configs.ModelShape(**{**SMALL.__dict__, "n_kv_heads": SMALL.n_q_heads})
    import copy
    W2 = copy.deepcopy(W)
    Dh = SMALL.head_dim
    for lw in W2.layers:
        for key in ("wk", "wv"):
            heads = lw[key].reshape(SMALL.n_kv_heads, Dh, -1)
            lw[key] = np.repeat(heads, G, axis=0).reshape(SMALL.n_q_heads * Dh, -1)
        for key in ("bk", "bv"):
            lw[key] = np.repeat(lw[key].reshape(SMALL.n_kv_heads, Dh), G, axis=0).reshape(-1)
    a = oracle.unsplit_logprob_one(W, SMALL, ids, vis, resp)
    b = oracle.unsplit_logprob_one(W2, mha, ids, vis, resp)
    assert np.max(np.abs(a - b)) < 1e-12


# ----------------------------------------------------------------------------------------
# multimodal RoPE (Qwen2.5-VL's 3-D positions for visual tokens; sections from the public
# model configuration, the paper being silent)
# ----------------------------------------------------------------------------------------
MROPE_SMALL = (2, 3, 3)  # sections of the Dh/2 = 8 pairs of SMALL


def video_positions(n_vis, n_text, grid, start=0):
    """3-D rotary positions of [visual block | text]: visual token (t, y, x) of a
    T x H x W grid at (start + 2t, start + y, start + x); text continues at one past the
    largest visual position with equal rows.  Returns (pos3 [3, n], next position)."""
    T, H, W = grid
    assert T * H * W == n_vis
    t, y, x = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    vis = np.stack([start + 2 * t.ravel(), start + y.ravel(), start + x.ravel()])
    nxt = int(vis.max()) + 1 if n_vis else start
    txt = np.tile(nxt + np.arange(n_text), (3, 1))
    return np.concatenate([vis, txt], axis=1).astype(np.int64), nxt + n_text


def test_mrope_with_equal_rows_is_rope():
    pos = np.array([0, 3, 17, 250])
    a = oracle.rope_angles_mrope(np.tile(pos, (3, 1)), 16, 1e6, MROPE_SMALL)
    np.testing.assert_array_equal(a, oracle.rope_angles(pos, 16, 1e6))


def test_mrope_matches_transformers_multimodal_rotary():
    rng = np.random.default_rng(11)
    for Dh, sec in ((16, MROPE_SMALL), (128, (16, 24, 24))):
        n = 13
        pos3 = rng.integers(0, 300, (3, n))
        q, k = rng.standard_normal((n, 4, Dh)), rng.standard_normal((n, 2, Dh))
        ang = oracle.rope_angles_mrope(pos3, Dh, 1e6, sec)
        qh, kh = hf_mrope(q, k, pos3, sec, 1e6)
        assert np.max(np.abs(oracle.apply_rope(q, ang) - qh)) < 1e-12
        assert np.max(np.abs(oracle.apply_rope(k, ang) - kh)) < 1e-12


def test_mrope_split_invariant():
    """Prefix over 3-D positions, then the response continuing at the prefix's next
    rotary position, equals the unsplit forward with the same positions."""
    w, W, bt = _setup(P=(21,), Vis=(12,), S=(7,), index=9)
    ids, vis, resp = _seq(bt, 0)
    pos3, nxt = video_positions(12, 9, (2, 2, 3))
    mr = (pos3, MROPE_SMALL)
    K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis, mrope=mr)
    lp = oracle.suffix_logprob_one(W, SMALL, K, V, h, resp, rope_start=nxt)
    lpu = oracle.unsplit_logprob_one(W, SMALL, ids, vis, resp, mrope=mr, rope_start=nxt)
    assert np.max(np.abs(lp - lpu)) < 1e-10
    # the multimodal positions matter
    K1, V1, h1, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    assert np.max(np.abs(K1 - K)) > 1e-3


# ----------------------------------------------------------------------------------------
# batching invariants and the decode step
# ----------------------------------------------------------------------------------------
def test_packed_batch_equals_each_alone_and_permutation():
    w, W, bt = _setup(P=(9, 1, 17), Vis=(5, 0, 16), S=(3, 0, 4), index=21)
    K, V, H = oracle.prefix_forward(W, SMALL, bt.cu_prefix, bt.token_ids, inputs.to_f32(bt.visual))
    lp = oracle.suffix_logprob(W, SMALL, bt.cu_prefix, bt.cu_suffix, K, V, H, bt.response_ids)
    lpu = oracle.unsplit_logprob(W, SMALL, bt.cu_prefix, bt.cu_suffix, bt.token_ids,
                                 inputs.to_f32(bt.visual), bt.response_ids)
    assert np.max(np.abs(lp - lpu)) < 1e-10
    for b in range(3):
        ids, vis, resp = _seq(bt, b)
        k, v, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
        cp = bt.cu_prefix
        np.testing.assert_array_equal(K[:, cp[b]:cp[b + 1]], k)
        np.testing.assert_array_equal(H[b], h)


def test_shared_prefix_suffixes_equal_unsplit_forward():
    """Shared prefixes (GRPO groups): every suffix scored against its group's one prefix
    pass equals the unsplit causal forward of [that prefix ; that response]."""
    w, W, bt = _setup(P=(9, 14, 5), Vis=(5, 10, 0), S=(3, 4, 2), index=23)
    K, V, H = oracle.prefix_forward(W, SMALL, bt.cu_prefix, bt.token_ids, inputs.to_f32(bt.visual))
    grp = np.array([1, 0, 1, 1, 2], np.int32)           # prefix 1 serves three responses
    lens = [4, 0, 6, 1, 3]
    cs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    resp = np.random.default_rng(5).integers(0, SMALL.vocab, int(cs[-1])).astype(np.int32)
    lp = oracle.suffix_logprob_grouped(W, SMALL, bt.cu_prefix, grp, cs, K, V, H, resp)
    for s_ in range(len(lens)):
        ids, vis, _ = _seq(bt, int(grp[s_]))
        ref = oracle.unsplit_logprob_one(W, SMALL, ids, vis, resp[cs[s_]:cs[s_ + 1]])
        assert np.max(np.abs(lp[cs[s_]:cs[s_ + 1]] - ref), initial=0.0) < 1e-10
    # suffixes of different prefixes differ (the pairing matters)
    lp_wrong = oracle.suffix_logprob_grouped(W, SMALL, bt.cu_prefix, np.zeros(5, np.int32), cs, K, V, H, resp)
    assert np.max(np.abs(lp_wrong[cs[2]:cs[3]] - lp[cs[2]:cs[3]])) > 1e-3


# ----------------------------------------------------------------------------------------
# prompt-token log-probabilities (teacher forcing over the prefix's own text tokens)
# ----------------------------------------------------------------------------------------
def _interleaved_prompt(bt, P, n_vis):
    """The batch's one prompt with its visual slots moved to the middle (text, visual, text),
    so that text tokens follow visual rows and visual rows follow text."""
    ids, vis, resp = _seq(bt, 0)
    text = ids[ids >= 0]
    a = len(text) // 3
    return np.concatenate([text[:a], np.full(n_vis, -1, np.int32), text[a:]]).astype(np.int32), vis, resp


def test_prompt_logprobs_match_transformers():
    w, W, bt = _setup(P=(26,), Vis=(9,), S=(3,), index=13)
    ids, vis, resp = _interleaved_prompt(bt, 26, 9)
    *_, logp = hf_qwen2(W, SMALL, ids, vis, resp, full_logp=True)
    lp = oracle.prompt_logprob_one(W, SMALL, ids, vis)
    scored = np.nonzero((ids >= 0) & (np.arange(26) > 0))[0]
    assert np.all(np.isnan(lp[np.setdiff1d(np.arange(26), scored)]))
    ref = np.array([logp[t - 1, ids[t]] for t in scored])
    assert np.max(np.abs(lp[scored] - ref)) < HF_TOL
    assert len(scored) == 26 - 9 - 1   # position 0 is text here


def test_prompt_logprobs_equal_response_scoring_of_the_same_tokens():
    # Scoring the prompt's text tail as a response over the shorter prefix gives the same values.
    w, W, bt = _setup(P=(30,), Vis=(14,), S=(2,), index=17)
    ids, vis, _ = _seq(bt, 0)
    lp = oracle.prompt_logprob_one(W, SMALL, ids, vis)
    for k in (14, 15, 22, 29):
        K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids[:k], vis)
        tail = oracle.suffix_logprob_one(W, SMALL, K, V, h, ids[k:])
        assert np.max(np.abs(lp[k:] - tail)) < 1e-10


def test_prompt_logprobs_packed_and_edge_cases():
    w, W, bt = _setup(P=(1, 9, 6, 5), Vis=(0, 4, 6, 0), S=(1, 1, 1, 1), index=19)
    lp = oracle.prompt_logprob(W, SMALL, bt.cu_prefix, bt.token_ids, inputs.to_f32(bt.visual))
    cu = bt.cu_prefix
    for b in range(4):
        ids, vis, _ = _seq(bt, b)
        np.testing.assert_array_equal(lp[cu[b]:cu[b + 1]], oracle.prompt_logprob_one(W, SMALL, ids, vis))
    assert np.isnan(lp[cu[0]])                      # a one-token prompt scores nothing
    assert np.all(np.isnan(lp[cu[2]:cu[3]]))        # an all-visual prompt scores nothing
    assert np.all(np.isfinite(lp[cu[3] + 1:cu[4]])) and np.all(lp[cu[3] + 1:cu[4]] < 0)


def test_prefix_is_response_independent():
    w, W, bt = _setup(P=(12,), Vis=(8,), S=(5,))
    ids, vis, resp = _seq(bt, 0)
    K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
    lp1 = oracle.suffix_logprob_one(W, SMALL, K, V, h, resp)
    resp2 = resp.copy()
    resp2[2:] = (resp2[2:] + 5) % SMALL.vocab
    lp2 = oracle.suffix_logprob_one(W, SMALL, K, V, h, resp2)
    # tokens before the change are scored identically, later ones are not
    np.testing.assert_array_equal(lp1[:2], lp2[:2])
    assert np.all(lp1[2:] != lp2[2:])


def test_decode_step_equals_suffix_of_length_two():
    w, W, bt = _setup(P=(10, 6), Vis=(7, 2), S=(2, 2), index=31)
    B, L = 2, SMALL.n_layers
    cap = 12
    ck = np.zeros((L, B, cap, SMALL.n_kv_heads, SMALL.head_dim))
    cv = np.zeros_like(ck)
    kv_len = np.array(bt.prefix_lens)
    toks = np.empty(B, np.int64)
    ref_lp = []
    for b in range(B):
        ids, vis, resp = _seq(bt, b)
        K, V, h, _ = oracle.prefix_forward_one(W, SMALL, ids, vis)
        ck[:, b, :len(ids)], cv[:, b, :len(ids)] = K, V
        toks[b] = resp[0]
        ref_lp.append(oracle.suffix_logprob_one(W, SMALL, K, V, h, resp)[1])
    logits, nxt, nk, nv = oracle.decode_step(W, SMALL, ck, cv, kv_len, toks)
    for b in range(B):
        resp = _seq(bt, b)[2]
        lp = logits[b] - (logits[b].max() + np.log(np.exp(logits[b] - logits[b].max()).sum()))
        assert abs(lp[resp[1]] - ref_lp[b]) < 1e-10
        assert nxt[b] == int(np.argmax(logits[b]))
