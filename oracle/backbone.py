"""CPU oracle of the prefix/suffix backbone path.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or call this module; the product path never does.  It
shares no code with the HIP library and imports nothing but numpy.

What it computes.  The paper (Section "Observation and Opportunity") splits
every model invocation at the first response position: the prefix pass
(prompt prefill over visual + text tokens) depends only on the input and the
weights and leaves boundary KV state; the suffix pass continues from that
boundary and scores the response tokens (Section "Cross-Phase Execution",
Phases 1 and 2).  Prefix and suffix log-probabilities together are the
full-sequence values.  The split changes *when* work runs, not what it
computes, so the result is exactly the standard causal language-model
log-likelihood of each response token given the prompt and the earlier
response tokens.  That plain definition, for a Qwen2-style decoder backbone
(RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU MLP; the paper's
models are Qwen2.5-VL), is what this module writes out, in float64.

Readings where the paper is silent (listed with the rest in the design notes):
rotate-half RoPE pairing (i, i + Dh/2) with angles t * theta^(-2i/Dh) formed in
float64; 1-D positions 0..P-1 for the prefix and P..P+S-1 for the suffix; q
head h reads kv head floor(h / G); attention scale 1/sqrt(Dh); no temperature
and no vocabulary masking; a final RMSNorm before an untied lm_head; the
response token j is scored from the hidden state at absolute position P-1+j,
so the prefix hands over that boundary state (h_last, before the final norm)
as its "prefix log-probability" output.

Parity pins live in tests/test_oracle_pins.py (independent Qwen2 library
implementation, torch scaled-dot-product attention and rms_norm, closed forms,
the split invariant, invariants over batching, brute force on tiny inputs).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


def _f(a):
    return None if a is None else np.asarray(a, dtype=F64)


# ----------------------------------------------------------------------------------------
# building blocks
# ----------------------------------------------------------------------------------------
def rmsnorm(x, w, eps):
    """RMSNorm: x / sqrt(mean(x^2) + eps) * w, per row."""
    x = _f(x)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * _f(w)


def silu(z):
    """SiLU z * sigmoid(z)."""
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def rope_angles(positions, head_dim: int, theta: float):
    """Angle t * theta^(-2i/Dh) for every position t and pair index i < Dh/2, in float64."""
    i = np.arange(head_dim // 2, dtype=F64)
    inv_freq = np.power(F64(theta), -2.0 * i / head_dim)
    return np.asarray(positions, dtype=F64)[:, None] * inv_freq[None, :]


def rope_angles_mrope(pos3, head_dim: int, theta: float, sections):
    """Multimodal RoPE angles: pair index i takes its position from row sec(i) of pos3
    [3, n] (temporal, height, width), where the Dh/2 pairs are split into consecutive
    sections of sizes sections[0..2]; angle = pos3[sec(i)] * theta^(-2i/Dh), float64.
    With the three rows equal this is rope_angles of that row."""
    pos3 = np.asarray(pos3, dtype=F64)
    assert pos3.shape[0] == 3 and sum(sections) == head_dim // 2
    sec = np.repeat(np.arange(3), sections)            # section of every pair index
    i = np.arange(head_dim // 2, dtype=F64)
    inv_freq = np.power(F64(theta), -2.0 * i / head_dim)
    return pos3[sec, :].T * inv_freq[None, :]


def apply_rope(x, angles):
    """Rotate-half RoPE on x [n, H, Dh]: pair (i, i + Dh/2) is rotated by angles[:, i]."""
    half = x.shape[-1] // 2
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q, k, v, q_pos, k_pos, chunk: int = 1024):
    """Grouped-query attention with the causal rule "key position <= query position".

    q [nq, Hq, Dh]; k, v [nk, Hkv, Dh]; q head h reads kv head h // (Hq/Hkv).
    Returns [nq, Hq, Dh].
    """
    q, k, v = _f(q), _f(k), _f(v)
    nq, Hq, Dh = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    q_pos = np.asarray(q_pos)
    k_pos = np.asarray(k_pos)
    scale = 1.0 / math.sqrt(Dh)
    out = np.empty((nq, Hq, Dh), dtype=F64)
    for c0 in range(0, nq, chunk):
        c1 = min(nq, c0 + chunk)
        visible = k_pos[None, :] <= q_pos[c0:c1, None]
        for h in range(Hq):
            g = h // G
            s = (q[c0:c1, h, :] @ k[:, g, :].T) * scale
            s = np.where(visible, s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            p = np.exp(s - m)
            p /= p.sum(axis=1, keepdims=True)
            out[c0:c1, h, :] = p @ v[:, g, :]
    return out


def log_softmax_gather(logits, ids):
    """lp_r = logits[r, ids[r]] - logsumexp(logits[r, :]), max-shifted."""
    logits = _f(logits)
    m = logits.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(logits - m).sum(axis=1))
    return logits[np.arange(len(ids)), np.asarray(ids)] - lse


# ----------------------------------------------------------------------------------------
# one decoder layer over new tokens, with optional past keys/values
# ----------------------------------------------------------------------------------------
def decoder_layer(x, lw: Dict, cfg, positions, past_k=None, past_v=None, past_pos=None, angles=None):
    """Pre-norm decoder block.  Returns (x_out, k_new, v_new) with k_new post-RoPE.

    x [n, d] at absolute positions ``positions`` (token order: the causal rule);
    past_k/v [np, Hkv, Dh] are keys/values (post-RoPE) of earlier positions
    ``past_pos``.  RoPE rotates by ``angles`` [n, Dh/2] when given (multimodal
    positions), else by the 1-D angles of ``positions``.
    """
    n = x.shape[0]
    Hq, Hkv, Dh = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    h = rmsnorm(x, lw["attn_norm"], cfg.rms_eps)
    q = h @ _f(lw["wq"]).T
    k = h @ _f(lw["wk"]).T
    v = h @ _f(lw["wv"]).T
    if lw.get("bq") is not None:
        q = q + _f(lw["bq"])
    if lw.get("bk") is not None:
        k = k + _f(lw["bk"])
    if lw.get("bv") is not None:
        v = v + _f(lw["bv"])
    ang = rope_angles(positions, Dh, cfg.rope_theta) if angles is None else angles
    q = apply_rope(q.reshape(n, Hq, Dh), ang)
    k = apply_rope(k.reshape(n, Hkv, Dh), ang)
    v = v.reshape(n, Hkv, Dh)
    if past_k is not None and len(past_k):
        K = np.concatenate([_f(past_k), k], axis=0)
        V = np.concatenate([_f(past_v), v], axis=0)
        kpos = np.concatenate([np.asarray(past_pos), np.asarray(positions)])
    else:
        K, V, kpos = k, v, np.asarray(positions)
    o = attention(q, K, V, positions, kpos).reshape(n, Hq * Dh)
    x = x + o @ _f(lw["wo"]).T
    h2 = rmsnorm(x, lw["mlp_norm"], cfg.rms_eps)
    a = silu(h2 @ _f(lw["w_gate"]).T) * (h2 @ _f(lw["w_up"]).T)
    x = x + a @ _f(lw["w_down"]).T
    return x, k, v


def embed_prefix(embed, token_ids, visual):
    """Row t is embed[id_t] for a text id, else the next unused visual row (slot order)."""
    ids = np.asarray(token_ids)
    vis_slot = ids < 0
    nvis = int(vis_slot.sum())
    x = np.empty((len(ids), embed.shape[1]), dtype=F64)
    x[~vis_slot] = _f(embed[ids[~vis_slot]])
    if nvis:
        x[vis_slot] = _f(visual[:nvis])
    return x, nvis


# ----------------------------------------------------------------------------------------
# single sequence: prefix pass, suffix pass, unsplit forward
# ----------------------------------------------------------------------------------------
def prefix_forward_one(weights, cfg, token_ids, visual, mrope=None):
    """Prefix pass of one sequence (Section "Observation and Opportunity"; Phase 1).

    Returns (K, V, h_last, hidden): K, V [L, P, Hkv, Dh] post-RoPE keys and
    values of every prefix position, h_last [d] the residual stream at the last
    prefix position after the last layer (before the final norm), hidden [P, d].
    mrope = (pos3 [3, P], sections) rotates by multimodal positions instead of 0..P-1.
    """
    x, _ = embed_prefix(weights.embed, token_ids, visual)
    P = x.shape[0]
    pos = np.arange(P)
    ang = None if mrope is None else rope_angles_mrope(mrope[0], cfg.head_dim, cfg.rope_theta, mrope[1])
    Ks, Vs = [], []
    for lw in weights.layers:
        x, k, v = decoder_layer(x, lw, cfg, pos, angles=ang)
        Ks.append(k)
        Vs.append(v)
    return np.stack(Ks), np.stack(Vs), x[P - 1].copy(), x


def prompt_logprob_one(weights, cfg, token_ids, visual, mrope=None):
    """Teacher-forced log-probabilities of the prompt's own text tokens (the prefix-side
    log-probabilities of Section "Cross-Phase Execution": they depend on the prompt and
    the weights only, so the prefix pass can produce them).

    Entry t is log p(id_t | tokens before t), scored like a response token from the
    final hidden state one position earlier (row t-1 of the prefix pass), for every
    text token (id_t >= 0) after position 0.  NaN at position 0 and at visual slots:
    the model predicts no visual embedding.
    """
    ids = np.asarray(token_ids)
    out = np.full(len(ids), np.nan)
    t = np.nonzero(ids[1:] >= 0)[0] + 1
    if len(t) == 0:
        return out
    _, _, _, x = prefix_forward_one(weights, cfg, ids, visual, mrope)
    out[t] = score_rows(weights, cfg, x[t - 1], ids[t])
    return out


def score_rows(weights, cfg, z, ids):
    """Final RMSNorm, lm_head, and log-probability of ids under each row of z."""
    h = rmsnorm(z, weights.final_norm, cfg.rms_eps)
    out = np.empty(len(ids), dtype=F64)
    for r0 in range(0, len(ids), 256):
        logits = h[r0:r0 + 256] @ _f(weights.lm_head).T
        out[r0:r0 + 256] = log_softmax_gather(logits, ids[r0:r0 + 256])
    return out


def suffix_logprob_one(weights, cfg, K, V, h_last, response_ids, rope_start=None):
    """Suffix pass of one sequence (Phase 2): log p(r_j | prefix, r_<j) for every j.

    Response token j runs at position P + j and sees every prefix key (K, V from
    the prefix pass) and the response keys 0..j.  Token r_j is scored from the
    hidden state one position earlier: h_last for j = 0, else response row j-1.
    RoPE rotates token j by position rope_start + j (default P; after a prefix with
    multimodal positions, the prefix's next rotary position: text tokens have equal
    temporal, height and width positions, i.e. plain 1-D RoPE).
    """
    S = len(response_ids)
    if S == 0:
        return np.zeros(0, dtype=F64)
    P = K.shape[1]
    y = _f(weights.embed[np.asarray(response_ids)])
    pos = P + np.arange(S)
    ppos = np.arange(P)
    r0 = P if rope_start is None else int(rope_start)
    ang = rope_angles(r0 + np.arange(S), cfg.head_dim, cfg.rope_theta)
    for l, lw in enumerate(weights.layers):
        y, _, _ = decoder_layer(y, lw, cfg, pos, K[l], V[l], ppos, angles=ang)
    z = np.concatenate([_f(h_last)[None, :], y[:S - 1]], axis=0)
    return score_rows(weights, cfg, z, np.asarray(response_ids))


def unsplit_logprob_one(weights, cfg, token_ids, visual, response_ids, mrope=None, rope_start=None):
    """Causal forward over [prefix ; response] in one pass; lp_j from position P-1+j.
    With mrope = (pos3 [3, P], sections) the prefix rotates by multimodal positions and
    response token j by (rope_start + j) in all three rows."""
    xp, _ = embed_prefix(weights.embed, token_ids, visual)
    P, S = xp.shape[0], len(response_ids)
    x = np.concatenate([xp, _f(weights.embed[np.asarray(response_ids)])], axis=0)
    pos = np.arange(P + S)
    ang = None
    if mrope is not None:
        r0 = P if rope_start is None else int(rope_start)
        rows = np.concatenate([np.asarray(mrope[0]), np.tile(r0 + np.arange(S), (3, 1))], axis=1)
        ang = rope_angles_mrope(rows, cfg.head_dim, cfg.rope_theta, mrope[1])
    for lw in weights.layers:
        x, _, _ = decoder_layer(x, lw, cfg, pos, angles=ang)
    return score_rows(weights, cfg, x[P - 1:P - 1 + S], np.asarray(response_ids))


# ----------------------------------------------------------------------------------------
# packed batches (cu_seqlens)
# ----------------------------------------------------------------------------------------
def prefix_forward(weights, cfg, cu_prefix, token_ids, visual, seqs: Optional[Sequence[int]] = None):
    """Packed prefix pass.  Returns (K, V [L, T, Hkv, Dh], h_last [B, d]) in float64.

    Sequences not listed in ``seqs`` (default: all) are left as NaN.
    """
    cu = np.asarray(cu_prefix)
    B, T = len(cu) - 1, int(cu[-1])
    L = len(weights.layers)
    K = np.full((L, T, cfg.n_kv_heads, cfg.head_dim), np.nan)
    V = np.full_like(K, np.nan)
    H = np.full((B, cfg.d_model), np.nan)
    ids = np.asarray(token_ids)
    vis_start = np.concatenate([[0], np.cumsum([(ids[cu[b]:cu[b + 1]] < 0).sum() for b in range(B)])])
    for b in (range(B) if seqs is None else seqs):
        ib = ids[cu[b]:cu[b + 1]]
        vb = visual[vis_start[b]:vis_start[b + 1]]
        k, v, h, _ = prefix_forward_one(weights, cfg, ib, vb)
        K[:, cu[b]:cu[b + 1]] = k
        V[:, cu[b]:cu[b + 1]] = v
        H[b] = h
    return K, V, H


def prompt_logprob(weights, cfg, cu_prefix, token_ids, visual, seqs: Optional[Sequence[int]] = None):
    """Packed prompt-token log-probabilities [T] (prompt_logprob_one per sequence; NaN at
    each sequence's first token, at visual slots and for sequences not in ``seqs``)."""
    cu = np.asarray(cu_prefix)
    B = len(cu) - 1
    ids = np.asarray(token_ids)
    out = np.full(int(cu[-1]), np.nan)
    vis_start = np.concatenate([[0], np.cumsum([(ids[cu[b]:cu[b + 1]] < 0).sum() for b in range(B)])])
    for b in (range(B) if seqs is None else seqs):
        out[cu[b]:cu[b + 1]] = prompt_logprob_one(weights, cfg, ids[cu[b]:cu[b + 1]],
                                                  visual[vis_start[b]:vis_start[b + 1]])
    return out


def suffix_logprob(weights, cfg, cu_prefix, cu_suffix, K, V, h_last, response_ids,
                   seqs: Optional[Sequence[int]] = None):
    """Packed suffix pass: logprobs [R] in suffix order (NaN for sequences not in seqs)."""
    cp, cs = np.asarray(cu_prefix), np.asarray(cu_suffix)
    B, R = len(cp) - 1, int(cs[-1])
    out = np.full(R, np.nan)
    rid = np.asarray(response_ids)
    for b in (range(B) if seqs is None else seqs):
        out[cs[b]:cs[b + 1]] = suffix_logprob_one(
            weights, cfg, K[:, cp[b]:cp[b + 1]], V[:, cp[b]:cp[b + 1]], h_last[b],
            rid[cs[b]:cs[b + 1]])
    return out


def suffix_logprob_grouped(weights, cfg, cu_prefix, prefix_of_suffix, cu_suffix, K, V, h_last, response_ids):
    """Shared-prefix suffix pass (Section "Prefix Sharing": the responses of a GRPO group
    reuse their group's one prefix pass).  Suffix s is scored against prefix
    prefix_of_suffix[s]: its KV rows and its boundary state.  Returns logprobs [R]."""
    cp, cs = np.asarray(cu_prefix), np.asarray(cu_suffix)
    grp = np.asarray(prefix_of_suffix)
    out = np.empty(int(cs[-1]))
    rid = np.asarray(response_ids)
    for s in range(len(cs) - 1):
        p = int(grp[s])
        out[cs[s]:cs[s + 1]] = suffix_logprob_one(
            weights, cfg, K[:, cp[p]:cp[p + 1]], V[:, cp[p]:cp[p + 1]], h_last[p], rid[cs[s]:cs[s + 1]])
    return out


def unsplit_logprob(weights, cfg, cu_prefix, cu_suffix, token_ids, visual, response_ids):
    cp, cs = np.asarray(cu_prefix), np.asarray(cu_suffix)
    B = len(cp) - 1
    ids = np.asarray(token_ids)
    out = np.empty(int(cs[-1]))
    vo = 0
    for b in range(B):
        ib = ids[cp[b]:cp[b + 1]]
        nv = int((ib < 0).sum())
        out[cs[b]:cs[b + 1]] = unsplit_logprob_one(weights, cfg, ib, visual[vo:vo + nv],
                                                   np.asarray(response_ids)[cs[b]:cs[b + 1]])
        vo += nv
    return out


# ----------------------------------------------------------------------------------------
# decode step (the rollout side of the co-location workload)
# ----------------------------------------------------------------------------------------
def decode_step(weights, cfg, cache_k, cache_v, kv_len, token_ids):
    """One greedy decode step for B sequences.

    cache_k/v [L, B, cap, Hkv, Dh] hold post-RoPE keys/values of positions
    0..kv_len[b]-1.  The new token of sequence b runs at position kv_len[b],
    attends to those keys and itself, and the next id is the argmax of its
    logits (lowest id on ties).  Returns (logits [B, V], next_ids [B],
    new_k, new_v [L, B, Hkv, Dh]).
    """
    B = len(token_ids)
    L = len(weights.layers)
    logits = np.empty((B, weights.lm_head.shape[0]))
    nk = np.empty((L, B, cfg.n_kv_heads, cfg.head_dim))
    nv = np.empty_like(nk)
    for b in range(B):
        n = int(kv_len[b])
        x = _f(weights.embed[[int(token_ids[b])]])
        for l, lw in enumerate(weights.layers):
            x, k, v = decoder_layer(x, lw, cfg, np.array([n]), cache_k[l, b, :n], cache_v[l, b, :n],
                                    np.arange(n))
            nk[l, b], nv[l, b] = k[0], v[0]
        h = rmsnorm(x, weights.final_norm, cfg.rms_eps)
        logits[b] = (h @ _f(weights.lm_head).T)[0]
    return logits, np.argmax(logits, axis=1).astype(np.int32), nk, nv
