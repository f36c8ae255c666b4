"""Independent references used to pin the oracle (no code shared with it).

* ``hf_qwen2`` builds the transformers library's Qwen2 causal LM (the
  decoder family of the paper's Qwen2.5-VL models) in float64 with given
  weights and runs it over the unsplit sequence.
* ``brute_force`` is a scalar pure-Python forward written from the textbook
  definitions, for very small shapes.
"""
from __future__ import annotations

import math

import numpy as np
import torch


def hf_qwen2(weights, cfg, token_ids, visual, response_ids, full_logp=False):
    """Returns (logprobs [S], keys [L][P+S, Hkv, Dh], values, h_last_prefix [d]), and with
    full_logp the library's log-softmax over every position [P+S, V] as a fifth item."""
    from transformers import Qwen2Config, Qwen2ForCausalLM

    L = len(weights.layers)
    hc = Qwen2Config(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.ffn_dim,
                     num_hidden_layers=L, num_attention_heads=cfg.n_q_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     rope_theta=cfg.rope_theta, rms_norm_eps=cfg.rms_eps, tie_word_embeddings=False,
                     max_position_embeddings=8192, attn_implementation="eager")
    model = Qwen2ForCausalLM(hc).double().eval()
    t = lambda a: torch.tensor(np.asarray(a, np.float64))
    with torch.no_grad():
        model.model.embed_tokens.weight.copy_(t(weights.embed))
        model.lm_head.weight.copy_(t(weights.lm_head))
        model.model.norm.weight.copy_(t(weights.final_norm))
        for layer, lw in zip(model.model.layers, weights.layers):
            a = layer.self_attn
            a.q_proj.weight.copy_(t(lw["wq"]))
            a.k_proj.weight.copy_(t(lw["wk"]))
            a.v_proj.weight.copy_(t(lw["wv"]))
            for lin, key in ((a.q_proj, "bq"), (a.k_proj, "bk"), (a.v_proj, "bv")):
                lin.bias.copy_(t(lw[key]) if lw.get(key) is not None else torch.zeros_like(lin.bias))
            a.o_proj.weight.copy_(t(lw["wo"]))
            layer.mlp.gate_proj.weight.copy_(t(lw["w_gate"]))
            layer.mlp.up_proj.weight.copy_(t(lw["w_up"]))
            layer.mlp.down_proj.weight.copy_(t(lw["w_down"]))
            layer.input_layernorm.weight.copy_(t(lw["attn_norm"]))
            layer.post_attention_layernorm.weight.copy_(t(lw["mlp_norm"]))
    ids = np.asarray(token_ids)
    P, S = len(ids), len(response_ids)
    emb = model.model.embed_tokens.weight
    rows = []
    vi = 0
    for i in ids:
        if i < 0:
            rows.append(t(visual[vi]))
            vi += 1
        else:
            rows.append(emb[int(i)])
    for r in response_ids:
        rows.append(emb[int(r)])
    x = torch.stack(rows)[None]
    captured = {}
    hook = model.model.layers[-1].register_forward_hook(
        lambda mod, inp, out: captured.__setitem__("h", out[0] if isinstance(out, tuple) else out))
    with torch.no_grad():
        out = model(inputs_embeds=x, use_cache=True)
    hook.remove()
    logp = torch.log_softmax(out.logits[0], dim=-1)
    lp = np.array([float(logp[P - 1 + j, int(response_ids[j])]) for j in range(S)])
    keys = [out.past_key_values.layers[l].keys[0].transpose(0, 1).numpy() for l in range(L)]
    vals = [out.past_key_values.layers[l].values[0].transpose(0, 1).numpy() for l in range(L)]
    h = captured["h"]
    h = h[0] if h.dim() == 3 else h
    if full_logp:
        return lp, keys, vals, h[P - 1].numpy(), logp.numpy()
    return lp, keys, vals, h[P - 1].numpy()


def brute_force(weights, cfg, token_ids, visual, response_ids):
    """Scalar float64 forward over the full sequence; returns logprobs of the response."""
    d, Hq, Hkv, Dh = cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    eps, theta = cfg.rms_eps, cfg.rope_theta
    E = [[float(v) for v in row] for row in np.asarray(weights.embed)]
    seq = []
    vi = 0
    for i in token_ids:
        if i < 0:
            seq.append([float(v) for v in visual[vi]])
            vi += 1
        else:
            seq.append(list(E[int(i)]))
    P = len(seq)
    for r in response_ids:
        seq.append(list(E[int(r)]))
    N = len(seq)

    def mat(w):
        return [[float(v) for v in row] for row in np.asarray(w)]

    def linear(x, W, b=None):
        return [sum(W[o][i] * x[i] for i in range(len(x))) + (0.0 if b is None else float(b[o]))
                for o in range(len(W))]

    def norm(x, w):
        r = math.sqrt(sum(v * v for v in x) / len(x) + eps)
        return [x[i] / r * float(w[i]) for i in range(len(x))]

    def rot(vec, pos):
        out = list(vec)
        half = Dh // 2
        for i in range(half):
            ang = pos * math.pow(theta, -2.0 * i / Dh)
            c, s = math.cos(ang), math.sin(ang)
            out[i] = vec[i] * c - vec[i + half] * s
            out[i + half] = vec[i + half] * c + vec[i] * s
        return out

    x = seq
    for lw in weights.layers:
        Wq, Wk, Wv, Wo = mat(lw["wq"]), mat(lw["wk"]), mat(lw["wv"]), mat(lw["wo"])
        Wg, Wu, Wd = mat(lw["w_gate"]), mat(lw["w_up"]), mat(lw["w_down"])
        qs, ks, vs = [], [], []
        for t in range(N):
            h = norm(x[t], lw["attn_norm"])
            q, k, v = linear(h, Wq, lw.get("bq")), linear(h, Wk, lw.get("bk")), linear(h, Wv, lw.get("bv"))
            qs.append([rot(q[j * Dh:(j + 1) * Dh], t) for j in range(Hq)])
            ks.append([rot(k[j * Dh:(j + 1) * Dh], t) for j in range(Hkv)])
            vs.append([v[j * Dh:(j + 1) * Dh] for j in range(Hkv)])
        new_x = []
        for t in range(N):
            o = []
            for hq in range(Hq):
                g = hq // (Hq // Hkv)
                sc = [sum(qs[t][hq][i] * ks[u][g][i] for i in range(Dh)) / math.sqrt(Dh)
                      for u in range(t + 1)]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                tot = sum(ex)
                o.extend(sum(ex[u] / tot * vs[u][g][i] for u in range(t + 1)) for i in range(Dh))
            a = linear(o, Wo)
            xt = [x[t][i] + a[i] for i in range(d)]
            h2 = norm(xt, lw["mlp_norm"])
            gt, up = linear(h2, Wg), linear(h2, Wu)
            act = [gt[i] / (1.0 + math.exp(-gt[i])) * up[i] for i in range(len(gt))]
            dn = linear(act, Wd)
            new_x.append([xt[i] + dn[i] for i in range(d)])
        x = new_x
    Wl = mat(weights.lm_head)
    lps = []
    for j, r in enumerate(response_ids):
        h = norm(x[P - 1 + j], weights.final_norm)
        logits = linear(h, Wl)
        mx = max(logits)
        lse = mx + math.log(sum(math.exp(v - mx) for v in logits))
        lps.append(logits[int(r)] - lse)
    return np.array(lps)


def hf_mrope(q, k, pos3, sections, theta):
    """q [n, Hq, Dh], k [n, Hkv, Dh] rotated by transformers' Qwen2.5-VL multimodal RoPE
    (its section selection and rotate-half), fed float64 cos/sin of the three position rows."""
    import torch
    from transformers.models.qwen2_5_vl.modeling_qwen2_5_vl import apply_multimodal_rotary_pos_emb
    Dh = q.shape[-1]
    inv = torch.tensor(theta, dtype=torch.float64) ** (-torch.arange(0, Dh, 2, dtype=torch.float64) / Dh)
    pos = torch.tensor(np.asarray(pos3), dtype=torch.float64)          # [3, n]
    freqs = pos[:, None, :, None] * inv[None, None, None, :]            # [3, 1, n, Dh/2]
    emb = torch.cat([freqs, freqs], dim=-1)
    qt = torch.tensor(q).transpose(0, 1)[None]                          # [1, H, n, Dh]
    kt = torch.tensor(k).transpose(0, 1)[None]
    qo, ko = apply_multimodal_rotary_pos_emb(qt, kt, emb.cos(), emb.sin(), list(sections))
    return qo[0].transpose(0, 1).numpy(), ko[0].transpose(0, 1).numpy()
