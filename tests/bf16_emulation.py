"""Rounding-floor emulation of the 16-bit GPU path (a CPU diagnostic, not the oracle).

The oracle computes the plain definition in float64 on the bf16-rounded inputs.  The
16-bit GPU path computes the same thing, but must round some intermediates to the
model's 16-bit type: the operands of its matrix-core products (the normed activations
before the q/k/v and gate/up projections, the attention output before the o-proj, the
SwiGLU activation before the down projection, the final-norm rows before the lm_head),
the rotated queries and the stored keys/values, and the softmax probabilities of the
P.V product.  Everything else (the residual stream, the projections, the softmax
statistics, the logits, the log-softmax) is fp32 on the GPU, which is exact to ~1e-7
relative here.

This module runs the unsplit causal forward of one sequence in float64 and rounds to
the 16-bit type exactly at a chosen subset of those points, so that the contribution
of each point to |d logprob| can be measured against the oracle by ablation:

  norm   RMSNorm outputs feeding the q/k/v and gate/up projections
  q      queries after bias and rotation (the QK^T operand)
  kv     keys (after rotation) and values: what the boundary KV stores
  p      attention probabilities (relative to the row max) before P.V
  o      attention output before the o-proj
  act    SwiGLU product before the down projection
  final  final-norm rows before the lm_head

The split into prefix and suffix changes when work runs, not what it computes, so the
unsplit forward over [prefix ; response] has the same rounding points as the two
passes (the boundary state h_last is fp32).  It shares no code with the HIP path and
does not feed the oracle; tests/ may import it.

    python tests/bf16_emulation.py qwen7b_b4_p4096_s256 [--dtype bf16|f16] [--json OUT]

runs the ablation on the sequence the full-size parity test checks and prints
max/mean |d logprob| against the oracle for: every point rounded, every point but
one, and each point alone.

    python tests/bf16_emulation.py --floors [CASE ...]

writes tests/golden/bf16_floor.json: for each full-size parity case, max and mean
|d logprob| of the all-points bf16 emulation against the oracle values the test
compares with (tests/golden/*.npz), on the same tokens.  That is the error an ideal
bf16 implementation (every mandatory rounding, exact accumulation) leaves; the
full-size tests hold the GPU to it when it exceeds the 2e-2 target.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

POINTS = ("norm", "q", "kv", "p", "o", "act", "final")


def round_bf16(x):
    """Round to bfloat16, nearest-even, via fp32 (the GPU rounds fp32 values)."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32)
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return u.view(np.float32).astype(np.float64)


def round_f16(x):
    return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float64)


class Rounder:
    def __init__(self, dtype: str, points):
        self.fn = round_bf16 if dtype == "bf16" else round_f16
        self.points = frozenset(points)
        unknown = self.points - set(POINTS)
        assert not unknown, unknown

    def __call__(self, point, x):
        return self.fn(x) if point in self.points else x


def _rms(x, w, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def _rope(x, pos, theta):
    D = x.shape[-1]
    half = D // 2
    ang = pos.astype(np.float64)[:, None] * np.power(theta, -2.0 * np.arange(half) / D)[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def _attention(q, k, v, rnd, chunk=512):
    """Causal GQA attention over rows 0..n-1 (key index = position)."""
    n, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    out = np.empty_like(q)
    scale = 1.0 / math.sqrt(D)
    for c0 in range(0, n, chunk):
        c1 = min(n, c0 + chunk)
        nk = c1
        mask = np.arange(nk)[None, :] > np.arange(c0, c1)[:, None]
        for h in range(Hq):
            g = h // G
            s = (q[c0:c1, h] @ k[:nk, g].T) * scale
            s[mask] = -np.inf
            p = np.exp(s - s.max(axis=1, keepdims=True))
            l = p.sum(axis=1, keepdims=True)
            out[c0:c1, h] = (rnd("p", p) @ v[:nk, g]) / l
    return out


def _f(a):
    return None if a is None else np.asarray(a, np.float64)


def forward_hidden(W, cfg, token_ids, visual, response_ids, rnd: Rounder):
    """Final residual stream [P + S, d] of the causal forward over [prefix ; response] with
    16-bit rounding at rnd's points.  W holds float32 views of the stored weights
    (HostWeights.as_f32())."""
    f = _f
    ids = np.asarray(token_ids)
    P, S = len(ids), len(response_ids)
    E = W.embed
    x = np.empty((P + S, cfg.d_model))
    vis = ids < 0
    x[:P][~vis] = E[ids[~vis]]
    x[:P][vis] = visual[: int(vis.sum())]
    x[P:] = E[np.asarray(response_ids)]
    pos = np.arange(P + S)
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    n = P + S
    for lw in W.layers:
        h = rnd("norm", _rms(x, f(lw["attn_norm"]), cfg.rms_eps))
        q = h @ f(lw["wq"]).T
        k = h @ f(lw["wk"]).T
        v = h @ f(lw["wv"]).T
        for t, bn in ((q, "bq"), (k, "bk"), (v, "bv")):
            if lw.get(bn) is not None:
                t += f(lw[bn])
        q = rnd("q", _rope(q.reshape(n, Hq, D), pos, cfg.rope_theta))
        k = rnd("kv", _rope(k.reshape(n, Hkv, D), pos, cfg.rope_theta))
        v = rnd("kv", v.reshape(n, Hkv, D))
        o = rnd("o", _attention(q, k, v, rnd).reshape(n, Hq * D))
        x = x + o @ f(lw["wo"]).T
        h2 = rnd("norm", _rms(x, f(lw["mlp_norm"]), cfg.rms_eps))
        g = h2 @ f(lw["w_gate"]).T
        u = h2 @ f(lw["w_up"]).T
        with np.errstate(over="ignore"):
            a = rnd("act", g / (1.0 + np.exp(-g)) * u)
        del g, u
        x = x + a @ f(lw["w_down"]).T
        del a
    return x


def score(W, cfg, rows, ids, rnd: Rounder):
    """Log-probability of ids[i] under residual row rows[i]: final norm (rounded at the
    "final" point), lm_head, log-softmax over the vocabulary."""
    z = rnd("final", _rms(rows, _f(W.final_norm), cfg.rms_eps))
    lm = _f(W.lm_head)
    ids = np.asarray(ids)
    out = np.empty(len(ids))
    for r0 in range(0, len(ids), 128):
        lg = z[r0:r0 + 128] @ lm.T
        m = lg.max(axis=1, keepdims=True)
        lse = m[:, 0] + np.log(np.exp(lg - m).sum(axis=1))
        out[r0:r0 + 128] = lg[np.arange(len(lg)), ids[r0:r0 + 128]] - lse
    return out


def decode_logits(W, cfg, cache_k, cache_v, kv_len, token_ids, rnd: Rounder):
    """Logits [B, V] of one decode step (the new token of sequence b at position kv_len[b]
    over the cached keys/values 0..kv_len[b]-1, which are already 16-bit values) with
    rounding at rnd's points; the new token's own key/value is rounded at "kv"."""
    f = _f
    B = len(token_ids)
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    out = np.empty((B, W.lm_head.shape[0]))
    for b in range(B):
        n = int(kv_len[b])
        x = f(W.embed[[int(token_ids[b])]])
        pos = np.array([n])
        for l, lw in enumerate(W.layers):
            h = rnd("norm", _rms(x, f(lw["attn_norm"]), cfg.rms_eps))
            q, k, v = h @ f(lw["wq"]).T, h @ f(lw["wk"]).T, h @ f(lw["wv"]).T
            for t, bn in ((q, "bq"), (k, "bk"), (v, "bv")):
                if lw.get(bn) is not None:
                    t += f(lw[bn])
            q = rnd("q", _rope(q.reshape(1, Hq, D), pos, cfg.rope_theta))[0]
            k = rnd("kv", _rope(k.reshape(1, Hkv, D), pos, cfg.rope_theta))[0]
            v = rnd("kv", v.reshape(1, Hkv, D))[0]
            K = np.concatenate([f(cache_k[l, b, :n]), k[None]], axis=0)
            V = np.concatenate([f(cache_v[l, b, :n]), v[None]], axis=0)
            o = np.empty((Hq, D))
            for hh in range(Hq):
                g = hh // (Hq // Hkv)
                sc = K[:, g] @ q[hh] / math.sqrt(D)
                pr = np.exp(sc - sc.max())
                o[hh] = (rnd("p", pr) @ V[:, g]) / pr.sum()
            x = x + rnd("o", o.reshape(1, Hq * D)) @ f(lw["wo"]).T
            h2 = rnd("norm", _rms(x, f(lw["mlp_norm"]), cfg.rms_eps))
            g_, u_ = h2 @ f(lw["w_gate"]).T, h2 @ f(lw["w_up"]).T
            x = x + rnd("act", g_ / (1.0 + np.exp(-g_)) * u_) @ f(lw["w_down"]).T
        z = rnd("final", _rms(x, f(W.final_norm), cfg.rms_eps))
        out[b] = (z @ f(W.lm_head).T)[0]
    return out


def forward_logprobs(W, cfg, token_ids, visual, response_ids, rnd: Rounder):
    """log p(r_j | prefix, r_<j) of one sequence with 16-bit rounding at rnd's points."""
    P, S = len(token_ids), len(response_ids)
    x = forward_hidden(W, cfg, token_ids, visual, response_ids, rnd)
    return score(W, cfg, x[P - 1:P - 1 + S], response_ids, rnd)


def ablation(name: str, dtype: str = "bf16", seq: int = 0):
    """Max/mean |d logprob| against the oracle for the ablation arms on sequence seq."""
    import oracle
    from paper_2608_14498_amd import configs, inputs

    w = configs.with_model(configs.get(name), dtype=dtype)
    m = w.model
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    W = hw.as_f32()
    P, Vis, S = inputs.draw_lengths(w)
    cp, cs = bt.cu_prefix, bt.cu_suffix
    vo = int(sum(Vis[:seq]))
    ids = bt.token_ids[cp[seq]:cp[seq + 1]]
    vis = inputs.to_f32(bt.visual[vo:vo + Vis[seq]]).astype(np.float64)
    rid = bt.response_ids[cs[seq]:cs[seq + 1]]
    t0 = time.time()
    K, V, h, _ = oracle.prefix_forward_one(W, m, ids, vis)
    ref = oracle.suffix_logprob_one(W, m, K, V, h, rid)
    del K, V
    arms = [("exact", ())] + [("all", POINTS)]
    arms += [(f"all_but_{p}", tuple(x for x in POINTS if x != p)) for p in POINTS]
    arms += [(f"only_{p}", (p,)) for p in POINTS]
    res = {"workload": name, "dtype": dtype, "seq": seq, "tokens": int(len(rid)), "arms": {}}
    print(f"[emul] {name} {dtype} seq {seq}: oracle {time.time() - t0:.0f}s", flush=True)
    for tag, pts in arms:
        t1 = time.time()
        lp = forward_logprobs(W, m, ids, vis, rid, Rounder(dtype, pts))
        d = np.abs(lp - ref)
        res["arms"][tag] = dict(max=float(d.max()), mean=float(d.mean()), p99=float(np.quantile(d, 0.99)))
        print(f"[emul] {tag:14s} max {d.max():.4f} mean {d.mean():.4f} p99 {np.quantile(d, 0.99):.4f}"
              f" ({time.time() - t1:.0f}s)", flush=True)
    return res


# ----------------------------------------------------------------------------------------
# rounding floors of the full-size parity cases
# ----------------------------------------------------------------------------------------
FLOOR_PATH = os.path.join(HERE, "golden", "bf16_floor.json")


def _stats(got, ref):
    d = np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))
    return {"max": float(d.max()), "mean": float(d.mean()), "n": int(d.size)}


def _sequence(w, bt, b):
    from paper_2608_14498_amd import inputs

    P, Vis, _ = inputs.draw_lengths(w)
    cp = bt.cu_prefix
    vo = int(sum(Vis[:b]))
    ids = bt.token_ids[cp[b]:cp[b + 1]]
    return ids, inputs.to_f32(bt.visual[vo:vo + Vis[b]]).astype(np.float64)


def case_floor(case: str, dtype: str = "bf16"):
    """Max and mean |d logprob| between the all-points emulation and the stored oracle
    values of one full-size parity case ("fullsize:<workload>[:<golden suffix>]",
    "grouped:<workload>" or "prompt:<workload>"), on exactly the tokens the test checks."""
    from paper_2608_14498_amd import configs, inputs

    kind, name, *tag = case.split(":")
    w = configs.with_model(configs.get(name), dtype=dtype)
    m = w.model
    stem = {"fullsize": "fullsize_", "grouped": "fullsize_", "prompt": "fullsize_prompt_"}[kind]
    g = np.load(os.path.join(HERE, "golden", f"{stem}{name}{'_' + tag[0] if tag else ''}.npz"), allow_pickle=False)
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    W = hw.as_f32()
    rnd = Rounder(dtype, POINTS)
    b = int(g["seq"])
    ids, vis = _sequence(w, bt, b)
    cs = bt.cu_suffix
    if kind == "prompt":
        x = forward_hidden(W, m, ids, vis, np.zeros(0, np.int64), rnd)
        pos = np.asarray(g["prompt_pos"])
        return _stats(score(W, m, x[pos - 1], ids[pos], rnd), g["prompt_logprobs"])
    if kind == "grouped":
        got = [forward_logprobs(W, m, ids, vis, bt.response_ids[cs[r]:cs[r + 1]], rnd) for r in g["resp_idx"]]
        return _stats(np.stack(got), g["logprobs"])
    return _stats(forward_logprobs(W, m, ids, vis, bt.response_ids[cs[b]:cs[b + 1]], rnd), g["logprobs"])


FLOOR_CASES = ("fullsize:qwen7b_b4_p4096_s256", "fullsize:qwen32b_b2_p16384_s512", "fullsize:qwen7b_ragged_b8",
               "grouped:qwen7b_grpo_g4_p4096_n8_s256", "prompt:qwen7b_b4_p4096_s256", "prompt:qwen7b_ragged_b8")


def write_floors(cases):
    """Add the named cases' floors to FLOOR_PATH (keeps the others)."""
    rec = json.load(open(FLOOR_PATH)) if os.path.exists(FLOOR_PATH) else {}
    for c in cases:
        t0 = time.time()
        rec[c] = case_floor(c)
        rec[c]["seconds"] = round(time.time() - t0, 1)
        print(f"[floor] {c}: {rec[c]}", flush=True)
        with open(FLOOR_PATH, "w") as fh:
            json.dump(rec, fh, indent=1, sort_keys=True)


def load_floor(case: str):
    """Stored floor of a full-size case, or None."""
    if not os.path.exists(FLOOR_PATH):
        return None
    return json.load(open(FLOOR_PATH)).get(case)


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("workload", nargs="?")
    ap.add_argument("--dtype", default="bf16")
    ap.add_argument("--seq", type=int, default=0)
    ap.add_argument("--json", default=None)
    ap.add_argument("--floors", nargs="*", default=None,
                    help="write the rounding floors of these full-size cases (default: all) to "
                         "tests/golden/bf16_floor.json")
    a = ap.parse_args()
    if a.floors is not None:
        write_floors(a.floors or FLOOR_CASES)
    else:
        r = ablation(a.workload, a.dtype, a.seq)
        if a.json:
            with open(a.json, "w") as fh:
                json.dump(r, fh, indent=1)
