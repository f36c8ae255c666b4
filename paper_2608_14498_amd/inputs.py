"""Seeded synthetic inputs for the prefix/suffix backbone path.

This module is shared by the oracle-side tests and by the GPU path's callers.
It holds none of the method's arithmetic: it only draws random tensors,
rounds them to the storage type and lays out packed (ragged) batches.

Recipe (stands in for the paper's video RL datasets, which are not available):
  * every tensor has its own PCG64 stream, ``default_rng([workload.index,
    tensor_index, chunk])`` with chunks of ``CHUNK`` elements, so the values do
    not depend on how many threads draw them;
  * weight matrices N(0, 0.02); norm weights 1 (or 1 + 0.1 N(0,1) in the
    "random" test variant); q/k/v biases absent (or N(0, 0.1) in tests);
  * visual embeddings N(0, 1) (stand-ins for projector outputs), one block
    per sequence placed before its text tokens; token and response ids
    uniform over the vocabulary;
  * bf16 workloads draw in fp32 and round once, to nearest-even, to bf16; both
    the GPU path and the oracle consume exactly those rounded values;
  * f16 workloads are the same bf16 model stored in binary16: the bf16-rounded
    values converted to fp16 (exact inside fp16's normal range; the few weights
    below 2^-14 in magnitude land on the fp16 subnormal grid, changing them by
    at most 2^-25).  The oracle consumes the fp16 values.
bf16 tensors are held as their raw 16-bit patterns (``numpy.uint16``), f16 tensors
as ``numpy.float16``.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from .configs import Workload, ModelShape

CHUNK = 1 << 22

# tensor indices of the seed namespace
T_EMBED, T_LM_HEAD, T_FINAL_NORM = 1, 2, 3
T_VISUAL, T_TEXT_IDS, T_RESP_IDS, T_LENGTHS = 10, 11, 12, 13
T_DEC_K, T_DEC_V, T_DEC_IDS, T_DEC_LEN = 20, 21, 22, 23
LAYER_BASE, LAYER_STRIDE = 100, 16
LAYER_TENSORS = ["wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "attn_norm", "mlp_norm",
                 "bq", "bk", "bv"]


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# ----------------------------------------------------------------------------------------
# bf16 storage helpers (format conversion only)
# ----------------------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16, nearest-even, returning the 16-bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).copy()
    u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (u >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_f32(a: np.ndarray) -> np.ndarray:
    """Float32 values of a stored tensor (bf16 patterns and fp16 are widened exactly)."""
    if a is None:
        return None
    if a.dtype == np.uint16:
        return bf16_bits_to_f32(a)
    return np.asarray(a, dtype=np.float32)


def _storage(dtype: str):
    return {"bf16": np.uint16, "f16": np.float16}.get(dtype, np.float32)


# ----------------------------------------------------------------------------------------
# chunked, threaded normal draws
# ----------------------------------------------------------------------------------------
def _draw_normal(shape, seed: List[int], std: float, dtype: str, mean: float = 0.0) -> np.ndarray:
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=_storage(dtype))
    nchunks = (n + CHUNK - 1) // CHUNK

    def work(c):
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        rng = np.random.default_rng(list(seed) + [c])
        v = np.empty(hi - lo, dtype=np.float32)
        rng.standard_normal(out=v, dtype=np.float32)
        if std != 1.0:
            v *= np.float32(std)
        if mean != 0.0:
            v += np.float32(mean)
        if dtype in ("bf16", "f16"):
            # the model is defined by the bf16-rounded draw; an "f16" model stores those
            # same values in binary16 (exact within fp16's normal range)
            u = v.view(np.uint32)
            t = (u >> np.uint32(16)) & np.uint32(1)
            t += np.uint32(0x7FFF)
            u += t
            u >>= np.uint32(16)
            if dtype == "bf16":
                out[lo:hi] = u
            else:
                out[lo:hi] = (u << np.uint32(16)).view(np.float32).astype(np.float16)
        else:
            out[lo:hi] = v

    if nchunks <= 1:
        for c in range(nchunks):
            work(c)
    else:
        with ThreadPoolExecutor(min(_threads(), nchunks)) as ex:
            list(ex.map(work, range(nchunks)))
    return out.reshape(shape)


def _ones(shape, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return np.full(shape, 0x3F80, dtype=np.uint16)
    return np.ones(shape, dtype=_storage(dtype))


# ----------------------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------------------
@dataclass
class HostWeights:
    model: ModelShape
    embed: np.ndarray
    lm_head: np.ndarray
    final_norm: np.ndarray
    layers: List[Dict[str, Optional[np.ndarray]]]

    def as_f32(self) -> "HostWeights":
        """Float32 copy (16-bit storage widened exactly) for the oracle."""
        return HostWeights(self.model, to_f32(self.embed), to_f32(self.lm_head),
                           to_f32(self.final_norm),
                           [{k: to_f32(v) for k, v in lw.items()} for lw in self.layers])


def make_weights(w: Workload, norm: str = "ones", bias: bool = False,
                 layers: Optional[int] = None) -> HostWeights:
    """Seeded random weights, nn.Linear layout [out, in], row-major."""
    m = w.model
    dt = m.dtype
    d, hd = m.d_model, m.head_dim
    nl = m.n_layers if layers is None else layers
    out_layers = []
    for l in range(nl):
        base = LAYER_BASE + LAYER_STRIDE * l
        seed = lambda j: [w.index, base + j]
        lw = {
            "wq": _draw_normal((m.n_q_heads * hd, d), seed(0), 0.02, dt),
            "wk": _draw_normal((m.n_kv_heads * hd, d), seed(1), 0.02, dt),
            "wv": _draw_normal((m.n_kv_heads * hd, d), seed(2), 0.02, dt),
            "wo": _draw_normal((d, m.n_q_heads * hd), seed(3), 0.02, dt),
            "w_gate": _draw_normal((m.ffn_dim, d), seed(4), 0.02, dt),
            "w_up": _draw_normal((m.ffn_dim, d), seed(5), 0.02, dt),
            "w_down": _draw_normal((d, m.ffn_dim), seed(6), 0.02, dt),
        }
        if norm == "random":
            lw["attn_norm"] = _draw_normal((d,), seed(7), 0.1, dt, mean=1.0)
            lw["mlp_norm"] = _draw_normal((d,), seed(8), 0.1, dt, mean=1.0)
        else:
            lw["attn_norm"] = _ones((d,), dt)
            lw["mlp_norm"] = _ones((d,), dt)
        if bias:
            lw["bq"] = _draw_normal((m.n_q_heads * hd,), seed(9), 0.1, dt)
            lw["bk"] = _draw_normal((m.n_kv_heads * hd,), seed(10), 0.1, dt)
            lw["bv"] = _draw_normal((m.n_kv_heads * hd,), seed(11), 0.1, dt)
        else:
            lw["bq"] = lw["bk"] = lw["bv"] = None
        out_layers.append(lw)
    embed = _draw_normal((m.vocab, d), [w.index, T_EMBED], 0.02, dt)
    lm_head = _draw_normal((m.vocab, d), [w.index, T_LM_HEAD], 0.02, dt)
    if norm == "random":
        final_norm = _draw_normal((d,), [w.index, T_FINAL_NORM], 0.1, dt, mean=1.0)
    else:
        final_norm = _ones((d,), dt)
    return HostWeights(m, embed, lm_head, final_norm, out_layers)


# ----------------------------------------------------------------------------------------
# packed batches
# ----------------------------------------------------------------------------------------
@dataclass
class HostBatch:
    prefix_lens: List[int]
    visual_lens: List[int]
    suffix_lens: List[int]
    cu_prefix: np.ndarray          # int32 [B+1]
    cu_suffix: np.ndarray          # int32 [B+1]
    token_ids: np.ndarray          # int32 [T]; -1 marks a visual slot
    visual: np.ndarray             # [N_vis, d] storage dtype, consumed in slot order
    response_ids: np.ndarray       # int32 [R]
    prefix_of_suffix: Optional[np.ndarray] = None   # int32 [n_suffix] when prefixes are shared

    @property
    def batch(self) -> int:
        return len(self.prefix_lens)

    @property
    def T(self) -> int:
        return int(self.cu_prefix[-1])

    @property
    def R(self) -> int:
        return int(self.cu_suffix[-1])


def draw_lengths(w: Workload):
    """Per-sequence (prefix, visual, suffix) lengths; ragged workloads draw them."""
    if w.ragged is None:
        return list(w.prefix_lens), list(w.visual_lens), list(w.suffix_lens)
    r = w.ragged
    rng = np.random.default_rng([w.index, T_LENGTHS])
    p = rng.integers(r["prefix_lo"], r["prefix_hi"] + 1, r["batch"])
    s = rng.integers(r["suffix_lo"], r["suffix_hi"] + 1, r["batch"])
    n_text = np.floor(r["text_frac"] * p).astype(np.int64)
    return [int(x) for x in p], [int(x) for x in p - n_text], [int(x) for x in s]


def make_batch(w: Workload, lengths=None) -> HostBatch:
    m = w.model
    P, Vis, S = lengths if lengths is not None else draw_lengths(w)
    B = len(P)
    cu_p = np.zeros(B + 1, np.int32)
    cu_p[1:] = np.cumsum(P)
    cu_s = np.zeros(len(S) + 1, np.int32)
    cu_s[1:] = np.cumsum(S)
    grp = None
    if w.group:  # responses grouped by prompt: suffix s belongs to prefix s // group
        assert len(S) == B * w.group
        grp = np.repeat(np.arange(B, dtype=np.int32), w.group)
    T, R, NV = int(cu_p[-1]), int(cu_s[-1]), int(sum(Vis))
    text = np.random.default_rng([w.index, T_TEXT_IDS]).integers(0, m.vocab, T - NV, dtype=np.int32)
    ids = np.empty(T, np.int32)
    ti = 0
    for b in range(B):
        o, nv, nt = int(cu_p[b]), Vis[b], P[b] - Vis[b]
        assert 0 <= nv <= P[b]
        ids[o:o + nv] = -1
        ids[o + nv:o + P[b]] = text[ti:ti + nt]
        ti += nt
    visual = _draw_normal((NV, m.d_model), [w.index, T_VISUAL], 1.0, m.dtype)
    resp = np.random.default_rng([w.index, T_RESP_IDS]).integers(0, m.vocab, R, dtype=np.int32)
    return HostBatch(list(P), list(Vis), list(S), cu_p, cu_s, ids, visual, resp, grp)


# ----------------------------------------------------------------------------------------
# decode-step state (co-location workload)
# ----------------------------------------------------------------------------------------
@dataclass
class HostDecode:
    cache_k: np.ndarray            # [L, B, cap, Hkv, Dh] storage dtype
    cache_v: np.ndarray
    kv_len: np.ndarray             # int32 [B]
    token_ids: np.ndarray          # int32 [B]
    cap: int


def make_decode(w: Workload, batch: Optional[int] = None, kv_len=None, cap: Optional[int] = None
                ) -> HostDecode:
    m = w.model
    spec = w.decode or {}
    B = batch if batch is not None else spec["batch"]
    cap = cap if cap is not None else spec["cap"]
    if kv_len is None:
        kv_len = np.full(B, spec["kv_len"], np.int32)
    kv_len = np.asarray(kv_len, np.int32)
    shape = (m.n_layers, B, cap, m.n_kv_heads, m.head_dim)
    ck = _draw_normal(shape, [w.index, T_DEC_K], 1.0, m.dtype)
    cv = _draw_normal(shape, [w.index, T_DEC_V], 1.0, m.dtype)
    ids = np.random.default_rng([w.index, T_DEC_IDS]).integers(0, m.vocab, B, dtype=np.int32)
    return HostDecode(ck, cv, kv_len, ids, cap)
