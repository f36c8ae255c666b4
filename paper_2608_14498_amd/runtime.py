"""Device-side convenience layer: torch owns the memory, the HIP library computes.

``DeviceModel`` uploads seeded host weights once, binds them with rp_create and
offers prefix / suffix / decode calls that allocate outputs and workspaces with
torch and call the C entry points on a torch stream.  Nothing here computes any
part of the method.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import binding as rb
from .configs import ModelShape


def to_device(a: Optional[np.ndarray], device) -> Optional[torch.Tensor]:
    """Upload a stored host tensor (float32, int32, or bf16 bit patterns as uint16)."""
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    if a.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.to(device, non_blocking=False)


def stream_ptr(stream: Optional[torch.cuda.Stream] = None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def prompt_positions(cu: Sequence[int], token_ids: np.ndarray) -> np.ndarray:
    """Packed positions of every scorable prompt token: text tokens (id >= 0) that are
    not the first token of their sequence (host int32)."""
    ids = np.asarray(token_ids)
    first = np.zeros(len(ids), bool)
    first[np.asarray(cu[:-1], np.int64)] = True
    return np.nonzero((ids >= 0) & ~first)[0].astype(np.int32)


class DeviceModel:
    """Weights resident in HBM plus a model handle of the HIP library."""

    def __init__(self, host_weights, max_position: int, device: str = "cuda", weight_layout: int = 0):
        """weight_layout (rb.RP_WO_TRANSPOSED | rb.RP_W_DOWN_TRANSPOSED) stores those row-parallel
        projections transposed, [in, out], as a training engine's shards would lay them out."""
        m: ModelShape = host_weights.model
        self.shape = m
        self.device = torch.device(device)
        self.dtype = {"bf16": torch.bfloat16, "f16": torch.float16}.get(m.dtype, torch.float32)
        self.max_position = int(max_position)
        up = lambda a: to_device(a, self.device)
        self.embed = up(host_weights.embed)
        self.lm_head = up(host_weights.lm_head)
        self.final_norm = up(host_weights.final_norm)
        stored_t = {"wo": weight_layout & rb.RP_WO_TRANSPOSED, "w_down": weight_layout & rb.RP_W_DOWN_TRANSPOSED}
        self.layers = [{k: up(np.ascontiguousarray(v.T) if stored_t.get(k) else v) for k, v in lw.items()}
                       for lw in host_weights.layers]
        p = rb._ptr
        arr = (rb.RpLayerWeights * m.n_layers)()
        for i, lw in enumerate(self.layers):
            for name, _ in rb.RpLayerWeights._fields_:
                setattr(arr[i], name, p(lw.get(name)))
        self._layer_arr = arr
        self._weights = rb.RpWeights(p(self.embed), p(self.final_norm), p(self.lm_head), arr)
        self.config = rb.make_config(m, self.max_position, weight_layout)
        self.handle = rb.rp_create(self.config, self._weights)

    def close(self):
        if getattr(self, "handle", None):
            rb.rp_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- helpers
    def alloc_kv(self, rows: int):
        m = self.shape
        shape = (m.n_layers, rows, m.n_kv_heads, m.head_dim)
        k = torch.empty(shape, dtype=self.dtype, device=self.device)
        v = torch.empty(shape, dtype=self.dtype, device=self.device)
        return k, v

    def workspace(self, nbytes: int) -> torch.Tensor:
        return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=self.device)

    # ---------------------------------------------------------------- passes
    def prefix(self, cu: Sequence[int], token_ids: torch.Tensor, visual: Optional[torch.Tensor],
               kv=None, h_last=None, hidden_out=None, workspace=None, stream=None, positions=None,
               mrope_section=None, flags: int = 0):
        """Prefix pass.  Returns (K, V, h_last) with K/V [L, T, Hkv, Dh].  With positions
        (device int32 [3, T]) and mrope_section, RoPE uses multimodal 3-D positions; flags
        (rb.RP_PREFIX_LAST_ROWS_ONLY) select options of rp_prefix_forward_flags."""
        m = self.shape
        B, T = len(cu) - 1, int(cu[-1])
        K, V = kv if kv is not None else self.alloc_kv(T)
        if h_last is None:
            h_last = torch.empty((B, m.d_model), dtype=torch.float32, device=self.device)
        nbytes = rb.rp_prefix_workspace_bytes(self.handle, B, cu)
        ws = workspace if workspace is not None else self.workspace(nbytes)
        n_visual = 0 if visual is None else visual.shape[0]
        if flags:
            rb.rp_prefix_forward_flags(self.handle, stream_ptr(stream), B, cu, token_ids, visual, n_visual,
                                       positions, mrope_section, flags, rb.make_kv(K, V, K[0].numel()), h_last,
                                       hidden_out, ws, ws.numel())
        elif positions is None:
            rb.rp_prefix_forward(self.handle, stream_ptr(stream), B, cu, token_ids, visual, n_visual,
                                 rb.make_kv(K, V, K[0].numel()), h_last, hidden_out, ws, ws.numel())
        else:
            rb.rp_prefix_forward_mrope(self.handle, stream_ptr(stream), B, cu, token_ids, visual, n_visual,
                                       positions, mrope_section, rb.make_kv(K, V, K[0].numel()), h_last,
                                       hidden_out, ws, ws.numel())
        return K, V, h_last

    def suffix(self, prefix_cu, suffix_cu, K, V, h_last, response_ids, logprobs=None, workspace=None,
               stream=None):
        B, R = len(prefix_cu) - 1, int(suffix_cu[-1])
        if logprobs is None:
            logprobs = torch.empty(max(R, 1), dtype=torch.float32, device=self.device)[:R]
        nbytes = rb.rp_suffix_workspace_bytes(self.handle, B, prefix_cu, suffix_cu)
        ws = workspace if workspace is not None else self.workspace(nbytes)
        rb.rp_suffix_logprob(self.handle, stream_ptr(stream), B, prefix_cu, suffix_cu,
                             rb.make_kv(K, V, K[0].numel()), h_last, response_ids, logprobs, ws, ws.numel())
        return logprobs

    def suffix_grouped(self, prefix_cu, prefix_of_suffix, suffix_cu, K, V, h_last, response_ids, logprobs=None,
                       workspace=None, stream=None, flags: int = 0, rope_pos0=None):
        """Suffix pass where suffix s reads prefix prefix_of_suffix[s] (shared prefixes);
        flags = rb.RP_SUFFIX_FUSED_LOGPROB scores without storing the logits; rope_pos0[p]
        is the rotary position of the first response token after prefix p (default P_p)."""
        P, S, R = len(prefix_cu) - 1, len(suffix_cu) - 1, int(suffix_cu[-1])
        if logprobs is None:
            logprobs = torch.empty(max(R, 1), dtype=torch.float32, device=self.device)[:R]
        nbytes = rb.rp_suffix_grouped_workspace_bytes(self.handle, P, prefix_cu, S, prefix_of_suffix, suffix_cu,
                                                      flags)
        ws = workspace if workspace is not None else self.workspace(nbytes)
        rb.rp_suffix_logprob_grouped(self.handle, stream_ptr(stream), P, prefix_cu, S, prefix_of_suffix,
                                     suffix_cu, rope_pos0, flags, rb.make_kv(K, V, K[0].numel()), h_last,
                                     response_ids, logprobs, ws, ws.numel())
        return logprobs

    def prompt_logprobs(self, cu, token_ids, hidden, positions, logprobs=None, workspace=None, stream=None,
                        flags: int = 0):
        """Teacher-forced log-probs of the prompt tokens at packed positions (device int32),
        scored from the prefix pass's hidden_out (device fp32 [T, d])."""
        B, n = len(cu) - 1, int(positions.numel())
        if logprobs is None:
            logprobs = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)[:n]
        nbytes = rb.rp_prompt_logprob_workspace_bytes(self.handle, n, flags)
        ws = workspace if workspace is not None else self.workspace(nbytes)
        rb.rp_prompt_logprob(self.handle, stream_ptr(stream), B, cu, token_ids, hidden, n, positions, flags,
                             logprobs, ws, ws.numel())
        return logprobs

    def decode(self, cache_k, cache_v, kv_len, token_ids, logits=None, next_ids=None, workspace=None,
               stream=None):
        B, cap = cache_k.shape[1], cache_k.shape[2]
        if next_ids is None:
            next_ids = torch.empty(B, dtype=torch.int32, device=self.device)
        nbytes = rb.rp_decode_workspace_bytes(self.handle, B, cap)
        ws = workspace if workspace is not None else self.workspace(nbytes)
        rb.rp_decode_step(self.handle, stream_ptr(stream), B, rb.make_kv(cache_k, cache_v, cache_k[0].numel()),
                          cap, kv_len, token_ids, logits, next_ids, ws, ws.numel())
        return next_ids
