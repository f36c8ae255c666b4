"""ctypes binding of the C ABI in include/rollplex.h.

Functions keep the C names and only marshal arguments: torch tensors (or raw
integer addresses) become device pointers, Python sequences of lengths become
host int32 arrays, and a non-OK status raises ``RollplexError`` with the
library's message.  Every step of the computation runs in the HIP library.
Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, Structure, byref, c_char_p, c_double, c_float, c_int, c_int32, c_int64, \
    c_size_t, c_uint32, c_void_p
from typing import Optional, Sequence

# RP_LIBRARY selects another build of the same library (the host-sanitized one of
# build.py --sanitize); by default the in-tree gfx950 build.
LIB_PATH = os.environ.get("RP_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib",
                                                        "librollplex.so")

RP_OK, RP_ERR_INVALID_ARG, RP_ERR_SHAPE, RP_ERR_UNSUPPORTED, RP_ERR_WORKSPACE, RP_ERR_HIP = range(6)
RP_F32, RP_BF16, RP_F16 = 0, 1, 2
_DTYPES = {"f32": RP_F32, "bf16": RP_BF16, "f16": RP_F16}
RP_MAX_SEQS = 256
RP_SUFFIX_FUSED_LOGPROB = 1
RP_WO_TRANSPOSED, RP_W_DOWN_TRANSPOSED = 1, 2
RP_PREFIX_LAST_ROWS_ONLY = 1
SYMBOLS = ["rp_create", "rp_destroy", "rp_prefix_workspace_bytes", "rp_prefix_forward", "rp_prefix_forward_mrope",
           "rp_prefix_forward_flags",
           "rp_suffix_workspace_bytes", "rp_suffix_logprob", "rp_suffix_grouped_workspace_bytes",
           "rp_suffix_logprob_grouped", "rp_prompt_logprob_workspace_bytes", "rp_prompt_logprob",
           "rp_decode_workspace_bytes",
           "rp_decode_step", "rp_decode_step_static", "rp_stream_create_cu_masked", "rp_stream_destroy",
           "rp_device_cu_count", "rp_calibrate_mfma", "rp_calibrate_read", "rp_last_error", "rp_status_string", "rp_version",
           "rp_profile_enable", "rp_profile_collect", "rp_profile_count", "rp_profile_read",
           "rp_profile_reset"]


class RollplexError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status


class RpConfig(Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_q_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("ffn_dim", c_int32),
                ("vocab", c_int32), ("max_position", c_int32), ("rms_eps", c_float),
                ("rope_theta", c_double), ("dtype", c_int), ("weight_layout", c_uint32)]


class RpLayerWeights(Structure):
    _fields_ = [(n, c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "bq", "bk", "bv", "wo",
                                        "mlp_norm", "w_gate", "w_up", "w_down")]


class RpWeights(Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("layers", POINTER(RpLayerWeights))]


class RpKV(Structure):
    _fields_ = [("k", c_void_p), ("v", c_void_p), ("layer_stride", c_int64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing "
                               f"(run python -m paper_2608_14498_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "rp_create": (c_int, [POINTER(RpConfig), POINTER(RpWeights), POINTER(c_void_p)]),
            "rp_destroy": (None, [c_void_p]),
            "rp_prefix_workspace_bytes": (c_int, [c_void_p, c_int32, POINTER(c_int32), POINTER(c_size_t)]),
            "rp_prefix_forward": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                          c_int64, RpKV, c_void_p, c_void_p, c_void_p, c_size_t]),
            "rp_suffix_workspace_bytes": (c_int, [c_void_p, c_int32, POINTER(c_int32), POINTER(c_int32),
                                                  POINTER(c_size_t)]),
            "rp_suffix_logprob": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32), POINTER(c_int32),
                                          RpKV, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t]),
            "rp_suffix_grouped_workspace_bytes": (c_int, [c_void_p, c_int32, POINTER(c_int32), c_int32,
                                                          POINTER(c_int32), POINTER(c_int32), c_uint32,
                                                          POINTER(c_size_t)]),
            "rp_suffix_logprob_grouped": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32), c_int32,
                                                  POINTER(c_int32), POINTER(c_int32), POINTER(c_int32), c_uint32,
                                                  RpKV, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t]),
            "rp_prefix_forward_mrope": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                                c_int64, c_void_p, POINTER(c_int32), RpKV, c_void_p, c_void_p,
                                                c_void_p, c_size_t]),
            "rp_prefix_forward_flags": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                                c_int64, c_void_p, POINTER(c_int32), c_uint32, RpKV, c_void_p,
                                                c_void_p, c_void_p, c_size_t]),
            "rp_prompt_logprob_workspace_bytes": (c_int, [c_void_p, c_int32, c_uint32, POINTER(c_size_t)]),
            "rp_prompt_logprob": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                          c_int32, c_void_p, c_uint32, c_void_p, c_void_p, c_size_t]),
            "rp_decode_workspace_bytes": (c_int, [c_void_p, c_int32, c_int32, POINTER(c_size_t)]),
            "rp_calibrate_mfma": (c_int, [c_void_p, c_int, c_int32, c_int32, c_void_p, c_size_t,
                                          POINTER(c_double)]),
            "rp_calibrate_read": (c_int, [c_void_p, c_void_p, c_int64, c_int32, c_void_p, c_size_t]),
            "rp_decode_step": (c_int, [c_void_p, c_void_p, c_int32, RpKV, c_int32, c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_void_p, c_size_t]),
            "rp_decode_step_static": (c_int, [c_void_p, c_void_p, c_int32, RpKV, c_int32, c_void_p, c_void_p,
                                              c_void_p, c_void_p]),
            "rp_stream_create_cu_masked": (c_int, [c_int, POINTER(c_uint32), c_uint32, POINTER(c_void_p)]),
            "rp_stream_destroy": (c_int, [c_void_p]),
            "rp_device_cu_count": (c_int, [c_int]),
            "rp_last_error": (c_char_p, []),
            "rp_status_string": (c_char_p, [c_int]),
            "rp_version": (c_char_p, []),
            "rp_profile_enable": (c_int, [c_int, c_int32]),
            "rp_profile_collect": (c_int, []),
            "rp_profile_count": (c_int32, []),
            "rp_profile_read": (c_int, [c_int32, POINTER(c_char_p), POINTER(c_int64), POINTER(c_double)]),
            "rp_profile_reset": (None, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _status_name(s: int) -> str:
    try:
        return lib().rp_status_string(s).decode()
    except Exception:  # pragma: no cover
        return f"status {s}"


def _check(status: int):
    if status != RP_OK:
        raise RollplexError(status, lib().rp_last_error().decode())


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _i32(seq: Optional[Sequence[int]]):
    if seq is None:
        return None
    vals = [int(v) for v in seq]
    return (c_int32 * len(vals))(*vals)


def make_config(model, max_position: int, weight_layout: int = 0) -> RpConfig:
    return RpConfig(model.n_layers, model.d_model, model.n_q_heads, model.n_kv_heads, model.head_dim,
                    model.ffn_dim, model.vocab, int(max_position), float(model.rms_eps),
                    float(model.rope_theta), _DTYPES[model.dtype], int(weight_layout))


def make_kv(k, v, layer_stride: int) -> RpKV:
    return RpKV(_ptr(k), _ptr(v), int(layer_stride))


# ------------------------------------------------------------------------------------------
# the C entry points
# ------------------------------------------------------------------------------------------
def rp_create(config: RpConfig, weights: RpWeights) -> int:
    h = c_void_p()
    _check(lib().rp_create(byref(config), byref(weights), byref(h)))
    return h.value


def rp_destroy(model: int) -> None:
    lib().rp_destroy(model)


def rp_prefix_workspace_bytes(model: int, B: int, cu_seqlens) -> int:
    n = c_size_t()
    _check(lib().rp_prefix_workspace_bytes(model, B, _i32(cu_seqlens), byref(n)))
    return n.value


def rp_prefix_forward(model: int, stream, B: int, cu_seqlens, token_ids, visual_embeds, n_visual: int,
                      kv_out: RpKV, h_last, hidden_out, workspace, workspace_bytes: int) -> None:
    _check(lib().rp_prefix_forward(model, _ptr(stream), B, _i32(cu_seqlens), _ptr(token_ids),
                                   _ptr(visual_embeds), int(n_visual), kv_out, _ptr(h_last),
                                   _ptr(hidden_out), _ptr(workspace), int(workspace_bytes)))


def rp_suffix_workspace_bytes(model: int, B: int, prefix_cu, suffix_cu) -> int:
    n = c_size_t()
    _check(lib().rp_suffix_workspace_bytes(model, B, _i32(prefix_cu), _i32(suffix_cu), byref(n)))
    return n.value


def rp_suffix_logprob(model: int, stream, B: int, prefix_cu, suffix_cu, kv: RpKV, h_last, response_ids,
                      logprobs, workspace, workspace_bytes: int) -> None:
    _check(lib().rp_suffix_logprob(model, _ptr(stream), B, _i32(prefix_cu), _i32(suffix_cu), kv,
                                   _ptr(h_last), _ptr(response_ids), _ptr(logprobs), _ptr(workspace),
                                   int(workspace_bytes)))


def rp_suffix_grouped_workspace_bytes(model: int, n_prefix: int, prefix_cu, n_suffix: int, prefix_of_suffix,
                                      suffix_cu, flags: int = 0) -> int:
    n = c_size_t()
    _check(lib().rp_suffix_grouped_workspace_bytes(model, n_prefix, _i32(prefix_cu), n_suffix,
                                                   _i32(prefix_of_suffix), _i32(suffix_cu), int(flags), byref(n)))
    return n.value


def rp_suffix_logprob_grouped(model: int, stream, n_prefix: int, prefix_cu, n_suffix: int, prefix_of_suffix,
                              suffix_cu, rope_pos0, flags: int, kv: RpKV, h_last, response_ids, logprobs, workspace,
                              workspace_bytes: int) -> None:
    _check(lib().rp_suffix_logprob_grouped(model, _ptr(stream), n_prefix, _i32(prefix_cu), n_suffix,
                                           _i32(prefix_of_suffix), _i32(suffix_cu), _i32(rope_pos0), int(flags),
                                           kv, _ptr(h_last), _ptr(response_ids), _ptr(logprobs), _ptr(workspace),
                                           int(workspace_bytes)))


def rp_prefix_forward_mrope(model: int, stream, B: int, cu_seqlens, token_ids, visual_embeds, n_visual: int,
                            positions, mrope_section, kv_out: RpKV, h_last, hidden_out, workspace,
                            workspace_bytes: int) -> None:
    _check(lib().rp_prefix_forward_mrope(model, _ptr(stream), B, _i32(cu_seqlens), _ptr(token_ids),
                                         _ptr(visual_embeds), int(n_visual), _ptr(positions), _i32(mrope_section),
                                         kv_out, _ptr(h_last), _ptr(hidden_out), _ptr(workspace),
                                         int(workspace_bytes)))


def rp_prompt_logprob_workspace_bytes(model: int, n_rows: int, flags: int = 0) -> int:
    n = c_size_t()
    _check(lib().rp_prompt_logprob_workspace_bytes(model, int(n_rows), int(flags), byref(n)))
    return n.value


def rp_prompt_logprob(model: int, stream, B: int, cu_seqlens, token_ids, hidden, n_rows: int, positions,
                      flags: int, logprobs, workspace, workspace_bytes: int) -> None:
    _check(lib().rp_prompt_logprob(model, _ptr(stream), B, _i32(cu_seqlens), _ptr(token_ids), _ptr(hidden),
                                   int(n_rows), _ptr(positions), int(flags), _ptr(logprobs), _ptr(workspace),
                                   int(workspace_bytes)))


def rp_prefix_forward_flags(model: int, stream, B: int, cu_seqlens, token_ids, visual_embeds, n_visual: int,
                            positions, mrope_section, flags: int, kv_out: RpKV, h_last, hidden_out, workspace,
                            workspace_bytes: int) -> None:
    _check(lib().rp_prefix_forward_flags(model, _ptr(stream), B, _i32(cu_seqlens), _ptr(token_ids),
                                         _ptr(visual_embeds), int(n_visual), _ptr(positions), _i32(mrope_section),
                                         int(flags), kv_out, _ptr(h_last), _ptr(hidden_out), _ptr(workspace),
                                         int(workspace_bytes)))


def rp_decode_workspace_bytes(model: int, B: int, cap: int) -> int:
    n = c_size_t()
    _check(lib().rp_decode_workspace_bytes(model, B, cap, byref(n)))
    return n.value


def rp_decode_step(model: int, stream, B: int, cache: RpKV, cap: int, kv_len, token_ids, logits, next_ids,
                   workspace, workspace_bytes: int) -> None:
    _check(lib().rp_decode_step(model, _ptr(stream), B, cache, cap, _ptr(kv_len), _ptr(token_ids),
                                _ptr(logits), _ptr(next_ids), _ptr(workspace), int(workspace_bytes)))


RP_DECODE_STATIC_SCRATCH_BYTES = 96 << 20


def rp_decode_step_static(model: int, stream, B: int, cache: RpKV, cap: int, kv_len, token_ids, logits,
                          next_ids) -> None:
    """rp_decode_step with the library's static scratch instead of a workspace."""
    _check(lib().rp_decode_step_static(model, _ptr(stream), B, cache, cap, _ptr(kv_len), _ptr(token_ids),
                                       _ptr(logits), _ptr(next_ids)))


def rp_stream_create_cu_masked(device: int, mask_words: Sequence[int]) -> int:
    words = (c_uint32 * len(mask_words))(*[int(w) & 0xFFFFFFFF for w in mask_words])
    s = c_void_p()
    _check(lib().rp_stream_create_cu_masked(device, words, len(mask_words), byref(s)))
    return s.value


def rp_stream_destroy(stream: int) -> None:
    _check(lib().rp_stream_destroy(stream))


def rp_calibrate_mfma(stream, dtype: str, blocks: int, iters: int, sink, sink_bytes: int) -> float:
    """Launch the matrix-core probe; returns its flop count (time it on the same stream)."""
    f = c_double()
    _check(lib().rp_calibrate_mfma(_ptr(stream), _DTYPES[dtype], int(blocks), int(iters), _ptr(sink),
                                   int(sink_bytes), byref(f)))
    return f.value


def rp_calibrate_read(stream, src, nbytes: int, blocks: int, sink, sink_bytes: int) -> None:
    _check(lib().rp_calibrate_read(_ptr(stream), _ptr(src), int(nbytes), int(blocks), _ptr(sink),
                                   int(sink_bytes)))


def rp_device_cu_count(device: int = 0) -> int:
    return lib().rp_device_cu_count(device)


def rp_version() -> str:
    return lib().rp_version().decode()


def rp_profile_enable(enable: bool, max_launches: int = 1 << 14) -> None:
    _check(lib().rp_profile_enable(1 if enable else 0, int(max_launches)))


def rp_profile_collect() -> None:
    _check(lib().rp_profile_collect())


def rp_profile_reset() -> None:
    lib().rp_profile_reset()


def rp_profile_read_all() -> dict:
    """{kernel name: (launches, total_ms)} accumulated since the last reset."""
    out = {}
    for i in range(lib().rp_profile_count()):
        name, n, ms = c_char_p(), c_int64(), c_double()
        _check(lib().rp_profile_read(i, byref(name), byref(n), byref(ms)))
        out[name.value.decode()] = (n.value, ms.value)
    return out
