"""Model shapes and workloads of the prefix/suffix backbone path.

Shapes only: no arithmetic of the method lives here.  The backbone is the
LLM part of a Qwen2.5-VL-style vision-language model (the paper's evaluation
models, Section "Experimental Setup"); the sizes below are per-layer slices of
the 7B and 32B members plus a tiny fp32 model for exact checks.  The workload
shape follows the paper's video RL tasks: prompts that are mostly visual
tokens (79-98% of each sequence, Section "An Input-Heavy Workload"), an 8k
prompt + 2k response budget (Section "Experimental Setup").
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str                      # "f32", "bf16" or "f16": storage type of weights/activations/KV
    rms_eps: float = 1e-6
    rope_theta: float = 1e6

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def params_per_layer(self) -> int:
        d, hd = self.d_model, self.head_dim
        return (d * self.qkv_dim + self.n_q_heads * hd * d + 3 * d * self.ffn_dim)


@dataclass(frozen=True)
class Workload:
    index: int                       # seed namespace of the generator
    name: str
    model: ModelShape
    prefix_lens: Optional[List[int]] = None     # per sequence (None: drawn, ragged)
    visual_lens: Optional[List[int]] = None     # visual slots per sequence
    suffix_lens: Optional[List[int]] = None
    ragged: Optional[dict] = None               # draw spec for ragged batches
    decode: Optional[dict] = None               # co-location decode spec
    group: Optional[int] = None                 # responses per prompt sharing its prefix (GRPO);
                                                # suffix_lens then lists every response
    note: str = ""


TINY = ModelShape(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                  ffn_dim=688, vocab=2048, dtype="f32")
QWEN7B_SLICE = ModelShape(n_layers=4, d_model=3584, n_q_heads=28, n_kv_heads=4, head_dim=128,
                          ffn_dim=18944, vocab=152064, dtype="bf16")
QWEN32B_SLICE = ModelShape(n_layers=2, d_model=5120, n_q_heads=40, n_kv_heads=8, head_dim=128,
                           ffn_dim=27648, vocab=152064, dtype="bf16")

WORKLOADS = {
    "tiny_f32": Workload(0, "tiny_f32", TINY, prefix_lens=[512, 512], visual_lens=[448, 448],
                         suffix_lens=[64, 64]),
    "qwen7b_b4_p4096_s256": Workload(1, "qwen7b_b4_p4096_s256", QWEN7B_SLICE,
                                     prefix_lens=[4096] * 4, visual_lens=[3840] * 4,
                                     suffix_lens=[256] * 4),
    "qwen32b_b2_p16384_s512": Workload(2, "qwen32b_b2_p16384_s512", QWEN32B_SLICE,
                                       prefix_lens=[16384] * 2, visual_lens=[15872] * 2,
                                       suffix_lens=[512] * 2),
    "qwen7b_ragged_b8": Workload(3, "qwen7b_ragged_b8", QWEN7B_SLICE,
                                 ragged=dict(batch=8, prefix_lo=2048, prefix_hi=12288,
                                             text_frac=0.1, suffix_lo=64, suffix_hi=1024)),
    "qwen7b_coloc_p4x8192_d64": Workload(4, "qwen7b_coloc_p4x8192_d64", QWEN7B_SLICE,
                                         prefix_lens=[8192] * 4, visual_lens=[7680] * 4,
                                         suffix_lens=[0] * 4,
                                         decode=dict(batch=64, kv_len=8192, cap=8192 + 64)),
    # GRPO groups (Section "Experimental Setup": N = 8 responses per prompt; Section "Prefix
    # Sharing": a group's prefix runs once): 4 prompts x 8 responses of 256 tokens
    "qwen7b_grpo_g4_p4096_n8_s256": Workload(5, "qwen7b_grpo_g4_p4096_n8_s256", QWEN7B_SLICE,
                                             prefix_lens=[4096] * 4, visual_lens=[3840] * 4,
                                             suffix_lens=[256] * 32, group=8),
}

# the five benchmark configurations; other workloads are extra measurements
ORDER = ["tiny_f32", "qwen7b_b4_p4096_s256", "qwen32b_b2_p16384_s512", "qwen7b_ragged_b8",
         "qwen7b_coloc_p4x8192_d64"]


def get(name: str) -> Workload:
    return WORKLOADS[name]


def custom(model: ModelShape, prefix_lens, visual_lens, suffix_lens, index: int = 100,
           name: str = "custom") -> Workload:
    """A workload with explicit lengths (used by tests at small sizes)."""
    return Workload(index, name, model, prefix_lens=list(prefix_lens),
                    visual_lens=list(visual_lens), suffix_lens=list(suffix_lens))


def with_model(w: Workload, **changes) -> Workload:
    return replace(w, model=replace(w.model, **changes))
