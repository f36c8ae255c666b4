"""Algorithmic work counts and the overlap model used by the benchmark report.

Flop counts are those the method must perform (dense GEMM = 2 M N K; causal
attention counts only the visible half), not what a kernel happens to execute.
The overlap model is the paper's Eq. (1) (Section "Cross-Phase Execution").
"""
from __future__ import annotations

from typing import Dict, Sequence

# MI355X published peaks
PEAK_BF16_FLOPS = 2.5e15   # dense bf16 MFMA
PEAK_FP32_FLOPS = 157.3e12
PEAK_HBM_BPS = 8.0e12


def layer_gemm_flops_per_token(m) -> float:
    return 2.0 * m.params_per_layer


def prefix_flops(m, prefix_lens: Sequence[int], last_rows_only: bool = False) -> Dict[str, float]:
    """GEMM and attention flops of the prefix pass (all layers).  last_rows_only: the last
    layer runs its k/v projection for every row, and the q projection, attention (one
    query over P keys), o-proj and MLP only for each sequence's last row."""
    T = sum(prefix_lens)
    full = m.n_layers - (1 if last_rows_only else 0)
    gemm = full * T * layer_gemm_flops_per_token(m)
    # QK^T and PV over the causal half: 2 * (2 Hq Dh P(P+1)/2) per sequence per layer
    attn = full * sum(2.0 * m.n_q_heads * m.head_dim * P * (P + 1) for P in prefix_lens)
    if last_rows_only:
        kv = 2.0 * 2 * m.n_kv_heads * m.head_dim * m.d_model
        gemm += T * kv + len(prefix_lens) * (layer_gemm_flops_per_token(m) - kv)
        attn += sum(4.0 * m.n_q_heads * m.head_dim * P for P in prefix_lens)
    return {"gemm": gemm, "attention": attn, "total": gemm + attn}


def suffix_flops(m, prefix_lens: Sequence[int], suffix_lens: Sequence[int]) -> Dict[str, float]:
    R = sum(suffix_lens)
    gemm = m.n_layers * R * layer_gemm_flops_per_token(m)
    attn = m.n_layers * sum(4.0 * m.n_q_heads * m.head_dim * (S * P + S * (S + 1) / 2)
                            for P, S in zip(prefix_lens, suffix_lens))
    lm = 2.0 * R * m.d_model * m.vocab
    return {"gemm": gemm, "attention": attn, "lm_head": lm, "total": gemm + attn + lm}


def gemm_flops(M: int, N: int, K: int) -> float:
    return 2.0 * M * N * K


def logsoftmax_bytes(R: int, V: int) -> float:
    """Fused log-softmax + gather: read R fp32 rows of V logits, R ids, write R log-probs."""
    return 4.0 * R * V + 8.0 * R


def overlap_model(T_D: float, T_P: float, delta_D: float) -> Dict[str, float]:
    """Eq. (1): co-running prefix work (makespan T_P) with decode (alone T_D, slowed by
    delta_D) takes max(T_D + delta_D, T_P); the saving over running them back to back is
    S = T_D + T_P - max(T_D + delta_D, T_P) = min(T_P - delta_D, T_D)."""
    co = max(T_D + delta_D, T_P)
    saving = T_D + T_P - co
    regime = "decode-bounded" if T_D + delta_D >= T_P else "prefix-bounded"
    return {"serial": T_D + T_P, "co_run": co, "saving": saving, "regime": regime,
            "saving_closed_form": min(T_P - delta_D, T_D)}


def decode_interference(gen_alone: float, gen_corun: float) -> Dict[str, float]:
    """Decode slowdown delta_D and its relative size (Section "Resource Sharing Policy")."""
    d = gen_corun - gen_alone
    return {"delta_D": d, "relative": d / gen_alone}
