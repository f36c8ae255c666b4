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
