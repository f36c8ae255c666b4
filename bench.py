#!/usr/bin/env python3
"""Throughput of the prefix/suffix backbone path on one MI355X.

One step = the prefix pass (prompt prefill: KV + boundary state) followed by the
suffix pass (response log-probs over the cached KV) for one packed batch of
seeded synthetic inputs, all inputs resident in HBM.  Default workload: the
Qwen2.5-VL-7B-shaped 4-layer slice, batch 4, prefix 4096 (3840 visual + 256
text), suffix 256.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(w, hw, bt, prefix_len: int):
    """Time the CPU oracle (as it stands) on sequence 0 of the same workload."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle
    from paper_2608_14498_amd import inputs

    W = hw.as_f32()
    cp, cs = bt.cu_prefix, bt.cu_suffix
    ids = bt.token_ids[cp[0]:cp[1]]
    vis = inputs.to_f32(bt.visual[:bt.visual_lens[0]])
    resp = bt.response_ids[cs[0]:cs[1]]
    P = len(ids) if prefix_len <= 0 else min(prefix_len, len(ids))
    ids = ids[:P]
    vis = vis[:int((ids < 0).sum())]
    t0 = time.perf_counter()
    K, V, h, _ = oracle.prefix_forward_one(W, w.model, ids, vis)
    t1 = time.perf_counter()
    oracle.suffix_logprob_one(W, w.model, K, V, h, resp)
    t2 = time.perf_counter()
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    n_tok = P + len(resp)
    return {"value": n_tok / (t2 - t0), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"sequence 0 of the workload: prefix {P} + suffix {len(resp)} tokens, all "
                      f"{w.model.n_layers} layers, float64 numpy oracle; prefix {t1 - t0:.1f} s, "
                      f"suffix {t2 - t1:.1f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen7b_b4_p4096_s256")
    ap.add_argument("--profile-steps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-prefix-len", type=int, default=0,
                    help="truncate the CPU-baseline sample prefix (0 = full)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the path shards by "
              f"sequence and is measured on one GPU's share.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd import configs, inputs, perf
    from paper_2608_14498_amd.runtime import DeviceModel, to_device

    w = configs.get(args.workload)
    m = w.model
    log(f"workload {w.name}: generating seeded inputs")
    t0 = time.time()
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    log(f"inputs ready in {time.time() - t0:.1f} s; uploading")
    maxp = max(p + s for p, s in zip(bt.prefix_lens, bt.suffix_lens)) + 1
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    ids = to_device(bt.token_ids, dev)
    vis = to_device(bt.visual, dev) if bt.visual.shape[0] else None
    resp = to_device(bt.response_ids, dev)
    cu_p = [int(x) for x in bt.cu_prefix]
    cu_s = [int(x) for x in bt.cu_suffix]
    B, T, R = bt.batch, bt.T, bt.R
    K, V = dm.alloc_kv(T)
    h_last = torch.empty((B, m.d_model), dtype=torch.float32, device=dev)
    lp = torch.empty(max(R, 1), dtype=torch.float32, device=dev)
    ws_p = dm.workspace(rb.rp_prefix_workspace_bytes(dm.handle, B, cu_p))
    ws_s = dm.workspace(rb.rp_suffix_workspace_bytes(dm.handle, B, cu_p, cu_s))
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        dm.prefix(cu_p, ids, vis, kv=(K, V), h_last=h_last, workspace=ws_p, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        dm.suffix(cu_p, cu_s, K, V, h_last, resp, logprobs=lp[:R], workspace=ws_s, stream=stream)
        if ev is not None:
            ev[2].record(stream)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    log(f"timing {args.steps} steps")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        step(evs[i])
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    pre_ms = sorted(e[0].elapsed_time(e[1]) for e in evs)[args.steps // 2]
    suf_ms = sorted(e[1].elapsed_time(e[2]) for e in evs)[args.steps // 2]
    if not np.all(np.isfinite(lp[:R].cpu().numpy())):
        raise RuntimeError("non-finite log-probs")

    # per-kernel durations: HIP events around every launch, on the launch stream
    log(f"per-kernel timing over {args.profile_steps} steps")
    rb.rp_profile_reset()
    rb.rp_profile_enable(True, 4096)
    for _ in range(args.profile_steps):
        step()
        torch.cuda.synchronize()
        rb.rp_profile_collect()
    kern = rb.rp_profile_read_all()
    rb.rp_profile_enable(False)
    kernels = {k: {"launches": n, "avg_ms": ms / max(n, 1), "ms_per_step": ms / args.profile_steps}
               for k, (n, ms) in sorted(kern.items(), key=lambda kv: -kv[1][1])}

    pf = perf.prefix_flops(m, bt.prefix_lens)
    sf = perf.suffix_flops(m, bt.prefix_lens, bt.suffix_lens)
    peak = perf.PEAK_BF16_FLOPS if m.dtype == "bf16" else perf.PEAK_FP32_FLOPS
    gu_flops = perf.gemm_flops(T, 2 * m.ffn_dim, m.d_model)
    gu = kernels.get("prefix.gemm_gate_up")
    roofline = None
    if gu:
        ach = gu_flops / (gu["avg_ms"] * 1e-3) / 1e12
        roofline = {"kernel": "gemm_gate_up (prefix)", "bound": "mfma", "achieved": ach,
                    "peak": peak / 1e12, "unit": "TFLOP/s", "frac": ach / (peak / 1e12),
                    "traffic": None, "algorithmic_per_launch": gu_flops}
    ls = kernels.get("suffix.logsoftmax_gather")
    k12 = None
    if ls:
        gbs = perf.logsoftmax_bytes(R, m.vocab) / (ls["avg_ms"] * 1e-3) / 1e9
        k12 = {"bound": "hbm", "achieved": gbs, "peak": perf.PEAK_HBM_BPS / 1e9, "unit": "GB/s",
               "frac": gbs / (perf.PEAK_HBM_BPS / 1e9)}

    out = {
        "metric": "prefix prefill tokens/s + suffix logprob tokens/s; % bf16 MFMA peak",
        "value": (T + R) / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": m.dtype,
        "data": "synthetic (seeded; N(0,0.02) weights, N(0,1) visual embeddings, uniform ids)",
        "config": {"workload": w.name, "layers": m.n_layers, "d_model": m.d_model,
                   "q_heads": m.n_q_heads, "kv_heads": m.n_kv_heads, "head_dim": m.head_dim,
                   "ffn": m.ffn_dim, "vocab": m.vocab, "batch": B, "prefix_tokens": T,
                   "suffix_tokens": R, "parallelism": "single GPU"},
        "prefix_tokens_per_s": T / (pre_ms * 1e-3),
        "suffix_tokens_per_s": R / (suf_ms * 1e-3),
        "prefix_ms": pre_ms,
        "suffix_ms": suf_ms,
        "prefix_tflops": pf["total"] / (pre_ms * 1e-3) / 1e12,
        "prefix_mfma_frac": pf["total"] / (pre_ms * 1e-3) / peak,
        "suffix_tflops": sf["total"] / (suf_ms * 1e-3) / 1e12,
        "suffix_mfma_frac": sf["total"] / (suf_ms * 1e-3) / peak,
        "roofline": roofline,
        "logsoftmax_roofline": k12,
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        log("CPU baseline: oracle on sequence 0")
        out["cpu_baseline"] = cpu_baseline(w, hw, bt, args.cpu_prefix_len)
    dm.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
