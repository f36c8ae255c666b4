#!/usr/bin/env python3
"""Throughput of the prefix/suffix backbone path on one MI355X.

One step = the prefix pass (prompt prefill: KV + boundary state) followed by the
suffix pass (response log-probs over the cached KV) for one packed batch of
seeded synthetic inputs, all inputs resident in HBM.  Default workload: the
largest single-GPU configuration, the Qwen2.5-VL-32B-shaped 2-layer slice,
batch 2, prefix 16384 (15872 visual + 512 text), suffix 512.  The default run
also reports the 7B-slice workloads (uniform and ragged batches) under
"workloads" and the co-location arms of Eq. (1) under "colocation".

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
    if prefix_len < 0:  # automatic bound: about 10-30 s of float64 work on the host
        prefix_len = 4096 if w.model.d_model * w.model.n_layers * len(ids) > 4 * 3584 * 4096 else 0
    P = len(ids) if prefix_len <= 0 else min(prefix_len, len(ids))
    ids = ids[:P]
    vis = vis[:int((ids < 0).sum())]
    t0 = time.perf_counter()
    K, V, h, _ = oracle.prefix_forward_one(W, w.model, ids, vis)
    t1 = time.perf_counter()
    oracle.suffix_logprob_one(W, w.model, K, V, h, resp)
    t2 = time.perf_counter()
    pools = threadpool_info()
    threads = max([p.get("num_threads", 1) for p in pools] or [1])
    blas = ", ".join(sorted({f"{p.get('internal_api')} {p.get('version')}" for p in pools if p.get("user_api") == "blas"}))
    cpu = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    n_tok = P + len(resp)
    return {"value": n_tok / (t2 - t0), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"sequence 0 of the workload{'' if P == len(bt.token_ids[cp[0]:cp[1]]) else f' (its first {P} prefix tokens)'}: "
                      f"prefix {P} + suffix {len(resp)} tokens, all "
                      f"{w.model.n_layers} layers, float64 numpy oracle; prefix {t1 - t0:.1f} s, "
                      f"suffix {t2 - t1:.1f} s",
            "prefix_s": t1 - t0, "suffix_s": t2 - t1, "cpu_model": cpu, "numpy": np.__version__, "blas": blas}


def colocation(args, w):
    """Prefix pass on one stream beside repeated decode steps on another (one GPU).

    Arms: each alone on all CUs; co-run on two unmasked streams (the analog of the
    paper's MPS-Default, Section "Resource Sharing Policy"); co-run with disjoint CU
    masks giving decode k CUs (the analog of its static SM partitions).  Reports the
    decode slowdown delta_D and the critical-path saving S of Eq. (1).
    """
    import torch

    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd import inputs, perf
    from paper_2608_14498_amd.runtime import DeviceModel, to_device

    m = w.model
    spec = w.decode
    log(f"workload {w.name}: generating seeded inputs")
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    Bd, cap, kvl = spec["batch"], spec["cap"], spec["kv_len"]
    maxp = max(max(bt.prefix_lens), cap) + 1
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    ids = to_device(bt.token_ids, dev)
    vis = to_device(bt.visual, dev)
    cu_p = [int(x) for x in bt.cu_prefix]
    B, T = bt.batch, bt.T
    K, V = dm.alloc_kv(T)
    h_last = torch.empty((B, m.d_model), dtype=torch.float32, device=dev)
    ws_p = dm.workspace(rb.rp_prefix_workspace_bytes(dm.handle, B, cu_p))
    # decode state: the KV cache (N(0,1), drawn on the device with a seeded generator),
    # constant context: every step writes slot kv_len and attends to kv_len + 1 keys
    gen = torch.Generator(device=dev).manual_seed(w.index * 1000 + 20)
    shape = (m.n_layers, Bd, cap, m.n_kv_heads, m.head_dim)
    ck = torch.randn(shape, generator=gen, device=dev, dtype=torch.float32).to(dm.dtype)
    cv = torch.randn(shape, generator=gen, device=dev, dtype=torch.float32).to(dm.dtype)
    kv_len = torch.full((Bd,), kvl, dtype=torch.int32, device=dev)
    tok = torch.randint(0, m.vocab, (Bd,), generator=gen, device=dev, dtype=torch.int32)
    nxt = torch.empty(Bd, dtype=torch.int32, device=dev)
    ws_d = dm.workspace(rb.rp_decode_workspace_bytes(dm.handle, Bd, cap))
    kv_d = rb.make_kv(ck, cv, ck[0].numel())

    def prefix_on(stream):
        dm.prefix(cu_p, ids, vis, kv=(K, V), h_last=h_last, workspace=ws_p, stream=stream)

    def decode_on(stream, n):
        for _ in range(n):
            rb.rp_decode_step(dm.handle, stream.cuda_stream, Bd, kv_d, cap, kv_len, tok, None, nxt, ws_d,
                              ws_d.numel())

    def timed(fn, stream):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    main = torch.cuda.current_stream()
    for _ in range(2):
        prefix_on(main)
        decode_on(main, 3)
    torch.cuda.synchronize()
    T_P = min(timed(lambda: prefix_on(main), main) for _ in range(3))
    step_ms = min(timed(lambda: decode_on(main, 10), main) for _ in range(3)) / 10
    n_steps = max(1, int(round(T_P / step_ms)))
    log(f"prefix alone {T_P:.2f} ms, decode step alone {step_ms:.3f} ms -> {n_steps} steps per window")
    rb.rp_profile_reset()
    rb.rp_profile_enable(True, 4096)
    for _ in range(3):
        decode_on(main, 1)
        torch.cuda.synchronize()
        rb.rp_profile_collect()
    decode_kernels = {k: {"launches": n, "avg_ms": ms / max(n, 1), "ms_per_step": ms / 3}
                      for k, (n, ms) in sorted(rb.rp_profile_read_all().items(), key=lambda kv: -kv[1][1])}
    rb.rp_profile_enable(False)
    for k, v in decode_kernels.items():
        log(f"  decode kernel {k:24s} {v['ms_per_step']:.3f} ms/step")

    ncu = rb.rp_device_cu_count(0)
    words = (ncu + 31) // 32

    def mask(lo, hi):
        wv = [0] * words
        for i in range(lo, hi):
            wv[i // 32] |= 1 << (i % 32)
        return wv

    def corun(sa, sd, steps):
        """Returns (prefix ms, decode ms, makespan ms) with both enqueued together."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        torch.cuda.synchronize()
        ev[0].record(sa)
        ev[2].record(sd)
        prefix_on(sa)
        decode_on(sd, steps)
        ev[1].record(sa)
        ev[3].record(sd)
        torch.cuda.synchronize()
        t_p, t_d = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
        start_gap = ev[0].elapsed_time(ev[2])
        makespan = max(t_p, start_gap + t_d) - min(0.0, start_gap)
        return t_p, t_d, makespan

    arms = []
    for regime, steps in (("balanced", n_steps), ("prefix-bounded", max(1, n_steps // 2)),
                          ("decode-bounded", 2 * n_steps)):
        T_D = step_ms * steps
        streams = [("unmasked (MPS-Default analog)", torch.cuda.Stream(), torch.cuda.Stream(), None)]
        if regime == "balanced":
            for k in (32, 64, 80, 96, 112, 128):
                sd = rb.rp_stream_create_cu_masked(0, mask(0, k))
                sa = rb.rp_stream_create_cu_masked(0, mask(k, ncu))
                streams.append((f"decode {k} CUs / prefix {ncu - k} CUs", torch.cuda.ExternalStream(sa),
                                torch.cuda.ExternalStream(sd), (sa, sd)))
        for name, sa, sd, raw in streams:
            corun(sa, sd, steps)  # warm
            t_p, t_d, mk = min((corun(sa, sd, steps) for _ in range(3)), key=lambda r: r[2])
            model = perf.overlap_model(T_D, T_P, t_d - T_D)
            arms.append({"regime": regime, "arm": name, "decode_steps": steps, "T_P_alone_ms": T_P,
                         "T_D_alone_ms": T_D, "prefix_corun_ms": t_p, "decode_corun_ms": t_d,
                         "makespan_ms": mk, "delta_D_ms": t_d - T_D, "serial_ms": T_P + T_D,
                         "saving_measured_ms": T_P + T_D - mk, "saving_eq1_ms": model["saving"],
                         "eq1_regime": model["regime"],
                         "prefix_tokens_per_s": T / (t_p * 1e-3),
                         "decode_tokens_per_s": Bd * steps / (t_d * 1e-3)})
            log(f"{regime:15s} {name:36s} prefix {t_p:7.2f} ms decode {t_d:7.2f} ms makespan {mk:7.2f} "
                f"(serial {T_P + T_D:7.2f})")
            if raw:
                rb.rp_stream_destroy(raw[0])
                rb.rp_stream_destroy(raw[1])
    best = min((a for a in arms if a["regime"] == "balanced"), key=lambda a: a["makespan_ms"])
    serial = next(a for a in arms if a["regime"] == "balanced")
    out = {
        "metric": "co-location: prefix tokens/s and decode tokens/s co-running vs alone; Eq. (1) saving",
        "value": T / (best["makespan_ms"] * 1e-3),
        "unit": "prefix tokens/s over the co-run makespan",
        "n_gpus": 1, "steps": n_steps, "warmup": 2, "ms_per_step": best["makespan_ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": m.dtype,
        "data": "synthetic (seeded)",
        "config": {"workload": w.name, "prefix_batch": B, "prefix_len": bt.prefix_lens[0],
                   "decode_batch": Bd, "decode_kv": kvl, "cus": ncu},
        "prefix_alone_ms": T_P, "prefix_alone_tokens_per_s": T / (T_P * 1e-3),
        "decode_step_alone_ms": step_ms, "decode_alone_tokens_per_s": Bd / (step_ms * 1e-3),
        "decode_kernels": decode_kernels, "best_balanced_arm": best["arm"],
        "balanced_serial_ms": serial["serial_ms"], "balanced_best_makespan_ms": best["makespan_ms"],
        "balanced_best_saving_ms": best["saving_measured_ms"], "arms": arms,
    }
    dm.close()
    del K, V, ck, cv, ws_p, ws_d
    torch.cuda.empty_cache()
    return out


def measured_traffic(kernel_src: str, path: str, sha_key: str = "gemm_source_sha1"):
    """HBM bytes per launch of a kernel from the committed rocprofv3 counter runs, or None
    when the kernel source has changed since those counters were taken."""
    import hashlib

    try:
        rec = json.load(open(os.path.join(ROOT, path)))
        cur = hashlib.sha1(open(os.path.join(ROOT, kernel_src), "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    return rec["traffic_bytes_per_launch"] if rec.get(sha_key) == cur else None


HEADLINE = "qwen32b_b2_p16384_s512"
EXTRA_WORKLOADS = ("qwen7b_b4_p4096_s256", "qwen7b_ragged_b8")
COLOCATION = "qwen7b_coloc_p4x8192_d64"


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--profile-steps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-prefix-len", type=int, default=-1,
                    help="truncate the CPU-baseline sample prefix (0 = full, -1 = bounded automatically)")
    ap.add_argument("--dtype", choices=["bf16", "f16"], default=None,
                    help="run the workload's model in this 16-bit storage type (default: as named)")
    ap.add_argument("--f16-variant", action="store_true",
                    help="also time the workload with its model stored in fp16")
    ap.add_argument("--no-fused-variant", action="store_true",
                    help="skip timing the suffix with the fused lm_head + log-sum-exp scoring")
    ap.add_argument("--no-transposed-variant", action="store_true",
                    help="skip timing the step with o_proj / down weights stored transposed")
    ap.add_argument("--no-last-rows-variant", action="store_true",
                    help="skip timing the prefix with RP_PREFIX_LAST_ROWS_ONLY")
    ap.add_argument("--no-measured-peaks", action="store_true",
                    help="skip the matrix-core probe and the device-copy bandwidth measurement")
    ap.add_argument("--no-prompt-logprobs", action="store_true",
                    help="skip timing the prompt-token log-probs (rp_prompt_logprob)")
    ap.add_argument("--no-extra-workloads", action="store_true",
                    help="report the named workload only (no 7B-slice workloads, no co-location arms)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch

        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the path shards by "
              f"sequence and is measured on one GPU's share.", file=sys.stderr)
        sys.exit(2)

    from paper_2608_14498_amd import configs

    w = configs.get(args.workload)
    if args.dtype:
        w = configs.with_model(w, dtype=args.dtype)
    if w.decode is not None:
        print(json.dumps(colocation(args, w)), flush=True)
        return
    out = workload_record(w, args, headline=True)
    if not args.no_extra_workloads and args.workload == HEADLINE and not args.dtype:
        out["workloads"] = {}
        for name in EXTRA_WORKLOADS:
            out["workloads"][name] = workload_record(configs.get(name), args, headline=False)
        out["colocation"] = colocation(args, configs.get(COLOCATION))
    print(json.dumps(out), flush=True)


def workload_record(w, args, headline: bool) -> dict:
    """Time one prefix + suffix workload.  The headline record carries the contract's keys,
    the variants, the measured peaks and the CPU baseline; the others the throughputs, MFMA
    fractions and rooflines only."""
    from paper_2608_14498_amd import configs, perf

    m = w.model
    res = run_passes(w, args, profile=True, prompt=headline)
    T, R, B, kernels = res["T"], res["R"], res["B"], res["kernels"]
    ms_step, pre_ms, suf_ms = res["ms_step"], res["pre_ms"], res["suf_ms"]
    bt = res["bt"]

    pf = perf.prefix_flops(m, bt.prefix_lens)
    grp = bt.prefix_of_suffix
    pre_of_suf = bt.prefix_lens if grp is None else [bt.prefix_lens[g] for g in grp]
    sf = perf.suffix_flops(m, pre_of_suf, bt.suffix_lens)
    peak = perf.PEAK_FP32_FLOPS if m.dtype == "f32" else perf.PEAK_BF16_FLOPS
    gu_flops = perf.gemm_flops(T, 2 * m.ffn_dim, m.d_model)
    gu = kernels.get("prefix.gemm_gate_up")
    roofline = None
    if gu:
        ach = gu_flops / (gu["avg_ms"] * 1e-3) / 1e12
        traffic = None
        if m.dtype == "bf16":
            traffic = measured_traffic("paper_2608_14498_amd/csrc/gemm.hip",
                                       f"profiles/gemm_gate_up_{w.name}_traffic.json")
        roofline = {"kernel": "prefix.gemm_gate_up (fused SwiGLU)", "bound": "mfma", "achieved": ach,
                    "peak": peak / 1e12, "unit": "TFLOP/s", "frac": ach / (peak / 1e12),
                    "traffic": traffic, "algorithmic_per_launch": gu_flops,
                    "algorithmic_per_unit": "2 * 2F * d flop per prefix token (T tokens per launch)",
                    "algorithmic_bytes_per_launch": 2 * (T * m.d_model + 2 * m.ffn_dim * m.d_model
                                                         + T * m.ffn_dim)}
    ls = kernels.get("suffix.logsoftmax_gather")
    k12 = None
    if ls:
        gbs = perf.logsoftmax_bytes(R, m.vocab) / (ls["avg_ms"] * 1e-3) / 1e9
        k12 = {"bound": "hbm", "achieved": gbs, "peak": perf.PEAK_HBM_BPS / 1e9, "unit": "GB/s",
               "frac": gbs / (perf.PEAK_HBM_BPS / 1e9), "algorithmic_bytes_per_launch": perf.logsoftmax_bytes(R, m.vocab),
               "traffic": None}
        if m.dtype == "bf16":
            k12["traffic"] = measured_traffic("paper_2608_14498_amd/csrc/elementwise.hip",
                                              f"profiles/logsoftmax_gather_{w.name}_traffic.json",
                                              "elementwise_source_sha1")

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
                   "suffix_tokens": R, "parallelism": "single GPU",
                   **({} if bt.prefix_of_suffix is None else
                      {"responses_per_prompt": w.group, "responses": len(bt.suffix_lens)})},
        "prefix_tokens_per_s": T / (pre_ms * 1e-3),
        "suffix_tokens_per_s": R / (suf_ms * 1e-3),
        "prefix_ms": pre_ms,
        "suffix_ms": suf_ms,
        "prefix_tflops": pf["total"] / (pre_ms * 1e-3) / 1e12,
        "prefix_mfma_frac": pf["total"] / (pre_ms * 1e-3) / peak,
        "suffix_tflops": sf["total"] / (suf_ms * 1e-3) / 1e12,
        "suffix_mfma_frac": sf["total"] / (suf_ms * 1e-3) / peak,
        "step_ms": res["step_stats"],
        "roofline": roofline,
        "logsoftmax_roofline": k12,
    }
    if not headline:
        out["kernels"] = {k: v for k, v in kernels.items() if v["ms_per_step"] >= 0.05}
        return out
    out["prompt_logprobs"] = res["prompt"]
    out["kernels"] = kernels
    if m.dtype == "bf16" and args.f16_variant:
        # the same model stored in fp16 (bf16 weights converted exactly): same kernels with
        # fp16 MFMA
        wf = configs.with_model(w, dtype="f16")
        rf = run_passes(wf, args, profile=False)
        out["f16_variant"] = {
            "value": (rf["T"] + rf["R"]) / (rf["ms_step"] * 1e-3), "unit": "tokens/s",
            "ms_per_step": rf["ms_step"], "prefix_ms": rf["pre_ms"], "suffix_ms": rf["suf_ms"],
            "prefix_mfma_frac": pf["total"] / (rf["pre_ms"] * 1e-3) / perf.PEAK_BF16_FLOPS}
    if m.dtype != "f32" and not args.no_fused_variant:
        # the suffix scored by the lm_head with an online log-sum-exp epilogue: the [R, V]
        # logits are never stored (RP_SUFFIX_FUSED_LOGPROB)
        from paper_2608_14498_amd import binding as rb

        rfu = run_passes(w, args, profile=False, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
        out["fused_logprob_variant"] = {
            "value": (rfu["T"] + rfu["R"]) / (rfu["ms_step"] * 1e-3), "unit": "tokens/s",
            "ms_per_step": rfu["ms_step"], "suffix_ms": rfu["suf_ms"],
            "suffix_tokens_per_s": rfu["R"] / (rfu["suf_ms"] * 1e-3)}
    if m.dtype != "f32" and not args.no_transposed_variant:
        # the row-parallel projections (o_proj, down) stored transposed and read in
        # transpose mode (Case 2 weight sharing), same results bit for bit
        from paper_2608_14498_amd import binding as rb

        rt = run_passes(w, args, profile=True, weight_layout=rb.RP_WO_TRANSPOSED | rb.RP_W_DOWN_TRANSPOSED)
        kt = rt["kernels"]
        out["transposed_weights_variant"] = {
            "value": (rt["T"] + rt["R"]) / (rt["ms_step"] * 1e-3), "unit": "tokens/s",
            "ms_per_step": rt["ms_step"], "prefix_ms": rt["pre_ms"], "suffix_ms": rt["suf_ms"],
            "kernels": {k: kt[k] for k in ("prefix.gemm_o_proj", "prefix.gemm_down", "suffix.gemm_o_proj",
                                           "suffix.gemm_down") if k in kt}}
    if not args.no_last_rows_variant:
        # labelled optimisation: the last layer carries only each sequence's last row past
        # its K/V projection (all the suffix pass reads); TFLOP/s counts executed flops
        from paper_2608_14498_amd import binding as rb

        rl = run_passes(w, args, profile=True, prefix_flags=rb.RP_PREFIX_LAST_ROWS_ONLY)
        pfl = perf.prefix_flops(m, bt.prefix_lens, last_rows_only=True)
        kl = rl["kernels"]
        out["last_rows_only_variant"] = {
            "label": "prefix last layer past K/V only at each sequence's last row (RP_PREFIX_LAST_ROWS_ONLY)",
            "value": (rl["T"] + rl["R"]) / (rl["ms_step"] * 1e-3), "unit": "tokens/s",
            "ms_per_step": rl["ms_step"], "prefix_ms": rl["pre_ms"], "suffix_ms": rl["suf_ms"],
            "prefix_tokens_per_s": rl["T"] / (rl["pre_ms"] * 1e-3),
            "prefix_executed_tflop": pfl["total"] / 1e12,
            "prefix_tflops": pfl["total"] / (rl["pre_ms"] * 1e-3) / 1e12,
            "prefix_mfma_frac": pfl["total"] / (rl["pre_ms"] * 1e-3) / peak,
            "kernels": {k: v for k, v in kl.items() if k.startswith("prefix.tail")}}
    if not args.no_measured_peaks:
        mp = measured_peaks()
        out["measured_peaks"] = mp
        if roofline and m.dtype == "bf16":
            roofline["frac_of_measured_peak"] = roofline["achieved"] / mp["mfma_bf16_tflops"]
        if k12:
            k12["frac_of_measured_read"] = k12["achieved"] / mp["hbm_read_gbps"]
    if not args.no_cpu_baseline:
        log("CPU baseline: oracle on sequence 0")
        out["cpu_baseline"] = cpu_baseline(w, res["hw"], bt, args.cpu_prefix_len)
    return out


def run_passes(w, args, profile: bool, flags: int = 0, weight_layout: int = 0, prompt: bool = False,
               prefix_flags: int = 0):
    """Time prefix + suffix steps of workload w; optionally per-kernel durations and the
    prompt-token log-probs."""
    import numpy as np
    import torch

    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd import inputs
    from paper_2608_14498_amd.runtime import DeviceModel, to_device

    m = w.model
    log(f"workload {w.name} ({m.dtype}): generating seeded inputs")
    t0 = time.time()
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    log(f"inputs ready in {time.time() - t0:.1f} s; uploading")
    grp = bt.prefix_of_suffix
    pre_of_suf = bt.prefix_lens if grp is None else [bt.prefix_lens[g] for g in grp]
    maxp = max(p + s for p, s in zip(pre_of_suf, bt.suffix_lens)) + 1
    dm = DeviceModel(hw, maxp, weight_layout=weight_layout)
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
    grouped = grp is not None or flags != 0
    if not grouped:
        ws_s = dm.workspace(rb.rp_suffix_workspace_bytes(dm.handle, B, cu_p, cu_s))
    else:
        grp_l = [int(g) for g in grp] if grp is not None else list(range(B))
        ws_s = dm.workspace(rb.rp_suffix_grouped_workspace_bytes(dm.handle, B, cu_p, len(grp_l), grp_l, cu_s,
                                                                 flags))
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        dm.prefix(cu_p, ids, vis, kv=(K, V), h_last=h_last, workspace=ws_p, stream=stream, flags=prefix_flags)
        if ev is not None:
            ev[1].record(stream)
        if not grouped:
            dm.suffix(cu_p, cu_s, K, V, h_last, resp, logprobs=lp[:R], workspace=ws_s, stream=stream)
        else:
            dm.suffix_grouped(cu_p, grp_l, cu_s, K, V, h_last, resp, logprobs=lp[:R], workspace=ws_s,
                              stream=stream, flags=flags)
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
    st = sorted(e[0].elapsed_time(e[2]) for e in evs)
    step_stats = {"median": st[len(st) // 2], "mean": sum(st) / len(st), "min": st[0]}
    if not np.all(np.isfinite(lp[:R].cpu().numpy())):
        raise RuntimeError("non-finite log-probs")

    kernels = {}
    if profile:
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
    prompt_res = None
    if prompt and not args.no_prompt_logprobs:
        prompt_res = time_prompt_logprobs(dm, args, bt, cu_p, ids, vis, (K, V), h_last, ws_p, stream)
    dm.close()
    del K, V, ids, vis, resp, ws_p, ws_s
    torch.cuda.empty_cache()
    return dict(T=T, R=R, B=B, bt=bt, hw=hw, ms_step=ms_step, pre_ms=pre_ms, suf_ms=suf_ms, kernels=kernels,
                step_stats=step_stats,
                prompt=prompt_res)


def measured_peaks():
    """Matrix-core rate of the MFMA probe (random bf16 operands, two waves per SIMD, about
    25 ms) and the HBM read bandwidth of a 4 GiB streaming read, on this GPU: the practical
    ceilings beside the published peaks."""
    import torch

    from paper_2608_14498_amd import binding as rb

    log("measured peaks: MFMA probe and HBM read probe")
    stream = torch.cuda.current_stream()
    cus = rb.rp_device_cu_count(0)
    blocks = 2 * cus
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    rb.rp_calibrate_mfma(stream.cuda_stream, "bf16", blocks, 2000, sink, sink.numel() * 4)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    flops = rb.rp_calibrate_mfma(stream.cuda_stream, "bf16", blocks, 100000, sink, sink.numel() * 4)
    b.record(stream)
    torch.cuda.synchronize()
    mfma = flops / (a.elapsed_time(b) * 1e-3) / 1e12
    if not bool(torch.isfinite(sink).all()):
        raise RuntimeError("MFMA probe produced non-finite sums")
    n = 4 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    rblocks = 16 * cus
    rsink = torch.empty(rblocks * 256, dtype=torch.int32, device="cuda")
    rb.rp_calibrate_read(stream.cuda_stream, src, n, rblocks, rsink, rsink.numel() * 4)
    a.record(stream)
    for _ in range(3):
        rb.rp_calibrate_read(stream.cuda_stream, src, n, rblocks, rsink, rsink.numel() * 4)
    b.record(stream)
    torch.cuda.synchronize()
    read = 3.0 * n / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, rsink, sink
    torch.cuda.empty_cache()
    return {"mfma_bf16_tflops": mfma, "mfma_probe": f"{blocks} workgroups x 4 waves, 100000 x 8 MFMA 32x32x16 each",
            "hbm_read_gbps": read, "read_probe": f"4 GiB streamed by {rblocks} workgroups, 16-byte loads"}


def time_prompt_logprobs(dm, args, bt, cu_p, ids, vis, kv, h_last, ws_p, stream):
    """Teacher-forced log-probs of every prompt text token, scored from the prefix pass's
    hidden states (rp_prompt_logprob), plain and with the fused lm_head scoring."""
    import numpy as np
    import torch

    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd.runtime import prompt_positions, to_device

    m = dm.shape
    hidden = torch.empty((bt.T, m.d_model), dtype=torch.float32, device=dm.device)
    dm.prefix(cu_p, ids, vis, kv=kv, h_last=h_last, hidden_out=hidden, workspace=ws_p, stream=stream)
    pos = to_device(prompt_positions(cu_p, bt.token_ids), dm.device)
    n = int(pos.numel())
    out = {"rows": n}
    variants = [("plain", 0)] + ([("fused", rb.RP_SUFFIX_FUSED_LOGPROB)] if m.dtype != "f32" else [])
    for name, flags in variants:
        ws = dm.workspace(rb.rp_prompt_logprob_workspace_bytes(dm.handle, n, flags))
        lp = torch.empty(max(n, 1), dtype=torch.float32, device=dm.device)[:n]
        for _ in range(2):
            dm.prompt_logprobs(cu_p, ids, hidden, pos, logprobs=lp, workspace=ws, stream=stream, flags=flags)
        reps = max(args.steps, 5)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            dm.prompt_logprobs(cu_p, ids, hidden, pos, logprobs=lp, workspace=ws, stream=stream, flags=flags)
        b.record(stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        if not np.all(np.isfinite(lp.cpu().numpy())):
            raise RuntimeError("non-finite prompt log-probs")
        out[f"{name}_ms"] = ms
        out[f"{name}_rows_per_s"] = n / (ms * 1e-3)
        del ws, lp
    del hidden
    log(f"prompt log-probs: {out}")
    return out


if __name__ == "__main__":
    main()
