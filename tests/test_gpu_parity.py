"""GPU parity: the HIP path (through the C ABI) against the float64 CPU oracle.

Tolerances: |d logprob| <= 1e-4 for the fp32 model and <= 2e-2 for the 16-bit models
(fp32 accumulation), as required of the path.  A bf16 case that misses 2e-2 must stay
within the error of an ideal bf16 implementation of the same tokens (TargetCheck in
tests/gpu_helpers.py, computed by tests/bf16_emulation.py) and is then reported as an
expected failure naming both values.  KV and h_last are compared as
max error relative to the largest reference magnitude: bf16 storage of K/V alone
contributes up to 2^-9 relative per element, and activations are rounded to bf16
between kernels, so 3e-2 bounds the bf16 cases; the fp32 model must match to 1e-5.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from paper_2608_14498_amd import configs, inputs
from tests.gpu_helpers import TargetCheck, emulated_suffix, gpu_run, max_abs, oracle_run, rel_err

pytestmark = pytest.mark.gpu


def _report(name, K, V, H, lp, Ko, Vo, Ho, lpo):
    r = dict(kv=max(rel_err(K, Ko), rel_err(V, Vo)), h=rel_err(H, Ho), lp=max_abs(lp, lpo))
    print(f"[parity] {name}: {r}", flush=True)
    return r


def test_tiny_fp32_config_matches_oracle():
    w = configs.get("tiny_f32")
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    got = gpu_run(w, hw, bt)
    ref = oracle_run(w, hw, bt)
    r = _report("tiny_f32", *got, *ref)
    assert r["lp"] <= 1e-4
    assert r["kv"] <= 1e-5 and r["h"] <= 1e-5


BF16_SMALL = configs.ModelShape(n_layers=2, d_model=384, n_q_heads=6, n_kv_heads=2, head_dim=128,
                                ffn_dim=768, vocab=1000, dtype="bf16")
BF16_D64 = configs.ModelShape(n_layers=2, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=64,
                              ffn_dim=512, vocab=2051, dtype="bf16")
# wide enough (K >= 2048) that the suffix GEMMs split K and SwiGLU runs unfused; two layers,
# so that the down projection's partials are summed by the next layer's attention norm
BF16_WIDE = configs.ModelShape(n_layers=2, d_model=2048, n_q_heads=16, n_kv_heads=2, head_dim=128,
                               ffn_dim=4096, vocab=1000, dtype="bf16")
# contraction depths of 5, 3 and 7 slabs of 64 (q/k/v and gate/up, O-proj, down) and of 2,
# 2 and 1: the tiled GEMM's slab ring ends after every possible remainder, and on the
# shortest K ranges its prologue re-loads the last slab
BF16_ODD_K = configs.ModelShape(n_layers=2, d_model=320, n_q_heads=3, n_kv_heads=1, head_dim=64,
                                ffn_dim=448, vocab=1000, dtype="bf16")
BF16_SHORT_K = configs.ModelShape(n_layers=2, d_model=128, n_q_heads=2, n_kv_heads=1, head_dim=64,
                                  ffn_dim=64, vocab=1000, dtype="bf16")
# the same models stored in fp16 (same kernels, fp16 MFMA)
F16_SMALL = replace(BF16_SMALL, dtype="f16")
F16_D64 = replace(BF16_D64, dtype="f16")
F16_WIDE = replace(BF16_WIDE, dtype="f16")


@pytest.mark.parametrize("model,norm,bias", [(BF16_SMALL, "ones", False), (BF16_SMALL, "random", True),
                                             (BF16_D64, "random", True), (BF16_WIDE, "random", True),
                                             (BF16_ODD_K, "random", True), (BF16_SHORT_K, "random", True),
                                             (F16_SMALL, "random", True), (F16_D64, "random", True),
                                             (F16_WIDE, "random", True)])
def test_bf16_ragged_batch_matches_oracle(model, norm, bias):
    P, Vis, S = [1, 70, 300, 129], [0, 60, 256, 100], [3, 0, 65, 130]
    w = configs.custom(model, P, Vis, S, index=41)
    hw = inputs.make_weights(w, norm=norm, bias=bias)
    bt = inputs.make_batch(w)
    got = gpu_run(w, hw, bt)
    ref = oracle_run(w, hw, bt)
    name = f"{model.dtype} d={model.d_model} D={model.head_dim} {norm} bias={bias}"
    r = _report(name, *got, *ref)
    assert r["kv"] <= 3e-2 and r["h"] <= 3e-2
    chk = TargetCheck(model.dtype)
    chk.check(name, got[3], ref[3], lambda: emulated_suffix(w, hw, bt))
    chk.finish()


def test_fp32_ragged_edges_match_oracle():
    model = configs.TINY
    P, Vis, S = [1, 65, 200], [1, 0, 190], [2, 1, 0]
    w = configs.custom(model, P, Vis, S, index=43)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    got = gpu_run(w, hw, bt)
    ref = oracle_run(w, hw, bt)
    r = _report("fp32 edges", *got, *ref)
    assert r["lp"] <= 1e-4 and r["kv"] <= 1e-5 and r["h"] <= 1e-5


@pytest.mark.parametrize("model", [BF16_SMALL, configs.TINY, BF16_WIDE, F16_WIDE])
def test_packing_is_bitwise_invariant(model):
    """A packed ragged batch gives exactly the per-sequence results of running each alone."""
    P, Vis, S = [90, 257, 3], [80, 200, 0], [17, 40, 5]
    w = configs.custom(model, P, Vis, S, index=47)
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    K, V, H, lp = gpu_run(w, hw, bt, max_position=400)
    for b in range(3):
        cp, cs = bt.cu_prefix, bt.cu_suffix
        vo = sum(Vis[:b])
        one = inputs.HostBatch([P[b]], [Vis[b]], [S[b]], np.array([0, P[b]], np.int32),
                               np.array([0, S[b]], np.int32), bt.token_ids[cp[b]:cp[b + 1]],
                               bt.visual[vo:vo + Vis[b]], bt.response_ids[cs[b]:cs[b + 1]])
        k1, v1, h1, lp1 = gpu_run(w, hw, one, max_position=400)
        assert np.array_equal(K[:, cp[b]:cp[b + 1]], k1)
        assert np.array_equal(V[:, cp[b]:cp[b + 1]], v1)
        assert np.array_equal(H[b], h1[0])
        assert np.array_equal(lp[cs[b]:cs[b + 1]], lp1)


@pytest.mark.parametrize("model", [BF16_SMALL, F16_D64])
def test_split_kv_suffix_matches_oracle_and_is_bitwise_invariant(model):
    """Prefixes long enough that the suffix attention splits each sequence's keys (4096
    keys a split: 1, 1, 3 and 2 ways here) next to ones that do not split.  Matches the
    oracle; each sequence run alone gives bitwise its packed result (the split count is a
    function of the sequence's prefix length alone); and responses scored against a
    shared prefix equal bitwise the plain pass over a copy of it."""
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    P, Vis, S = [4100, 300, 12300, 8300], [0, 0, 0, 0], [130, 5, 300, 1]
    w = configs.custom(model, P, Vis, S, index=67)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    maxp = max(P) + max(S) + 1
    K, V, H, lp = gpu_run(w, hw, bt, max_position=maxp)
    for b in range(len(P)):
        cp, cs = bt.cu_prefix, bt.cu_suffix
        one = inputs.HostBatch([P[b]], [0], [S[b]], np.array([0, P[b]], np.int32), np.array([0, S[b]], np.int32),
                               bt.token_ids[cp[b]:cp[b + 1]], bt.visual[:0], bt.response_ids[cs[b]:cs[b + 1]])
        k1, v1, h1, lp1 = gpu_run(w, hw, one, max_position=maxp)
        assert np.array_equal(lp[cs[b]:cs[b + 1]], lp1), b
        assert np.array_equal(H[b], h1[0]), b
    # two responses on prefix 2 and one on prefix 3, grouped vs over copies of the prefix
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    cp = [int(x) for x in bt.cu_prefix]
    Kd, Vd, hd = dm.prefix(cp, to_device(bt.token_ids, dev), None)
    grp, lens = [2, 3, 2], [40, 7, 129]
    gcs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    resp = np.random.default_rng(68).integers(0, model.vocab, int(gcs[-1])).astype(np.int32)
    rd = to_device(resp, dev)
    lpg = dm.suffix_grouped(cp, grp, gcs.tolist(), Kd, Vd, hd, rd)
    Kc = torch.cat([Kd[:, cp[g]:cp[g + 1]] for g in grp], dim=1).contiguous()
    Vc = torch.cat([Vd[:, cp[g]:cp[g + 1]] for g in grp], dim=1).contiguous()
    hc = hd[torch.as_tensor(grp, device=dev).long()].contiguous()
    ccu = np.concatenate([[0], np.cumsum([P[g] for g in grp])]).astype(np.int32).tolist()
    lpc = dm.suffix(ccu, gcs.tolist(), Kc, Vc, hc, rd)
    torch.cuda.synchronize()
    assert torch.equal(lpg, lpc)
    dm.close()
    ref = oracle_run(w, hw, bt)
    name = f"split-KV {model.dtype} D={model.head_dim}"
    r = _report(name, K, V, H, lp, *ref)
    assert r["kv"] <= 3e-2 and r["h"] <= 3e-2
    chk = TargetCheck(model.dtype)
    chk.check(name, lp, ref[3], lambda: emulated_suffix(w, hw, bt))
    chk.finish()


# A GPU run that included the bf16 decode step at head_dim 64 and the last-rows-only
# prefix at head_dim 64 with 1-D positions faulted (illegal memory access) and no cause has
# been shown; the library returns RP_ERR_UNSUPPORTED for both until one is, and these cases
# stay skipped (they must not run on a GPU before a cause is found and fixed).
UNEXPLAINED_FAULT = pytest.mark.skip(reason="disabled in the library (RP_ERR_UNSUPPORTED): a GPU memory fault "
                                            "in a run that included this combination has no known cause")


@pytest.mark.parametrize("model,cap,lens", [(BF16_SMALL, 300, [0, 1, 63, 256, 299]),
                                            (configs.TINY, 300, [0, 1, 63, 256, 299]),
                                            (F16_SMALL, 300, [0, 1, 63, 256, 299]),
                                            # 1024-key chunks (16-bit: three per workgroup),
                                            # chunk and workgroup edges
                                            (BF16_SMALL, 1100, [511, 512, 1023, 700, 1099]),
                                            (configs.TINY, 1100, [0, 513, 1024, 1099, 5]),
                                            (BF16_SMALL, 3300, [1023, 1024, 2047, 3071, 3072, 3299, 0]),
                                            (configs.TINY, 3300, [3072, 2048, 1, 3299]),
                                            (F16_D64, 400, [0, 131, 399]),
                                            pytest.param(BF16_D64, 400, [0, 131, 399], marks=UNEXPLAINED_FAULT)])
def test_decode_step_matches_oracle(model, cap, lens):
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    w = configs.custom(model, [1], [0], [1], index=53)
    hw = inputs.make_weights(w, norm="random", bias=True)
    B = len(lens)
    kv_len = np.array(lens, np.int32)
    dec = inputs.make_decode(w, batch=B, kv_len=kv_len, cap=cap)
    dm = DeviceModel(hw, cap + 1)
    ck, cv = to_device(dec.cache_k, dm.device), to_device(dec.cache_v, dm.device)
    logits = torch.empty((B, model.vocab), dtype=torch.float32, device=dm.device)
    nxt = dm.decode(ck, cv, to_device(dec.kv_len, dm.device), to_device(dec.token_ids, dm.device), logits=logits)
    torch.cuda.synchronize()
    W = hw.as_f32()
    lo, no, nk, nv = oracle.decode_step(W, model, inputs.to_f32(dec.cache_k), inputs.to_f32(dec.cache_v),
                                        dec.kv_len, dec.token_ids)
    lg = logits.cpu().numpy()
    tol = 1e-4 if model.dtype == "f32" else 2e-2
    err = max_abs(lg, lo)
    print(f"[parity] decode {model.dtype}: logits max|d|={err}", flush=True)
    assert err <= tol
    got_ids = nxt.cpu().numpy()
    # no logits buffer: 16-bit models take the argmax inside the lm_head product; the same
    # step again (it rewrites the same cache slot with the same values) picks the same ids
    nxt2 = dm.decode(ck, cv, to_device(dec.kv_len, dm.device), to_device(dec.token_ids, dm.device))
    torch.cuda.synchronize()
    assert np.array_equal(nxt2.cpu().numpy(), got_ids)
    for b in range(B):
        top2 = np.sort(lo[b])[-2:]
        if top2[1] - top2[0] > 2 * tol:
            assert got_ids[b] == no[b]
        else:  # near tie: the GPU's choice must be (near-)maximal
            assert lo[b, got_ids[b]] >= top2[1] - 2 * tol
    ckg = ck.float().cpu().numpy()
    for b in range(B):
        s = kv_len[b]
        assert rel_err(ckg[:, b, s], nk[:, b]) <= (1e-5 if model.dtype == "f32" else 3e-2)
    # slots other than the new one are untouched
    mask = np.ones(cap, bool)
    ref_k = inputs.to_f32(dec.cache_k)
    for b in range(B):
        mask[:] = True
        mask[kv_len[b]] = False
        assert np.array_equal(ckg[:, b, mask], ref_k[:, b, mask])
    dm.close()


@pytest.mark.parametrize("model", [BF16_SMALL, configs.TINY, F16_D64, BF16_WIDE, F16_WIDE])
def test_shared_prefix_suffix_matches_oracle_and_duplicated_prefix(model):
    """GRPO groups: several responses scored against one prefix pass (Section "Prefix
    Sharing").  Matches the oracle, and is bitwise the plain suffix pass run over a copy
    of each response's prefix KV and boundary state."""
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    P, Vis = [70, 129, 33], [40, 100, 0]
    w = configs.custom(model, P, Vis, [1, 1, 1], index=61)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    grp = np.array([1, 0, 1, 1, 0, 1], np.int32)   # prefix 1 serves four responses, prefix 2 none
    lens = [5, 0, 65, 1, 17, 30]
    cs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    resp = np.random.default_rng(62).integers(0, model.vocab, int(cs[-1])).astype(np.int32)
    cp = [int(x) for x in bt.cu_prefix]
    dm = DeviceModel(hw, max(P) + max(lens) + 1)
    dev = dm.device
    K, V, h = dm.prefix(cp, to_device(bt.token_ids, dev), to_device(bt.visual, dev))
    rd = to_device(resp, dev)
    lp = dm.suffix_grouped(cp, grp.tolist(), cs.tolist(), K, V, h, rd)
    # the same responses over an explicit copy of each one's prefix
    Kd = torch.cat([K[:, cp[g]:cp[g + 1]] for g in grp], dim=1).contiguous()
    Vd = torch.cat([V[:, cp[g]:cp[g + 1]] for g in grp], dim=1).contiguous()
    hd = h[torch.as_tensor(grp, device=dev).long()].contiguous()
    dcu = np.concatenate([[0], np.cumsum([P[g] for g in grp])]).astype(np.int32).tolist()
    lpd = dm.suffix(dcu, cs.tolist(), Kd, Vd, hd, rd)
    torch.cuda.synchronize()
    assert torch.equal(lp, lpd)
    W = hw.as_f32()
    Ko, Vo, Ho = oracle.prefix_forward(W, model, bt.cu_prefix, bt.token_ids, inputs.to_f32(bt.visual))
    lpo = oracle.suffix_logprob_grouped(W, model, bt.cu_prefix, grp, cs, Ko, Vo, Ho, resp)
    got = lp.cpu().numpy()
    dm.close()
    print(f"[parity] shared prefix {model.dtype}: max|d logprob| = {max_abs(got, lpo)}", flush=True)
    from types import SimpleNamespace
    grouped = SimpleNamespace(cu_prefix=bt.cu_prefix, token_ids=bt.token_ids, visual=bt.visual, cu_suffix=cs,
                              response_ids=resp)
    chk = TargetCheck(model.dtype)
    chk.check(f"shared prefix {model.dtype} d={model.d_model}", got, lpo,
              lambda: emulated_suffix(w, hw, grouped, prefix_of_suffix=grp))
    chk.finish()


@pytest.mark.parametrize("model", [BF16_SMALL, BF16_D64, F16_SMALL])
def test_fused_logprob_scoring_matches_plain_and_oracle(model):
    """lm_head with the online log-sum-exp epilogue (RP_SUFFIX_FUSED_LOGPROB): the same
    log-probs as storing the logits and running the log-softmax kernel, up to fp32
    summation order; vocabularies 1000 and 2051 leave partial 256-column tiles."""
    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    P, Vis, S = [1, 70, 300, 129], [0, 60, 256, 100], [3, 0, 65, 130]
    w = configs.custom(model, P, Vis, S, index=71)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    dm = DeviceModel(hw, max(p + s for p, s in zip(P, S)) + 1)
    dev = dm.device
    cp, cs = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    K, V, h = dm.prefix(cp, to_device(bt.token_ids, dev), to_device(bt.visual, dev))
    rid = to_device(bt.response_ids, dev)
    lp = dm.suffix(cp, cs, K, V, h, rid)
    lpf = dm.suffix_grouped(cp, list(range(len(P))), cs, K, V, h, rid, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
    torch.cuda.synchronize()
    d = float((lpf - lp).abs().max().item())
    W = hw.as_f32()
    Ko, Vo, Ho = oracle.prefix_forward(W, model, bt.cu_prefix, bt.token_ids, inputs.to_f32(bt.visual))
    lpo = oracle.suffix_logprob(W, model, bt.cu_prefix, bt.cu_suffix, Ko, Vo, Ho, bt.response_ids)
    err = max_abs(lpf.cpu().numpy(), lpo)
    print(f"[parity] fused scoring {model.dtype} V={model.vocab}: vs plain {d}, vs oracle {err}", flush=True)
    assert d <= 1e-5
    assert err <= 2e-2
    dm.close()


@pytest.mark.parametrize("model,sections", [(BF16_SMALL, (16, 24, 24)), (configs.TINY, (8, 12, 12)),
                                            (F16_SMALL, (16, 24, 24))])
def test_mrope_prefix_and_suffix_match_oracle(model, sections):
    """Multimodal RoPE: visual tokens of a video grid at 3-D positions, text after them, the
    responses continuing at each prefix's next rotary position."""
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    from tests.test_oracle_pins import video_positions
    P, Vis, S = [70, 300, 129], [60, 256, 100], [9, 65, 0]
    grids = [(3, 4, 5), (4, 8, 8), (4, 5, 5)]
    w = configs.custom(model, P, Vis, S, index=81)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    pos, nxt = zip(*[video_positions(v, p - v, g) for p, v, g in zip(P, Vis, grids)])
    pos3 = np.concatenate(pos, axis=1).astype(np.int32)              # [3, T]
    maxp = max(max(int(n) + s for n, s in zip(nxt, S)), max(p + s for p, s in zip(P, S))) + 1
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    cp, cs = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    K, V, h = dm.prefix(cp, to_device(bt.token_ids, dev), to_device(bt.visual, dev),
                        positions=torch.as_tensor(pos3, device=dev).contiguous(), mrope_section=list(sections))
    lp = dm.suffix_grouped(cp, list(range(len(P))), cs, K, V, h, to_device(bt.response_ids, dev),
                           rope_pos0=[int(n) for n in nxt])
    torch.cuda.synchronize()
    W = hw.as_f32()
    vo = np.concatenate([[0], np.cumsum(Vis)])
    vis = inputs.to_f32(bt.visual)
    errs = dict(k=0.0, lp=0.0)
    for b in range(len(P)):
        ids = bt.token_ids[cp[b]:cp[b + 1]]
        k, v, hl, _ = oracle.prefix_forward_one(W, model, ids, vis[vo[b]:vo[b + 1]], mrope=(pos[b], sections))
        errs["k"] = max(errs["k"], rel_err(K[:, cp[b]:cp[b + 1]].float().cpu().numpy(), k))
        lpo = oracle.suffix_logprob_one(W, model, k, v, hl, bt.response_ids[cs[b]:cs[b + 1]], rope_start=nxt[b])
        errs["lp"] = max(errs["lp"], max_abs(lp[cs[b]:cs[b + 1]].cpu().numpy(), lpo))
    print(f"[parity] mrope {model.dtype} D={model.head_dim}: {errs}", flush=True)
    f32 = model.dtype == "f32"
    assert errs["lp"] <= (1e-4 if f32 else 2e-2)
    assert errs["k"] <= (1e-5 if f32 else 3e-2)
    dm.close()


@pytest.mark.parametrize("model,flags", [(configs.TINY, 0), (BF16_D64, 0), (BF16_D64, 1), (F16_SMALL, 1)])
def test_prompt_logprobs_match_oracle(model, flags):
    """Prompt-token log-probs from the prefix pass's hidden states: every text position of
    ragged prompts laid out text, visual, text (one all-visual), repeated and shuffled, plus
    positions that score nothing (first tokens, visual slots, out of range: NaN)."""
    from paper_2608_14498_amd.runtime import DeviceModel, prompt_positions, to_device
    P, Vis = [1, 70, 300, 129, 40], [0, 60, 256, 100, 40]
    w = configs.custom(model, P, Vis, [0] * len(P), index=83)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    cp = [int(x) for x in bt.cu_prefix]
    T = cp[-1]
    ids = bt.token_ids.copy()
    for b in range(len(P)):
        seg = ids[cp[b]:cp[b + 1]]
        text = seg[seg >= 0]
        a = len(text) // 3
        ids[cp[b]:cp[b + 1]] = np.concatenate([text[:a], np.full(Vis[b], -1, np.int32), text[a:]])
    good = prompt_positions(cp, ids)
    bad = np.array([0, cp[1], cp[2], cp[1] + 5, cp[4] + 7, T, -1, T + 9], np.int32)
    pos = np.concatenate([good, bad, good[:7]]).astype(np.int32)
    np.random.default_rng(5).shuffle(pos)
    dm = DeviceModel(hw, max(P) + 1)
    dev = dm.device
    ids_d = to_device(ids, dev)
    hidden = torch.empty((T, model.d_model), dtype=torch.float32, device=dev)
    dm.prefix(cp, ids_d, to_device(bt.visual, dev), hidden_out=hidden)
    lp = dm.prompt_logprobs(cp, ids_d, hidden, to_device(pos, dev), flags=flags)
    torch.cuda.synchronize()
    got = lp.cpu().numpy()
    full = oracle.prompt_logprob(hw.as_f32(), model, cp, ids, inputs.to_f32(bt.visual))
    exp = np.array([full[t] if 0 <= t < T else np.nan for t in pos])
    assert np.array_equal(np.isnan(got), np.isnan(exp))
    assert np.isfinite(exp).sum() == len(good) + 7
    err = max_abs(got, exp)
    print(f"[parity] prompt log-probs {model.dtype} V={model.vocab} flags={flags}: rows {len(pos)} "
          f"|d lp| {err:.3g}", flush=True)
    assert err <= (1e-4 if model.dtype == "f32" else 2e-2)
    dm.close()


@pytest.mark.parametrize("model", [configs.TINY, BF16_SMALL, BF16_WIDE, F16_D64])
def test_transposed_row_parallel_weights(model):
    """Case-2 storage: wo and w_down stored [in, out] and read in transpose mode.  The MFMAs
    see the same k order, so prefix, suffix (split-K at d = 2048) and decode step are
    bitwise those of the nn.Linear layout; the suffix also matches the oracle."""
    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    P, Vis, S = [70, 300, 129], [60, 256, 100], [9, 65, 130]
    w = configs.custom(model, P, Vis, S, index=85)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    # 40 decode rows: the skinny GEMM's two-row-block form (33..64 rows) in both layouts
    cap, lens = 400, [0, 131, 399] + [(37 * i + 5) % 400 for i in range(37)]
    dec = inputs.make_decode(w, batch=len(lens), kv_len=np.array(lens, np.int32), cap=cap)
    cp, cs = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    outs = []
    for layout in (0, rb.RP_WO_TRANSPOSED, rb.RP_WO_TRANSPOSED | rb.RP_W_DOWN_TRANSPOSED):
        dm = DeviceModel(hw, cap + 1, weight_layout=layout)
        dev = dm.device
        K, V, h = dm.prefix(cp, to_device(bt.token_ids, dev), to_device(bt.visual, dev))
        lp = dm.suffix(cp, cs, K, V, h, to_device(bt.response_ids, dev))
        ck, cv = to_device(dec.cache_k, dev), to_device(dec.cache_v, dev)
        logits = torch.empty((len(lens), model.vocab), dtype=torch.float32, device=dev)
        nxt = dm.decode(ck, cv, to_device(dec.kv_len, dev), to_device(dec.token_ids, dev), logits=logits)
        torch.cuda.synchronize()
        outs.append([t.cpu() for t in (K, V, h, lp, logits, nxt, ck)])
        dm.close()
    names = ("K", "V", "h_last", "logprobs", "decode logits", "next ids", "cache")
    for o in outs[1:]:
        for n, a, b in zip(names, outs[0], o):
            assert torch.equal(a, b), n
    lpo = oracle.suffix_logprob(hw.as_f32(), model, cp, cs,
                                *oracle.prefix_forward(hw.as_f32(), model, cp, bt.token_ids,
                                                       inputs.to_f32(bt.visual))[:3], bt.response_ids)
    err = max_abs(outs[-1][3].numpy(), lpo)
    print(f"[parity] transposed wo/w_down {model.dtype} d={model.d_model}: bitwise equal, |d lp| {err:.3g}",
          flush=True)
    chk = TargetCheck(model.dtype)
    chk.check(f"transposed wo/w_down {model.dtype} d={model.d_model}", outs[-1][3].numpy(), lpo,
              lambda: emulated_suffix(w, hw, bt))
    chk.finish()


@pytest.mark.parametrize("model,mrope", [(configs.TINY, False), (BF16_SMALL, False), (BF16_D64, True),
                                         (F16_SMALL, False), (BF16_WIDE, False),
                                         pytest.param(BF16_D64, False, marks=UNEXPLAINED_FAULT)])
def test_prefix_last_rows_only(model, mrope):
    """RP_PREFIX_LAST_ROWS_ONLY: the last layer past its K/V projection runs only at each
    sequence's last row.  K/V are bitwise those of the full pass, h_last equals the full
    pass's up to summation order, and both meet the oracle bar (so do the suffix log-probs
    scored from them).  P = 1 leaves the last row's query with only its own key."""
    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    from tests.test_oracle_pins import video_positions
    P, Vis, S = [1, 70, 300, 129], [0, 60, 256, 100], [3, 9, 65, 130]
    w = configs.custom(model, P, Vis, S, index=87)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    cp, cs = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    dm = DeviceModel(hw, max(p + s for p, s in zip(P, S)) + 1)
    dev = dm.device
    ids, vis = to_device(bt.token_ids, dev), to_device(bt.visual, dev)
    kw, rope0 = {}, None
    sec = (8, 12, 12) if model.head_dim == 64 else (16, 24, 24)
    if mrope:
        grids = [(1, 1, 1), (3, 4, 5), (4, 8, 8), (4, 5, 5)]
        pos, nxt = zip(*[video_positions(v, p - v, g) if v else (np.zeros((3, p), np.int64), p)
                         for p, v, g in zip(P, Vis, grids)])
        kw = dict(positions=torch.as_tensor(np.concatenate(pos, axis=1).astype(np.int32), device=dev).contiguous(),
                  mrope_section=list(sec))
        rope0 = [int(n) for n in nxt]
    Kf, Vf, hf = dm.prefix(cp, ids, vis, **kw)
    Kt, Vt, ht = dm.prefix(cp, ids, vis, flags=rb.RP_PREFIX_LAST_ROWS_ONLY, **kw)
    lp = dm.suffix_grouped(cp, list(range(len(P))), cs, Kt, Vt, ht, to_device(bt.response_ids, dev),
                           rope_pos0=rope0)
    torch.cuda.synchronize()
    assert torch.equal(Kf, Kt) and torch.equal(Vf, Vt)
    f32 = model.dtype == "f32"
    d_full = rel_err(ht.cpu().numpy(), hf.cpu().numpy())
    W = hw.as_f32()
    vo = np.concatenate([[0], np.cumsum(Vis)])
    visf = inputs.to_f32(bt.visual)
    e_h, e_lp = 0.0, 0.0
    for b in range(len(P)):
        idb = bt.token_ids[cp[b]:cp[b + 1]]
        mr = (pos[b], sec) if mrope else None
        k, v, hl, _ = oracle.prefix_forward_one(W, model, idb, visf[vo[b]:vo[b + 1]], mrope=mr)
        e_h = max(e_h, rel_err(ht[b].cpu().numpy(), hl))
        lpo = oracle.suffix_logprob_one(W, model, k, v, hl, bt.response_ids[cs[b]:cs[b + 1]],
                                        rope_start=None if rope0 is None else rope0[b])
        e_lp = max(e_lp, max_abs(lp[cs[b]:cs[b + 1]].cpu().numpy(), lpo))
    print(f"[parity] last-rows-only prefix {model.dtype} d={model.d_model} mrope={mrope}: h vs full {d_full:.3g}, "
          f"h vs oracle {e_h:.3g}, |d lp| {e_lp:.3g}", flush=True)
    assert d_full <= (1e-5 if f32 else 1e-2)
    assert e_h <= (1e-5 if f32 else 3e-2)
    assert e_lp <= (1e-4 if f32 else 2e-2)
    dm.close()


@pytest.mark.parametrize("model", [configs.TINY, BF16_D64])
def test_maximum_batch_of_256_sequences(model):
    """RP_MAX_SEQS sequences in one call (the kernel-argument sequence table at capacity):
    prefixes of 1..40 tokens, suffixes of 0..8, plus a shared-prefix call whose 256
    responses read 32 of those prefixes."""
    from paper_2608_14498_amd import binding as rb
    from paper_2608_14498_amd.runtime import DeviceModel, to_device
    n = rb.RP_MAX_SEQS
    P = [1 + (b * 7) % 40 for b in range(n)]
    Vis = [p // 2 for p in P]
    S = [b % 9 for b in range(n)]
    w = configs.custom(model, P, Vis, S, index=89)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    got = gpu_run(w, hw, bt)
    ref = oracle_run(w, hw, bt)
    r = _report(f"{n} sequences {model.dtype}", *got, *ref)
    f32 = model.dtype == "f32"
    assert r["lp"] <= (1e-4 if f32 else 2e-2)
    assert r["kv"] <= (1e-5 if f32 else 3e-2) and r["h"] <= (1e-5 if f32 else 3e-2)
    # 256 responses over the first 32 prefixes (8 each), read through the grouped call
    grp = [b // 8 for b in range(n)]
    cp = [int(x) for x in bt.cu_prefix]
    cs = [int(x) for x in bt.cu_suffix]
    dm = DeviceModel(hw, max(P) + max(S) + 1)
    dev = dm.device
    K, V, h = dm.prefix(cp, to_device(bt.token_ids, dev), to_device(bt.visual, dev))
    lp = dm.suffix_grouped(cp, grp, cs, K, V, h, to_device(bt.response_ids, dev)).cpu().numpy()
    dm.close()
    Ko, Vo, Ho = ref[0], ref[1], ref[2]
    lpo = oracle.suffix_logprob_grouped(hw.as_f32(), model, bt.cu_prefix, grp, bt.cu_suffix, Ko, Vo, Ho,
                                        bt.response_ids)
    err = max_abs(lp, lpo)
    print(f"[parity] {n} grouped responses {model.dtype}: |d lp| {err:.3g}", flush=True)
    assert err <= (1e-4 if f32 else 2e-2)
