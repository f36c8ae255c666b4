"""Full-size parity: every benchmark workload at its real shapes, in the launch the
benchmark times (the whole packed batch through rp_prefix_forward, rp_suffix_logprob
and rp_decode_step), checked on sampled outputs against float64 oracle values that
tests/golden/make_fullsize.py stored (one sequence per workload; sequences of a packed
batch are independent).

Each bf16 workload also runs as the same model stored in fp16 (weights converted
exactly from their bf16 values; the oracle values of the bf16 weights stand in for
both, as the conversion moves only weights below 2^-14 and by at most 2^-25).

Bars: fp16: |d logprob| <= 2e-2.  bf16: the storage rounding of activations and K/V
alone (an exact-arithmetic forward that rounds the same intermediates to bf16)
deviates from the oracle by up to ~0.05 on these shapes, so full-size bf16 runs are
held to 0.1, twice that floor; the small-size bf16 tests keep 2e-2.  K/V and h_last
relative to their largest reference magnitude <= 3e-2; decode logits at sampled
vocabulary ids within the log-prob bar (relative to the row's largest logit
magnitude when that exceeds 1), and the argmax must be the oracle's unless the
oracle's top two logits are closer than the bar.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

from paper_2608_14498_amd import binding as rb
from paper_2608_14498_amd import configs, inputs
from paper_2608_14498_amd.runtime import DeviceModel, to_device

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NAMES = [n for n in configs.ORDER if configs.get(n).model.dtype != "f32"]
LP_TOL = {"f16": 2e-2, "bf16": 1e-1}
REL_TOL = 3e-2


def _golden(name):
    path = os.path.join(GOLDEN, f"fullsize_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle values for {name} (run tests/golden/make_fullsize.py {name})")
    g = np.load(path, allow_pickle=False)
    return {k: g[k] for k in g.files}


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("name", NAMES)
def test_fullsize_matches_oracle(name, dtype):
    g = _golden(name)
    w = configs.with_model(configs.get(name), dtype=dtype)
    m = w.model
    tol = LP_TOL[dtype]
    print(f"[fullsize] {name} {dtype}: generating inputs", flush=True)
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    maxp = max(p + s for p, s in zip(bt.prefix_lens, bt.suffix_lens)) + 1
    if w.decode is not None:
        maxp = max(maxp, int(w.decode["cap"]) + 1)
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    cu_p, cu_s = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    print(f"[fullsize] {name}: prefix T={cu_p[-1]} suffix R={cu_s[-1]}", flush=True)
    K, V, h = dm.prefix(cu_p, to_device(bt.token_ids, dev), to_device(bt.visual, dev) if bt.visual.shape[0] else None)
    b = int(g["seq"])
    rows = cu_p[b] + g["kv_pos"]
    k = K[:, torch.as_tensor(rows, device=dev)].float().cpu().numpy()
    v = V[:, torch.as_tensor(rows, device=dev)].float().cpu().numpy()
    hl = h[b].cpu().numpy()
    res = dict(k=_rel(k, g["k"]), v=_rel(v, g["v"]), h_last=_rel(hl, g["h_last"]))
    if cu_s[-1] > 0:
        rid = to_device(bt.response_ids, dev)
        lp = dm.suffix(cu_p, cu_s, K, V, h, rid)
        # the same scoring with the fused lm_head + online log-sum-exp (no stored logits)
        ident = list(range(len(cu_p) - 1))
        lpf = dm.suffix_grouped(cu_p, ident, cu_s, K, V, h, rid, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
        torch.cuda.synchronize()
        got = lp[cu_s[b]:cu_s[b + 1]].cpu().numpy()
        res["logprob"] = float(np.max(np.abs(got - g["logprobs"])))
        res["logprob_fused"] = float(np.max(np.abs(lpf[cu_s[b]:cu_s[b + 1]].cpu().numpy() - g["logprobs"])))
        res["fused_vs_plain"] = float((lpf - lp).abs().max().item())
    del K, V
    if "dec_rows" in g:
        dec = inputs.make_decode(w)
        ck, cv = to_device(dec.cache_k, dev), to_device(dec.cache_v, dev)
        logits = torch.empty((len(dec.token_ids), m.vocab), dtype=torch.float32, device=dev)
        nxt = dm.decode(ck, cv, to_device(dec.kv_len, dev), to_device(dec.token_ids, dev), logits=logits)
        torch.cuda.synchronize()
        lg = logits[torch.as_tensor(g["dec_rows"], device=dev)][:, torch.as_tensor(g["dec_vocab"], device=dev)].cpu().numpy()
        scale = np.maximum(np.max(np.abs(g["dec_logits"]), axis=1, keepdims=True), 1.0)
        res["decode_logits"] = float(np.max(np.abs(lg - g["dec_logits"]) / scale))
        am = nxt.cpu().numpy()[g["dec_rows"]]
        gap = g["dec_top2"][:, 1] - g["dec_top2"][:, 0]
        res["decode_argmax_ok"] = bool(np.all((am == g["dec_argmax"]) | (gap < tol)))
        del ck, cv
    dm.close()
    print(f"[fullsize] {name} {dtype}: {json.dumps(res)}", flush=True)
    assert res["k"] <= REL_TOL and res["v"] <= REL_TOL and res["h_last"] <= REL_TOL
    if "logprob" in res:
        assert res["logprob"] <= tol and res["logprob_fused"] <= tol
        # the fused epilogue reduces the same fp32 logits in another order
        assert res["fused_vs_plain"] <= 1e-4
    if "decode_logits" in res:
        assert res["decode_logits"] <= tol and res["decode_argmax_ok"]


GROUPED_NAME = "qwen7b_grpo_g4_p4096_n8_s256"


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_fullsize_grouped_responses_match_oracle(dtype):
    """GRPO groups at full size: 4 prompts of 4096 tokens run once, then 32 responses of
    256 tokens (8 per prompt) are scored in one grouped suffix launch over the shared
    prefix KV, stored logits and fused scoring both, as the benchmark runs them."""
    name = GROUPED_NAME
    g = _golden(name)
    w = configs.with_model(configs.get(name), dtype=dtype)
    tol = LP_TOL[dtype]
    print(f"[fullsize] {name} {dtype}: generating inputs", flush=True)
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    maxp = max(bt.prefix_lens) + max(bt.suffix_lens) + 1
    dm = DeviceModel(hw, maxp)
    dev = dm.device
    cu_p, cu_s = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
    grp = [int(x) for x in bt.prefix_of_suffix]
    print(f"[fullsize] {name}: prefix T={cu_p[-1]} suffix R={cu_s[-1]} ({len(grp)} responses)", flush=True)
    K, V, h = dm.prefix(cu_p, to_device(bt.token_ids, dev), to_device(bt.visual, dev))
    b = int(g["seq"])
    rows = cu_p[b] + g["kv_pos"]
    k = K[:, torch.as_tensor(rows, device=dev)].float().cpu().numpy()
    v = V[:, torch.as_tensor(rows, device=dev)].float().cpu().numpy()
    res = dict(k=_rel(k, g["k"]), v=_rel(v, g["v"]), h_last=_rel(h[b].cpu().numpy(), g["h_last"]))
    rid = to_device(bt.response_ids, dev)
    lp = dm.suffix_grouped(cu_p, grp, cu_s, K, V, h, rid)
    lpf = dm.suffix_grouped(cu_p, grp, cu_s, K, V, h, rid, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
    torch.cuda.synchronize()
    for tag, out in (("logprob", lp), ("logprob_fused", lpf)):
        res[tag] = max(float(np.max(np.abs(out[cu_s[r]:cu_s[r + 1]].cpu().numpy() - g["logprobs"][i])))
                       for i, r in enumerate(g["resp_idx"]))
    res["fused_vs_plain"] = float((lpf - lp).abs().max().item())
    del K, V
    dm.close()
    print(f"[fullsize] {name} {dtype}: {json.dumps(res)}", flush=True)
    assert res["k"] <= REL_TOL and res["v"] <= REL_TOL and res["h_last"] <= REL_TOL
    assert res["logprob"] <= tol and res["logprob_fused"] <= tol
    assert res["fused_vs_plain"] <= 1e-4


PROMPT_NAMES = ["qwen7b_b4_p4096_s256", "qwen7b_ragged_b8"]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("name", PROMPT_NAMES)
def test_fullsize_prompt_logprobs_match_oracle(name, dtype):
    """Prompt-token log-probs of every text token of the packed batch (the launch the
    benchmark times), plain and fused scoring, checked at the stored sampled positions."""
    from paper_2608_14498_amd.runtime import prompt_positions

    path = os.path.join(GOLDEN, f"fullsize_prompt_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle values (run tests/golden/make_fullsize.py --prompt {name})")
    g = np.load(path, allow_pickle=False)
    w = configs.with_model(configs.get(name), dtype=dtype)
    m = w.model
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    dm = DeviceModel(hw, max(bt.prefix_lens) + 1)
    dev = dm.device
    cu_p = [int(x) for x in bt.cu_prefix]
    ids = to_device(bt.token_ids, dev)
    hidden = torch.empty((cu_p[-1], m.d_model), dtype=torch.float32, device=dev)
    dm.prefix(cu_p, ids, to_device(bt.visual, dev), hidden_out=hidden)
    pos = prompt_positions(cu_p, bt.token_ids)
    print(f"[fullsize] {name} {dtype}: prompt rows {len(pos)}", flush=True)
    pos_d = to_device(pos, dev)
    lp = dm.prompt_logprobs(cu_p, ids, hidden, pos_d)
    lpf = dm.prompt_logprobs(cu_p, ids, hidden, pos_d, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
    torch.cuda.synchronize()
    want = cu_p[int(g["seq"])] + g["prompt_pos"]
    idx = np.searchsorted(pos, want)
    assert np.array_equal(pos[idx], want)
    got, gotf = lp.cpu().numpy(), lpf.cpu().numpy()
    res = dict(prompt=float(np.max(np.abs(got[idx] - g["prompt_logprobs"]))),
               prompt_fused=float(np.max(np.abs(gotf[idx] - g["prompt_logprobs"]))),
               fused_vs_plain=float(np.max(np.abs(gotf - got))), finite=bool(np.all(np.isfinite(got))))
    dm.close()
    print(f"[fullsize] {name} {dtype}: {json.dumps(res)}", flush=True)
    assert res["finite"]
    assert res["prompt"] <= LP_TOL[dtype] and res["prompt_fused"] <= LP_TOL[dtype]
    assert res["fused_vs_plain"] <= 1e-4
