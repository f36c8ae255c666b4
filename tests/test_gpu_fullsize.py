"""Full-size parity: every benchmark workload at its real shapes, in the launch the
benchmark times (the whole packed batch through rp_prefix_forward, rp_suffix_logprob
and rp_decode_step), checked on sampled outputs against float64 oracle values that
tests/golden/make_fullsize.py stored (one sequence per workload; sequences of a packed
batch are independent).

Each bf16 workload also runs as the same model stored in fp16 (weights converted
exactly from their bf16 values; the oracle values of the bf16 weights stand in for
both, as the conversion moves only weights below 2^-14 and by at most 2^-25).

Bars: |d logprob| <= 2e-2 for both 16-bit types.  On these shapes bf16 cannot meet
it: an exact-arithmetic forward that rounds only what any bf16 matrix-core
implementation must round (tests/bf16_emulation.py) already deviates from the oracle
by 0.05-0.07 on the checked tokens.  A bf16 case above 2e-2 is therefore held to that
stored floor (tests/golden/bf16_floor.json: max within 1.5x, mean within 1.25x) and
reported as an expected failure naming the measured and floor values (TargetCheck).
K/V and h_last relative to their largest reference magnitude <= 3e-2; decode logits at
sampled vocabulary ids within 2e-2 (relative to the row's largest logit magnitude when
that exceeds 1), and the argmax must be the oracle's unless the oracle's top two
logits are closer than that.
"""
from __future__ import annotations

import glob
import json
import os

import numpy as np
import pytest
import torch

from paper_2608_14498_amd import binding as rb
from paper_2608_14498_amd import configs, inputs
from paper_2608_14498_amd.runtime import DeviceModel, to_device
from tests.bf16_emulation import load_floor
from tests.gpu_helpers import LP_TARGET, TargetCheck

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NAMES = [n for n in configs.ORDER if configs.get(n).model.dtype != "f32"]
REL_TOL = 3e-2


def _golden(name, tag=""):
    path = os.path.join(GOLDEN, f"fullsize_{name}{'_' + tag if tag else ''}.npz")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle values for {name} (run tests/golden/make_fullsize.py {name})")
    g = np.load(path, allow_pickle=False)
    return {k: g[k] for k in g.files}


def _goldens(name):
    """(case tag, stored values) of every stored sequence of a workload: the default one
    and the tagged extra ones (the ragged batch's longest prefix and longest suffix)."""
    out = [("", _golden(name))]
    for path in sorted(glob.glob(os.path.join(GOLDEN, f"fullsize_{name}_*.npz"))):
        tag = os.path.basename(path)[len(f"fullsize_{name}_"):-4]
        out.append((tag, _golden(name, tag)))
    return out


def _floor(case):
    fl = load_floor(case)
    return None if fl is None else (fl["max"], fl["mean"])


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("name", NAMES)
def test_fullsize_matches_oracle(name, dtype):
    goldens = _goldens(name)
    w = configs.with_model(configs.get(name), dtype=dtype)
    m = w.model
    chk = TargetCheck(dtype)
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
    lp = lpf = None
    if cu_s[-1] > 0:
        rid = to_device(bt.response_ids, dev)
        lp = dm.suffix(cu_p, cu_s, K, V, h, rid)
        # the same scoring with the fused lm_head + online log-sum-exp (no stored logits)
        ident = list(range(len(cu_p) - 1))
        lpf = dm.suffix_grouped(cu_p, ident, cu_s, K, V, h, rid, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
        torch.cuda.synchronize()
    checks = []
    for tag, g in goldens:
        b = int(g["seq"])
        rows = cu_p[b] + g["kv_pos"]
        k = K[:, torch.as_tensor(rows, device=dev)].float().cpu().numpy()
        v = V[:, torch.as_tensor(rows, device=dev)].float().cpu().numpy()
        res = dict(seq=b, k=_rel(k, g["k"]), v=_rel(v, g["v"]), h_last=_rel(h[b].cpu().numpy(), g["h_last"]))
        if lp is not None:
            got = lp[cu_s[b]:cu_s[b + 1]].cpu().numpy()
            gotf = lpf[cu_s[b]:cu_s[b + 1]].cpu().numpy()
            res["logprob"] = float(np.max(np.abs(got - g["logprobs"])))
            res["logprob_mean"] = float(np.mean(np.abs(got - g["logprobs"])))
            res["logprob_fused"] = float(np.max(np.abs(gotf - g["logprobs"])))
            res["fused_vs_plain"] = float((lpf - lp).abs().max().item())
            case = f"fullsize:{name}" + (f":{tag}" if tag else "")
            checks.append((case, got, gotf, g["logprobs"]))
        print(f"[fullsize] {name} {dtype} {tag or 'seq'} {b}: {json.dumps(res)}", flush=True)
        assert res["k"] <= REL_TOL and res["v"] <= REL_TOL and res["h_last"] <= REL_TOL
        if lp is not None:
            # the fused epilogue reduces the same fp32 logits in another order
            assert res["fused_vs_plain"] <= 1e-4
    del K, V
    g = goldens[0][1]
    res = {}
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
        res["decode_argmax_ok"] = bool(np.all((am == g["dec_argmax"]) | (gap < LP_TARGET)))
        del ck, cv
        print(f"[fullsize] {name} {dtype} decode: {json.dumps(res)}", flush=True)
        assert res["decode_logits"] <= LP_TARGET and res["decode_argmax_ok"]
    dm.close()
    for case, got, gotf, want in checks:
        fl = _floor(case) if dtype == "bf16" else None
        chk.check(f"{case} {dtype}", got, want, floor=fl)
        chk.check(f"{case} {dtype} fused scoring", gotf, want, floor=fl)
    chk.finish()


GROUPED_NAME = "qwen7b_grpo_g4_p4096_n8_s256"


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_fullsize_grouped_responses_match_oracle(dtype):
    """GRPO groups at full size: 4 prompts of 4096 tokens run once, then 32 responses of
    256 tokens (8 per prompt) are scored in one grouped suffix launch over the shared
    prefix KV, stored logits and fused scoring both, as the benchmark runs them."""
    name = GROUPED_NAME
    g = _golden(name)
    w = configs.with_model(configs.get(name), dtype=dtype)
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
    sel = {}
    for tag, out in (("logprob", lp), ("logprob_fused", lpf)):
        sel[tag] = np.stack([out[cu_s[r]:cu_s[r + 1]].cpu().numpy() for r in g["resp_idx"]])
        res[tag] = float(np.max(np.abs(sel[tag] - g["logprobs"])))
    res["fused_vs_plain"] = float((lpf - lp).abs().max().item())
    del K, V
    dm.close()
    print(f"[fullsize] {name} {dtype}: {json.dumps(res)}", flush=True)
    assert res["k"] <= REL_TOL and res["v"] <= REL_TOL and res["h_last"] <= REL_TOL
    assert res["fused_vs_plain"] <= 1e-4
    chk = TargetCheck(dtype)
    fl = _floor(f"grouped:{name}") if dtype == "bf16" else None
    chk.check(f"grouped:{name} {dtype}", sel["logprob"], g["logprobs"], floor=fl)
    chk.check(f"grouped:{name} {dtype} fused scoring", sel["logprob_fused"], g["logprobs"], floor=fl)
    chk.finish()


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
    assert res["fused_vs_plain"] <= 1e-4
    chk = TargetCheck(dtype)
    fl = _floor(f"prompt:{name}") if dtype == "bf16" else None
    chk.check(f"prompt:{name} {dtype}", got[idx], g["prompt_logprobs"], floor=fl)
    chk.check(f"prompt:{name} {dtype} fused scoring", gotf[idx], g["prompt_logprobs"], floor=fl)
    chk.finish()
