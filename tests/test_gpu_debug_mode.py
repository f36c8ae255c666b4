"""RP_DEBUG (guard bytes after every workspace slice, range checks of device-side ids)
on the GPU.  The mode is read once per process, so each case runs in a child process:

  * with valid inputs every compute call (prefix, suffix, grouped suffix with fused
    scoring, prompt log-probs, decode step) passes its checks and returns exactly the
    results of the same calls without the mode;
  * an out-of-range token id, response id or kv_len is reported by the call
    (RP_ERR_INVALID_ARG / RP_ERR_SHAPE naming the array, index and value);
  * a host-forced write into a guard (RP_DEBUG_CORRUPT_GUARD) is reported (RP_ERR_HIP).

The kernels clamp ids and lengths, so none of these inputs makes a kernel read or write
outside its buffers; the guard write lands inside the caller's workspace.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r'''
import sys, numpy as np, torch
sys.path.insert(0, %(root)r)
from paper_2608_14498_amd import binding as rb, configs, inputs
from paper_2608_14498_amd.runtime import DeviceModel, prompt_positions, to_device
model = configs.ModelShape(n_layers=2, d_model=384, n_q_heads=6, n_kv_heads=2, head_dim=128, ffn_dim=768,
                           vocab=1000, dtype="bf16")
w = configs.custom(model, [70, 129, 33], [40, 100, 0], [9, 0, 65], index=131)
hw = inputs.make_weights(w, norm="random", bias=True)
bt = inputs.make_batch(w)
dm = DeviceModel(hw, 400)
dev = dm.device
cp, cs = [int(x) for x in bt.cu_prefix], [int(x) for x in bt.cu_suffix]
ids, vis, rid = to_device(bt.token_ids, dev), to_device(bt.visual, dev), to_device(bt.response_ids, dev)
case = sys.argv[1]
try:
    if case == "bad_token":
        bad = bt.token_ids.copy(); bad[75] = model.vocab + 5
        dm.prefix(cp, to_device(bad, dev), vis)
    elif case == "bad_response":
        K, V, h = dm.prefix(cp, ids, vis)
        bad = bt.response_ids.copy(); bad[3] = -2
        dm.suffix(cp, cs, K, V, h, to_device(bad, dev))
    elif case == "bad_kv_len":
        dec = inputs.make_decode(w, batch=3, kv_len=np.array([5, 300, 17], np.int32), cap=300)
        dm.decode(to_device(dec.cache_k, dev), to_device(dec.cache_v, dev), to_device(dec.kv_len, dev),
                  to_device(dec.token_ids, dev))
    else:  # "valid" (also the guard self-test when RP_DEBUG_CORRUPT_GUARD is set)
        K, V, h = dm.prefix(cp, ids, vis)
        lp = dm.suffix(cp, cs, K, V, h, rid)
        lpf = dm.suffix_grouped(cp, [0, 1, 2], cs, K, V, h, rid, flags=rb.RP_SUFFIX_FUSED_LOGPROB)
        hidden = torch.empty((cp[-1], model.d_model), dtype=torch.float32, device=dev)
        dm.prefix(cp, ids, vis, hidden_out=hidden)
        pos = to_device(prompt_positions(cp, bt.token_ids), dev)
        plp = dm.prompt_logprobs(cp, ids, hidden, pos)
        dec = inputs.make_decode(w, batch=3, kv_len=np.array([5, 299, 17], np.int32), cap=300)
        ck, cv = to_device(dec.cache_k, dev), to_device(dec.cache_v, dev)
        logits = torch.empty((3, model.vocab), dtype=torch.float32, device=dev)
        nxt = dm.decode(ck, cv, to_device(dec.kv_len, dev), to_device(dec.token_ids, dev), logits=logits)
        torch.cuda.synchronize()
        np.savez(sys.argv[2], K=K.view(torch.int16).cpu().numpy(), h=h.cpu().numpy(), lp=lp.cpu().numpy(),
                 lpf=lpf.cpu().numpy(), plp=plp.cpu().numpy(), logits=logits.cpu().numpy(), nxt=nxt.cpu().numpy(),
                 ck=ck.view(torch.int16).cpu().numpy())
    print("STATUS OK", flush=True)
except rb.RollplexError as e:
    print(f"STATUS {e.status} {e}", flush=True)
'''


def _run(case, tmp_path, debug=True, corrupt=False):
    env = dict(os.environ)
    env.pop("RP_DEBUG", None)
    env.pop("RP_DEBUG_CORRUPT_GUARD", None)
    if debug:
        env["RP_DEBUG"] = "1"
    if corrupt:
        env["RP_DEBUG_CORRUPT_GUARD"] = "1"
    out = str(tmp_path / f"{case}_{int(debug)}.npz")
    r = subprocess.run([sys.executable, "-c", CHILD % {"root": ROOT}, case, out], env=env, capture_output=True,
                       text=True, timeout=300)
    line = [l for l in r.stdout.splitlines() if l.startswith("STATUS")]
    assert r.returncode == 0 and line, r.stdout[-2000:] + r.stderr[-2000:]
    print(f"[debug] {case} debug={debug} corrupt={corrupt}: {line[-1]}", flush=True)
    return line[-1], out


def test_debug_mode_passes_valid_calls_with_identical_results(tmp_path):
    from paper_2608_14498_amd import binding as rb  # noqa: F401  (library present)
    st, with_dbg = _run("valid", tmp_path)
    assert st == "STATUS OK"
    st, without = _run("valid", tmp_path, debug=False)
    assert st == "STATUS OK"
    a, b = np.load(with_dbg), np.load(without)
    for k in a.files:
        assert np.array_equal(a[k], b[k], equal_nan=True), k


@pytest.mark.parametrize("case,status,needle", [("bad_token", 1, "token_ids[75] = 1005"),
                                                ("bad_response", 1, "response_ids[3] = -2"),
                                                ("bad_kv_len", 2, "kv_len[1] = 300")])
def test_debug_mode_reports_out_of_range_ids(tmp_path, case, status, needle):
    st, _ = _run(case, tmp_path)
    assert st.startswith(f"STATUS {status} ") and needle in st, st


def test_debug_mode_reports_an_overwritten_guard(tmp_path):
    st, _ = _run("valid", tmp_path, corrupt=True)
    assert st.startswith("STATUS 5 ") and "guard" in st, st
