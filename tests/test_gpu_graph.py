"""One decode step captured in a HIP graph and replayed.

rp_decode_step_static allocates nothing and issues only kernel launches on the caller's
stream (no memset, copy or host synchronisation outside RP_DEBUG), so a caller can capture
it.  The test captures one step, replays the graph three times with eager work between
the replays (a prefix pass and a torch reduction on the same device), restores the KV
cache before each replay (the step writes slot kv_len), and checks logits, next ids and
the written cache of every replay bitwise against the eager call.  Both the stored-logits
path and the fused lm_head + argmax path (no logits buffer) are captured.
"""
import numpy as np
import pytest
import torch

from paper_2608_14498_amd import binding as rb
from paper_2608_14498_amd import configs, inputs
from paper_2608_14498_amd.runtime import DeviceModel, to_device

pytestmark = pytest.mark.gpu

SMALL = configs.ModelShape(n_layers=2, d_model=384, n_q_heads=6, n_kv_heads=2, head_dim=128,
                           ffn_dim=768, vocab=1000, dtype="bf16")


@pytest.mark.parametrize("with_logits", [True, False])
def test_decode_step_graph_replays_equal_eager(with_logits):
    w = configs.custom(SMALL, [70, 33], [40, 0], [5, 9], index=121)
    hw = inputs.make_weights(w, norm="random", bias=True)
    bt = inputs.make_batch(w)
    B, cap = 6, 1100
    dec = inputs.make_decode(w, batch=B, kv_len=np.array([5, 1099, 700, 0, 1024, 333], np.int32), cap=cap)
    dm = DeviceModel(hw, cap + 1)
    try:
        dev = dm.device
        ck0, cv0 = to_device(dec.cache_k, dev), to_device(dec.cache_v, dev)
        ck, cv = ck0.clone(), cv0.clone()
        kv_len, tok = to_device(dec.kv_len, dev), to_device(dec.token_ids, dev)
        logits = torch.full((B, SMALL.vocab), float("nan"), device=dev) if with_logits else None
        nxt = torch.full((B,), -1, dtype=torch.int32, device=dev)
        kv = rb.make_kv(ck, cv, ck[0].numel())

        def step(stream):
            rb.rp_decode_step_static(dm.handle, stream, B, kv, cap, kv_len, tok, logits, nxt)

        # eager reference (also initialises the library's static scratch for this device)
        step(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ref_nxt = nxt.clone()
        ref_logits = logits.clone() if with_logits else None
        ref_k, ref_v = ck.clone(), cv.clone()

        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                step(side.cuda_stream)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()

        cp = [int(x) for x in bt.cu_prefix]
        ids, vis = to_device(bt.token_ids, dev), to_device(bt.visual, dev)
        for rep in range(3):
            # eager work between replays, then restore the state the step starts from
            dm.prefix(cp, ids, vis)
            _ = torch.randn(4096, device=dev).sum().item()
            ck.copy_(ck0)
            cv.copy_(cv0)
            nxt.fill_(-1)
            if with_logits:
                logits.fill_(float("nan"))
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            print(f"[graph] replay {rep} with_logits={with_logits}", flush=True)
            assert torch.equal(nxt, ref_nxt), f"replay {rep}: next ids"
            if with_logits:
                assert torch.equal(logits, ref_logits), f"replay {rep}: logits"
            assert torch.equal(ck.view(torch.int16), ref_k.view(torch.int16)), f"replay {rep}: K cache"
            assert torch.equal(cv.view(torch.int16), ref_v.view(torch.int16)), f"replay {rep}: V cache"
        del graph
    finally:
        dm.close()
