"""rp_decode_step_static (no workspace: the library's static scratch) against
rp_decode_step with a caller workspace, through the C ABI: logits, next ids and the
cache writes must be bitwise equal (same kernels, same order), over two calls in a
row, the second with a smaller batch and cache (the shared scratch keeps the first
call's contents).  A static call given no logits buffer takes the argmax inside the
lm_head product (16-bit models, at most 64 rows); its next ids must still equal those
of the workspace call, which stores the logits."""
import numpy as np
import pytest
import torch

from paper_2608_14498_amd import binding as rb
from paper_2608_14498_amd import configs, inputs
from paper_2608_14498_amd.runtime import DeviceModel, to_device

pytestmark = pytest.mark.gpu

SMALL = configs.ModelShape(n_layers=2, d_model=384, n_q_heads=6, n_kv_heads=2, head_dim=128,
                           ffn_dim=768, vocab=1000, dtype="bf16")


def _one_call(dm, w, B, cap, kv0, own_logits):
    m = w.model
    dec = inputs.make_decode(w, batch=B, kv_len=(np.arange(B) * 37 + kv0) % cap, cap=cap)
    dev = dm.device
    outs = []
    for static in (False, True):
        ck, cv = to_device(dec.cache_k, dev), to_device(dec.cache_v, dev)
        kv_len, tok = to_device(dec.kv_len, dev), to_device(dec.token_ids, dev)
        nxt = torch.full((B,), -1, dtype=torch.int32, device=dev)
        logits = None if (static and own_logits) else torch.full((B, m.vocab), float("nan"), device=dev)
        kv = rb.make_kv(ck, cv, ck[0].numel())
        stream = torch.cuda.current_stream().cuda_stream
        if static:
            rb.rp_decode_step_static(dm.handle, stream, B, kv, cap, kv_len, tok, logits, nxt)
        else:
            ws = dm.workspace(rb.rp_decode_workspace_bytes(dm.handle, B, cap))
            rb.rp_decode_step(dm.handle, stream, B, kv, cap, kv_len, tok, logits, nxt, ws, ws.numel())
        torch.cuda.synchronize()
        outs.append((None if logits is None else logits.cpu(), nxt.cpu(), ck.cpu(), cv.cpu()))
    (l0, n0, k0, v0), (l1, n1, k1, v1) = outs
    assert torch.equal(n0, n1), "next ids"
    assert torch.equal(k0.view(torch.int16), k1.view(torch.int16)) if k0.dtype != torch.float32 else torch.equal(k0, k1)
    assert torch.equal(v0.view(torch.int16), v1.view(torch.int16)) if v0.dtype != torch.float32 else torch.equal(v0, v1)
    if l1 is not None:
        assert torch.equal(l0, l1), "logits"
    assert int(n1.min()) >= 0 and int(n1.max()) < m.vocab
    return n1


@pytest.mark.parametrize("model", [SMALL, configs.TINY])
def test_static_decode_equals_workspace_decode_small(model):
    w = configs.custom(model, [1], [0], [1], index=111)
    dm = DeviceModel(inputs.make_weights(w, norm="random", bias=True), 1200)
    try:
        _one_call(dm, w, B=6, cap=1100, kv0=700, own_logits=False)
        _one_call(dm, w, B=3, cap=300, kv0=5, own_logits=True)
    finally:
        dm.close()


def test_static_decode_equals_workspace_decode_7b_slice():
    """The co-location workload's decode shape (64 sequences, cache 8256), then a smaller one."""
    w = configs.get("qwen7b_coloc_p4x8192_d64")
    dm = DeviceModel(inputs.make_weights(w), 8257)
    try:
        print("[no-alloc] 7B slice B=64 cap=8256", flush=True)
        _one_call(dm, w, B=64, cap=8256, kv0=8192, own_logits=False)
        print("[no-alloc] 7B slice B=16 cap=4096", flush=True)
        _one_call(dm, w, B=16, cap=4096, kv0=1000, own_logits=False)
        print("[no-alloc] 7B slice B=64 cap=8256, no logits buffer (fused argmax)", flush=True)
        _one_call(dm, w, B=64, cap=8256, kv0=8192, own_logits=True)
    finally:
        dm.close()
