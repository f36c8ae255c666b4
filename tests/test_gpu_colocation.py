"""Co-location correctness (Eq. (1) and Section "Resource Sharing Policy"): the prefix pass
on one stream while rollout decode steps run on another stream of the same GPU, either on
two unmasked streams (the analog of the paper's MPS-Default sharing) or on streams with
complementary CU masks (the analog of its static SM partitions).

Sharing the GPU changes when work runs, not what it computes: every kernel reads only its
own call's inputs and workspace, so the prefix K/V and boundary state and every decode
step's logits, next ids and cache writes must be bitwise those of running the two
serially.  The decode side is a greedy chain: step i writes cache slot kv_len0 + i and
feeds on the id that step i-1 chose.  The serial run's first decode step and its prefix
are also checked against the oracle.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from paper_2608_14498_amd import binding as rb
from paper_2608_14498_amd import configs, inputs
from paper_2608_14498_amd.runtime import DeviceModel, to_device
from tests.gpu_helpers import TargetCheck, max_abs, rel_err
from tests.test_gpu_parity import BF16_SMALL, BF16_WIDE

pytestmark = pytest.mark.gpu


def cu_mask(lo: int, hi: int, ncu: int):
    words = [0] * ((ncu + 31) // 32)
    for i in range(lo, hi):
        words[i // 32] |= 1 << (i % 32)
    return words


class Colo:
    """One prefix batch and one decode batch of a model, with per-run output buffers."""

    def __init__(self, w, hw, bt, dec, steps, to_host=True):
        self.w, self.hw, self.bt, self.dec = w, hw, bt, dec
        self.steps = steps
        self.to_host = to_host
        self.dm = DeviceModel(self.hw, max(max(bt.prefix_lens), dec.cap) + 1)
        dev = self.dm.device
        self.cu = [int(x) for x in self.bt.cu_prefix]
        self.ids = to_device(self.bt.token_ids, dev)
        self.vis = to_device(self.bt.visual, dev) if self.bt.visual.shape[0] else None
        self.ck0, self.cv0 = to_device(self.dec.cache_k, dev), to_device(self.dec.cache_v, dev)
        self.lens = [to_device(self.dec.kv_len + i, dev) for i in range(steps)]
        self.tok0 = to_device(self.dec.token_ids, dev)

    def run(self, s_prefix, s_decode):
        """Enqueue the prefix on s_prefix and the decode chain on s_decode (no ordering
        between them); returns every output after the device is idle."""
        dm, m = self.dm, self.w.model
        dev = dm.device
        B, T, Bd = len(self.cu) - 1, self.cu[-1], self.dec.token_ids.shape[0]
        K, V = dm.alloc_kv(T)
        K.fill_(float("nan"))
        V.fill_(float("nan"))
        h = torch.full((B, m.d_model), float("nan"), dtype=torch.float32, device=dev)
        ws_p = dm.workspace(rb.rp_prefix_workspace_bytes(dm.handle, B, self.cu))
        ws_d = dm.workspace(rb.rp_decode_workspace_bytes(dm.handle, Bd, self.dec.cap))
        ck, cv = self.ck0.clone(), self.cv0.clone()
        ids = [self.tok0] + [torch.full((Bd,), -7, dtype=torch.int32, device=dev) for _ in range(self.steps)]
        logits = [torch.full((Bd, m.vocab), float("nan"), dtype=torch.float32, device=dev) for _ in range(self.steps)]
        torch.cuda.synchronize()
        dm.prefix(self.cu, self.ids, self.vis, kv=(K, V), h_last=h, workspace=ws_p, stream=s_prefix)
        for i in range(self.steps):
            dm.decode(ck, cv, self.lens[i], ids[i], logits=logits[i], next_ids=ids[i + 1], workspace=ws_d,
                      stream=s_decode)
        torch.cuda.synchronize()
        out = dict(K=K, V=V, h_last=h, cache_k=ck, cache_v=cv, next_ids=torch.stack(ids[1:]),
                   logits=torch.stack(logits))
        del ws_p, ws_d
        return {k: v.cpu() for k, v in out.items()} if self.to_host else out

    def close(self):
        self.dm.close()


def same_bits(a: torch.Tensor, b: torch.Tensor) -> bool:
    return a.shape == b.shape and a.dtype == b.dtype and torch.equal(
        a.contiguous().flatten().view(torch.uint8), b.contiguous().flatten().view(torch.uint8))


def check_against_oracle(c: Colo, out):
    """The serial run's prefix and first decode step against the float64 oracle."""
    m = c.w.model
    W = c.hw.as_f32()
    f32 = m.dtype == "f32"
    vis = inputs.to_f32(c.bt.visual)
    Ko, Vo, Ho = oracle.prefix_forward(W, m, c.bt.cu_prefix, c.bt.token_ids, vis)
    assert max(rel_err(out["K"].float().numpy(), Ko), rel_err(out["V"].float().numpy(), Vo)) <= (1e-5 if f32 else 3e-2)
    assert rel_err(out["h_last"].numpy(), Ho) <= (1e-5 if f32 else 3e-2)
    lo, _, _, _ = oracle.decode_step(W, m, inputs.to_f32(c.dec.cache_k), inputs.to_f32(c.dec.cache_v),
                                     c.dec.kv_len, c.dec.token_ids)
    got = out["logits"][0].numpy()
    print(f"[colo] serial decode step 0 vs oracle: logits max|d| {max_abs(got, lo):.3g}", flush=True)

    def emulate():
        from tests import bf16_emulation as em
        return em.decode_logits(W, m, inputs.to_f32(c.dec.cache_k), inputs.to_f32(c.dec.cache_v), c.dec.kv_len,
                                c.dec.token_ids, em.Rounder(m.dtype, em.POINTS))

    chk = TargetCheck(m.dtype)
    chk.check(f"decode logits {m.dtype} d={m.d_model}", got, lo, emulate)
    return chk


def run_arms(c: Colo, ref, decode_cus, tag: str):
    """The co-run arms: two unmasked streams, then decode on the first k CUs and the
    prefix on the rest for every k in decode_cus; each must equal the serial run bit for
    bit."""
    ncu = rb.rp_device_cu_count(0)
    assert ncu > 0
    arms = [("unmasked streams", None)] + [(f"decode {k} CUs / prefix {ncu - k} CUs", k) for k in decode_cus]
    for name, k in arms:
            raw = None
            if k is None:
                sp, sd = torch.cuda.Stream(), torch.cuda.Stream()
            else:
                raw = (rb.rp_stream_create_cu_masked(0, cu_mask(k, ncu, ncu)), rb.rp_stream_create_cu_masked(0, cu_mask(0, k, ncu)))
                sp, sd = torch.cuda.ExternalStream(raw[0]), torch.cuda.ExternalStream(raw[1])
            try:
                got = c.run(sp, sd)
            finally:
                if raw:
                    rb.rp_stream_destroy(raw[0])
                    rb.rp_stream_destroy(raw[1])
            for key in ref:
                assert same_bits(got[key], ref[key]), f"{name}: {key}"
            del got
            print(f"[colo] {tag} {name}: bitwise equal to serial", flush=True)


@pytest.mark.parametrize("model", [BF16_SMALL, configs.TINY, BF16_WIDE])
def test_colocated_prefix_and_decode_equal_serial(model):
    P, Vis, S = [300, 129, 70, 1], [256, 100, 60, 0], [0, 0, 0, 0]
    w = configs.custom(model, P, Vis, S, index=97)
    hw = inputs.make_weights(w, norm="random", bias=True)
    dec = inputs.make_decode(w, batch=5, kv_len=np.full(5, 200, np.int32), cap=300)
    c = Colo(w, hw, inputs.make_batch(w), dec, steps=12)
    try:
        main = torch.cuda.current_stream()
        ref = c.run(main, main)
        chk = check_against_oracle(c, ref)
        run_arms(c, ref, (32, 128), f"{model.dtype} d={model.d_model}")
    finally:
        c.close()
    chk.finish()


COLO_NAME = "qwen7b_coloc_p4x8192_d64"


def test_fullsize_colocation_equal_serial_and_oracle():
    """The co-location workload at full size (prefix 4 x 8192 of the 7B slice beside 8 greedy
    decode steps of 64 sequences over an 8192-token KV), launched as the benchmark launches
    it: every co-run arm is bitwise the serial run, and the serial run matches the stored
    oracle values (sampled prefix K/V rows and h_last of sequence 0; the first decode step's
    logits at sampled vocabulary ids and argmax of two batch rows)."""
    import os

    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", f"fullsize_{COLO_NAME}.npz")
    g = np.load(path, allow_pickle=False)
    w = configs.get(COLO_NAME)
    print(f"[colo] {COLO_NAME}: generating inputs", flush=True)
    c = Colo(w, inputs.make_weights(w), inputs.make_batch(w), inputs.make_decode(w), steps=8, to_host=False)
    try:
        main = torch.cuda.current_stream()
        ref = c.run(main, main)
        b, cu = int(g["seq"]), c.cu
        rows = torch.as_tensor(cu[b] + g["kv_pos"], device=c.dm.device)
        res = dict(k=rel_err(ref["K"][:, rows].float().cpu().numpy(), g["k"]),
                   v=rel_err(ref["V"][:, rows].float().cpu().numpy(), g["v"]),
                   h_last=rel_err(ref["h_last"][b].cpu().numpy(), g["h_last"]))
        lg = ref["logits"][0][torch.as_tensor(g["dec_rows"], device=c.dm.device)].cpu().numpy()[:, g["dec_vocab"]]
        scale = np.maximum(np.max(np.abs(g["dec_logits"]), axis=1, keepdims=True), 1.0)
        res["decode_logits"] = float(np.max(np.abs(lg - g["dec_logits"]) / scale))
        am = ref["next_ids"][0].cpu().numpy()[g["dec_rows"]]
        gap = g["dec_top2"][:, 1] - g["dec_top2"][:, 0]
        res["decode_argmax_ok"] = bool(np.all((am == g["dec_argmax"]) | (gap < 2e-2)))
        print(f"[colo] {COLO_NAME} serial vs oracle: {res}", flush=True)
        assert res["k"] <= 3e-2 and res["v"] <= 3e-2 and res["h_last"] <= 3e-2
        assert res["decode_logits"] <= 2e-2 and res["decode_argmax_ok"]
        run_arms(c, ref, (96,), COLO_NAME)
    finally:
        c.close()
