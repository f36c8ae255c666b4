"""Write the oracle's expected values for the full-size parity tests.

    python tests/golden/make_fullsize.py WORKLOAD [WORKLOAD ...]
    python tests/golden/make_fullsize.py --prompt WORKLOAD [WORKLOAD ...]
    python tests/golden/make_fullsize.py --seq B --tag TAG WORKLOAD

The last form stores sequence B instead of the default one, in
tests/golden/fullsize_<workload>_<tag>.npz (the ragged batch's longest prefix and
longest suffix are stored that way, beside its shortest sequence).

For each named workload this runs the float64 CPU oracle (oracle/, nothing else
computes) on one sequence of the seeded synthetic batch, at the workload's real
shapes, and stores sampled outputs in tests/golden/fullsize_<workload>.npz:

  seq            index of the sequence in the packed batch
  kv_pos         sampled prefix positions (first, second, middle, last + random)
  k, v           [L, len(kv_pos), Hkv, Dh] post-RoPE keys / values at kv_pos
  h_last         [d] residual stream at the last prefix position
  logprobs       [S] log-probabilities of the sequence's response tokens; for a
                 workload of grouped responses, [2, S]: the first and the last
                 response of sequence seq's group
  resp_idx       (grouped responses only) the indices of those two responses
  dec_rows       decode-step batch rows checked (co-location workload only)
  dec_vocab      sampled vocabulary ids of the decode logits
  dec_logits     [len(dec_rows), len(dec_vocab)] oracle logits at dec_vocab
  dec_argmax     [len(dec_rows)] oracle argmax over the whole vocabulary
  dec_top2       [len(dec_rows), 2] the two largest oracle logits of each row

With --prompt it stores prompt-token log-probabilities instead, in
tests/golden/fullsize_prompt_<workload>.npz:

  seq              index of the sequence in the packed batch
  prompt_pos       sampled text positions t >= 1 of that prompt (first and last
                   text token + random)
  prompt_logprobs  log p(token t | tokens < t) at prompt_pos

Sequences are independent in a packed batch (the oracle has no cross-sequence
term), so one sequence's oracle values are the expected values of that sequence
in the full launch.  The inputs come from the seeded generators shared with the
GPU side (paper_2608_14498_amd/inputs.py, which holds no model arithmetic).
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2608_14498_amd import configs, inputs  # noqa: E402

N_KV_SAMPLES = 32
N_VOCAB_SAMPLES = 4096
DEC_ROWS = [0, 37]


def pick_sequence(w, P):
    """Sequence 0, except for ragged batches: the shortest one (keeps the oracle cheap)."""
    return int(np.argmin(P)) if w.ragged is not None else 0


def kv_positions(P: int, seed: int):
    rng = np.random.default_rng([seed, 900])
    fixed = [0, 1, P // 2, P - 1]
    extra = rng.choice(np.arange(2, P - 1), size=min(N_KV_SAMPLES - len(fixed), max(P - 3, 0)), replace=False)
    return np.unique(np.concatenate([fixed, extra])).astype(np.int64)


def make(name: str, seq=None, tag: str = "") -> str:
    t0 = time.time()
    w = configs.get(name)
    m = w.model
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    W = hw.as_f32()
    P, Vis, S = inputs.draw_lengths(w)
    b = pick_sequence(w, P) if seq is None else int(seq)
    cp, cs = bt.cu_prefix, bt.cu_suffix
    vo = int(sum(Vis[:b]))
    ids = bt.token_ids[cp[b]:cp[b + 1]]
    vis = inputs.to_f32(bt.visual[vo:vo + Vis[b]])
    K, V, h_last, _ = oracle.prefix_forward_one(W, m, ids, vis)
    pos = kv_positions(P[b], w.index)
    out = dict(seq=np.int64(b), kv_pos=pos, k=K[:, pos].astype(np.float32), v=V[:, pos].astype(np.float32),
               h_last=h_last.astype(np.float64))
    if w.group:
        # grouped responses: the first and the last response of prompt b's group, both
        # scored over that prompt's one prefix
        ridx = np.asarray([b * w.group, b * w.group + w.group - 1], np.int64)
        lps = [oracle.suffix_logprob_one(W, m, K, V, h_last, bt.response_ids[cs[r]:cs[r + 1]]) for r in ridx]
        out.update(resp_idx=ridx, logprobs=np.stack(lps).astype(np.float64))
    else:
        lp = oracle.suffix_logprob_one(W, m, K, V, h_last, bt.response_ids[cs[b]:cs[b + 1]])
        out.update(logprobs=lp.astype(np.float64))
    del K, V
    if w.decode is not None:
        dec = inputs.make_decode(w)
        rows = np.asarray(DEC_ROWS, np.int64)
        lo, amax, _, _ = oracle.decode_step(W, m, inputs.to_f32(dec.cache_k[:, rows]), inputs.to_f32(dec.cache_v[:, rows]),
                                            dec.kv_len[rows], dec.token_ids[rows])
        vocab = np.random.default_rng([w.index, 901]).choice(m.vocab, N_VOCAB_SAMPLES, replace=False)
        out.update(dec_rows=rows, dec_vocab=vocab.astype(np.int64), dec_logits=lo[:, vocab].astype(np.float64),
                   dec_argmax=np.asarray(amax, np.int64), dec_top2=np.sort(lo, axis=1)[:, -2:].astype(np.float64))
    meta = dict(workload=name, seconds=round(time.time() - t0, 1), prefix=int(P[b]), suffix=int(S[b]))
    path = os.path.join(HERE, f"fullsize_{name}{'_' + tag if tag else ''}.npz")
    np.savez_compressed(path, meta=np.array(json.dumps(meta)), **out)
    return path


def make_prompt(name: str) -> str:
    t0 = time.time()
    w = configs.get(name)
    m = w.model
    hw = inputs.make_weights(w)
    bt = inputs.make_batch(w)
    P, Vis, _ = inputs.draw_lengths(w)
    b = pick_sequence(w, P)
    cp = bt.cu_prefix
    vo = int(sum(Vis[:b]))
    ids = bt.token_ids[cp[b]:cp[b + 1]]
    vis = inputs.to_f32(bt.visual[vo:vo + Vis[b]])
    lp = oracle.prompt_logprob_one(hw.as_f32(), m, ids, vis)
    text = np.nonzero(np.isfinite(lp))[0]
    rng = np.random.default_rng([w.index, 902])
    pick = rng.choice(text[1:-1], size=min(N_KV_SAMPLES - 2, max(len(text) - 2, 0)), replace=False)
    pos = np.unique(np.concatenate([text[:1], text[-1:], pick])).astype(np.int64)
    meta = dict(workload=name, seconds=round(time.time() - t0, 1), prefix=int(P[b]), text=int(len(text)))
    path = os.path.join(HERE, f"fullsize_prompt_{name}.npz")
    np.savez_compressed(path, meta=np.array(json.dumps(meta)), seq=np.int64(b), prompt_pos=pos,
                        prompt_logprobs=lp[pos].astype(np.float64))
    return path


if __name__ == "__main__":
    args = sys.argv[1:]
    fn = make
    if args and args[0] == "--prompt":
        fn, args = make_prompt, args[1:]
    if args and args[0] == "--seq":
        assert args[2] == "--tag" and len(args) == 5, "usage: --seq B --tag TAG WORKLOAD"
        print(make(args[4], seq=int(args[1]), tag=args[3]), flush=True)
        sys.exit(0)
    for n in args:
        print(fn(n), flush=True)
