"""C-ABI checks that need no GPU: the library loads, exports every declared symbol,
and rejects bad arguments (with a message) before making any HIP call."""
import os
import re
import subprocess
import sys

import pytest

from paper_2608_14498_amd import binding as rb
from paper_2608_14498_amd import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rollplex.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rb.LIB_PATH):
        pytest.fail("librollplex.so is not built (python -m paper_2608_14498_amd.build)")
    return rb.lib()


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:rp_status|void|int|int32_t|const char \*)\s*(rp_\w+)\s*\(", text, re.M)))


def test_header_declares_what_binding_wraps():
    assert declared_symbols() == sorted(rb.SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", rb.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (rp_\w+)", out))
    missing = [s for s in declared_symbols() if s not in exported]
    assert not missing, missing
    assert "gfx950" in rb.rp_version()


FAKE = 0x7f0000000000  # never dereferenced: every call below fails validation first


def fake_weights(model, align=256):
    layers = (rb.RpLayerWeights * model.n_layers)()
    addr = FAKE
    for i in range(model.n_layers):
        for name, _ in rb.RpLayerWeights._fields_:
            if name in ("bq", "bk", "bv"):
                continue
            setattr(layers[i], name, addr)
            addr += align * 64
    w = rb.RpWeights(addr, addr + align * 64, addr + align * 128, layers)
    return w, layers


def make(model=configs.TINY, max_pos=1024, **over):
    cfg = rb.make_config(model, max_pos)
    for k, v in over.items():
        setattr(cfg, k, v)
    w, keep = fake_weights(model)
    return rb.rp_create(cfg, w), (w, keep)


def status_of(fn, *args):
    try:
        fn(*args)
    except rb.RollplexError as e:
        return e.status, str(e)
    return rb.RP_OK, ""


@pytest.mark.parametrize("field,value,status", [
    ("dtype", 7, rb.RP_ERR_INVALID_ARG),
    ("head_dim", 96, rb.RP_ERR_UNSUPPORTED),
    ("n_kv_heads", 3, rb.RP_ERR_SHAPE),
    ("n_layers", 0, rb.RP_ERR_SHAPE),
    ("rms_eps", 0.0, rb.RP_ERR_SHAPE),
    ("d_model", 100, rb.RP_ERR_UNSUPPORTED),
    ("weight_layout", 4, rb.RP_ERR_INVALID_ARG),
])
def test_create_rejects_bad_config(lib, field, value, status):
    cfg = rb.make_config(configs.TINY, 1024)
    setattr(cfg, field, value)
    w, _ = fake_weights(configs.TINY)
    st, msg = status_of(rb.rp_create, cfg, w)
    assert st == status and len(msg) > 12


def test_create_rejects_missing_and_misaligned_weights(lib):
    cfg = rb.make_config(configs.QWEN7B_SLICE, 8192)
    w, layers = fake_weights(configs.QWEN7B_SLICE)
    layers[1].w_up = None
    assert status_of(rb.rp_create, cfg, w)[0] == rb.RP_ERR_INVALID_ARG
    w, layers = fake_weights(configs.QWEN7B_SLICE)
    layers[0].wq = FAKE + 2
    st, msg = status_of(rb.rp_create, cfg, w)
    assert st == rb.RP_ERR_INVALID_ARG and "aligned" in msg


def test_create_and_workspace_sizes(lib):
    h, keep = make()
    try:
        n = rb.rp_prefix_workspace_bytes(h, 2, [0, 512, 1024])
        assert n > 1024 * 256 * 4
        s = rb.rp_suffix_workspace_bytes(h, 2, [0, 512, 1024], [0, 64, 128])
        assert s > 128 * 2048 * 4  # holds the fp32 logits
        assert rb.rp_suffix_workspace_bytes(h, 2, [0, 512, 1024], [0, 0, 0]) > 0
        assert rb.rp_decode_workspace_bytes(h, 4, 100) > 4 * 2048 * 4
    finally:
        rb.rp_destroy(h)


@pytest.mark.parametrize("B,cu,status", [
    (0, [0], rb.RP_ERR_SHAPE),
    (2, [1, 5, 9], rb.RP_ERR_SHAPE),
    (2, [0, 5, 5], rb.RP_ERR_SHAPE),
    (2, [0, 7, 3], rb.RP_ERR_SHAPE),
    (1, [0, 2000], rb.RP_ERR_SHAPE),          # longer than max_position
    (rb.RP_MAX_SEQS + 1, list(range(rb.RP_MAX_SEQS + 2)), rb.RP_ERR_SHAPE),
])
def test_bad_prefix_lengths(lib, B, cu, status):
    h, keep = make()
    try:
        st, msg = status_of(rb.rp_prefix_workspace_bytes, h, B, cu)
        assert st == status and msg
    finally:
        rb.rp_destroy(h)


def test_bad_suffix_lengths(lib):
    h, keep = make()
    try:
        assert status_of(rb.rp_suffix_workspace_bytes, h, 2, [0, 4, 8], [0, 3, 2])[0] == rb.RP_ERR_SHAPE
        assert status_of(rb.rp_suffix_workspace_bytes, h, 1, [0, 1000], [0, 30])[0] == rb.RP_ERR_SHAPE
        assert status_of(rb.rp_suffix_workspace_bytes, h, 1, [0, 10], [1, 30])[0] == rb.RP_ERR_SHAPE
    finally:
        rb.rp_destroy(h)


@pytest.mark.parametrize("n_prefix,pcu,n_suffix,grp,scu", [
    (2, [0, 4, 8], 3, [0, 2, 1], [0, 1, 2, 3]),      # prefix index out of range
    (2, [0, 4, 8], 2, [0, -1], [0, 1, 2]),           # negative prefix index
    (2, [0, 4, 8], 0, [], [0]),                      # no suffixes
    (2, [0, 4, 8], 2, [0, 1], [0, 3, 2]),            # decreasing suffix_cu
    (1, [0, 1010], 2, [0, 0], [0, 10, 30]),          # prefix + suffix > max_position
    (2, [0, 4, 4], 1, [0], [0, 2]),                  # empty prefix
])
def test_bad_grouped_suffix_arguments(lib, n_prefix, pcu, n_suffix, grp, scu):
    h, keep = make()
    try:
        st, msg = status_of(rb.rp_suffix_grouped_workspace_bytes, h, n_prefix, pcu, n_suffix, grp, scu)
        assert st == rb.RP_ERR_SHAPE and msg
    finally:
        rb.rp_destroy(h)


def test_grouped_suffix_workspace_and_validation(lib):
    h, keep = make()
    try:
        # eight responses of one prompt group over one prefix: same workspace as eight suffixes
        n = rb.rp_suffix_grouped_workspace_bytes(h, 1, [0, 512], 8, [0] * 8, list(range(0, 72, 8)))
        assert n == rb.rp_suffix_workspace_bytes(h, 8, list(range(0, 8 * 64 + 1, 64)), list(range(0, 72, 8)))
        m = configs.TINY
        kv = rb.make_kv(FAKE, FAKE + (1 << 30), 512 * m.n_kv_heads * m.head_dim)
        args = [h, None, 1, [0, 512], 2, [0, 0], [0, 3, 5], None, 0, kv, None, FAKE + (1 << 31),
                FAKE + (1 << 32), FAKE + (1 << 33), 1 << 30]
        assert status_of(rb.rp_suffix_logprob_grouped, *args)[0] == rb.RP_ERR_INVALID_ARG   # h_last NULL
        args[10] = FAKE + (1 << 34)
        need = rb.rp_suffix_grouped_workspace_bytes(h, 1, [0, 512], 2, [0, 0], [0, 3, 5])
        args[14] = need - 1
        assert status_of(rb.rp_suffix_logprob_grouped, *args)[0] == rb.RP_ERR_WORKSPACE
        args[14], args[8] = need, 6                                                        # unknown flag bits
        assert status_of(rb.rp_suffix_logprob_grouped, *args)[0] == rb.RP_ERR_INVALID_ARG
        args[8], args[7] = 0, [1022]                        # rotary positions past max_position
        assert status_of(rb.rp_suffix_logprob_grouped, *args)[0] == rb.RP_ERR_SHAPE
        args[7] = [-1]
        assert status_of(rb.rp_suffix_logprob_grouped, *args)[0] == rb.RP_ERR_SHAPE
        assert status_of(rb.rp_suffix_grouped_workspace_bytes, h, 1, [0, 512], 2, [0, 0], [0, 3, 5], 2)[0] == \
            rb.RP_ERR_INVALID_ARG
    finally:
        rb.rp_destroy(h)


def test_prefix_mrope_validation(lib):
    h, keep = make()
    try:
        args = list(_prefix_args(h))
        base = [args[0], args[1], args[2], args[3], args[4], args[5], args[6]]
        rest = args[7:]
        pos = FAKE + (1 << 35)
        assert status_of(rb.rp_prefix_forward_mrope, *base, None, [8, 12, 12], *rest)[0] == rb.RP_ERR_INVALID_ARG
        assert status_of(rb.rp_prefix_forward_mrope, *base, pos, [8, 12, 13], *rest)[0] == rb.RP_ERR_SHAPE
        assert status_of(rb.rp_prefix_forward_mrope, *base, pos, [-1, 17, 16], *rest)[0] == rb.RP_ERR_SHAPE
        assert status_of(rb.rp_prefix_forward_mrope, *base, pos + 4, [8, 12, 12], *rest)[0] == rb.RP_ERR_INVALID_ARG
    finally:
        rb.rp_destroy(h)


def test_prefix_flags_validation(lib):
    h, keep = make()
    try:
        args = list(_prefix_args(h))
        base, rest = args[:7], args[7:]
        last = rb.RP_PREFIX_LAST_ROWS_ONLY
        assert status_of(rb.rp_prefix_forward_flags, *base, None, None, 2, *rest)[0] == rb.RP_ERR_INVALID_ARG
        with_hidden = list(rest)
        with_hidden[2] = FAKE + (1 << 36)                       # hidden_out
        assert status_of(rb.rp_prefix_forward_flags, *base, None, None, last, *with_hidden)[0] == \
            rb.RP_ERR_INVALID_ARG
        assert status_of(rb.rp_prefix_forward_flags, *base, FAKE + (1 << 35), None, last, *rest)[0] == \
            rb.RP_ERR_INVALID_ARG
        bad_ws = list(rest)
        bad_ws[4] = 1000
        assert status_of(rb.rp_prefix_forward_flags, *base, None, None, last, *bad_ws)[0] == rb.RP_ERR_WORKSPACE
    finally:
        rb.rp_destroy(h)


def test_mfma_probe_validation(lib):
    assert status_of(rb.rp_calibrate_mfma, None, "f32", 1, 1, FAKE, 1 << 20)[0] == rb.RP_ERR_INVALID_ARG
    assert status_of(rb.rp_calibrate_mfma, None, "bf16", 0, 1, FAKE, 1 << 20)[0] == rb.RP_ERR_SHAPE
    assert status_of(rb.rp_calibrate_mfma, None, "bf16", 4, 1, FAKE, 4 * 256 * 4 - 1)[0] == rb.RP_ERR_WORKSPACE
    assert status_of(rb.rp_calibrate_mfma, None, "bf16", 4, 1, FAKE + 4, 1 << 20)[0] == rb.RP_ERR_INVALID_ARG
    assert status_of(rb.rp_calibrate_read, None, FAKE, 100, 4, FAKE, 1 << 20)[0] == rb.RP_ERR_SHAPE
    assert status_of(rb.rp_calibrate_read, None, FAKE, 1 << 20, 4, FAKE, 100)[0] == rb.RP_ERR_WORKSPACE
    assert status_of(rb.rp_calibrate_read, None, None, 1 << 20, 4, FAKE, 1 << 20)[0] == rb.RP_ERR_INVALID_ARG


def test_fused_scoring_workspace_holds_partials_not_logits(lib):
    h, keep = make(configs.QWEN7B_SLICE, max_pos=8192)
    try:
        args = (h, 1, [0, 4096], 8, [0] * 8, list(range(0, 8 * 256 + 1, 256)))
        plain = rb.rp_suffix_grouped_workspace_bytes(*args, 0)
        fused = rb.rp_suffix_grouped_workspace_bytes(*args, rb.RP_SUFFIX_FUSED_LOGPROB)
        R, V = 2048, configs.QWEN7B_SLICE.vocab
        parts = 2 * ((V + 255) // 256)
        assert plain - fused >= R * V * 4 - R * (parts * 8 + 4) - 4096
    finally:
        rb.rp_destroy(h)


def test_prompt_logprob_validation_and_workspace(lib):
    h, keep = make(configs.QWEN7B_SLICE, max_pos=8192)
    try:
        V, d = configs.QWEN7B_SLICE.vocab, configs.QWEN7B_SLICE.d_model
        plain = rb.rp_prompt_logprob_workspace_bytes(h, 1024)
        fused = rb.rp_prompt_logprob_workspace_bytes(h, 1024, rb.RP_SUFFIX_FUSED_LOGPROB)
        assert plain >= 1024 * (V * 4 + d * 2 + 4)
        assert fused < 1024 * (d * 2 + 4 + 8 * 2 * ((V + 255) // 256) + 4) + 4096
        assert rb.rp_prompt_logprob_workspace_bytes(h, 0) <= 4096
        assert status_of(rb.rp_prompt_logprob_workspace_bytes, h, -1)[0] == rb.RP_ERR_SHAPE
        assert status_of(rb.rp_prompt_logprob_workspace_bytes, h, 4, 2)[0] == rb.RP_ERR_INVALID_ARG
        need = rb.rp_prompt_logprob_workspace_bytes(h, 8)
        args = [h, None, 2, [0, 100, 300], FAKE, FAKE + (1 << 31), 8, FAKE + (1 << 32), 0, FAKE + (1 << 33),
                FAKE + (1 << 34), need]
        for i, st in ((4, rb.RP_ERR_INVALID_ARG), (5, rb.RP_ERR_INVALID_ARG), (7, rb.RP_ERR_INVALID_ARG),
                      (9, rb.RP_ERR_INVALID_ARG)):
            bad = list(args)
            bad[i] = None
            assert status_of(rb.rp_prompt_logprob, *bad)[0] == st, i
        bad = list(args); bad[11] = need - 1
        assert status_of(rb.rp_prompt_logprob, *bad)[0] == rb.RP_ERR_WORKSPACE
        bad = list(args); bad[5] = FAKE + 4                       # misaligned hidden
        assert status_of(rb.rp_prompt_logprob, *bad)[0] == rb.RP_ERR_INVALID_ARG
        bad = list(args); bad[6] = -3
        assert status_of(rb.rp_prompt_logprob, *bad)[0] == rb.RP_ERR_SHAPE
        bad = list(args); bad[3] = [0, 100, 100]                  # an empty prompt
        assert status_of(rb.rp_prompt_logprob, *bad)[0] == rb.RP_ERR_SHAPE
        bad = list(args); bad[8] = 4
        assert status_of(rb.rp_prompt_logprob, *bad)[0] == rb.RP_ERR_INVALID_ARG
        # no rows: nothing is launched and no pointer is needed
        rb.rp_prompt_logprob(h, None, 2, [0, 100, 300], None, None, 0, None, 0, None, FAKE, 4096)
    finally:
        rb.rp_destroy(h)


def _prefix_args(h, T=64, ws_bytes=None, stride=None, tokens=FAKE, ws=FAKE + (1 << 30)):
    m = configs.TINY
    kv = rb.make_kv(FAKE + (1 << 32), FAKE + (1 << 33),
                    stride if stride is not None else T * m.n_kv_heads * m.head_dim)
    need = rb.rp_prefix_workspace_bytes(h, 1, [0, T])
    return (h, None, 1, [0, T], tokens, None, 0, kv, FAKE + (1 << 34), None, ws,
            need if ws_bytes is None else ws_bytes)


def test_prefix_forward_validation(lib):
    h, keep = make()
    try:
        args = list(_prefix_args(h))
        args[4] = None
        assert status_of(rb.rp_prefix_forward, *args)[0] == rb.RP_ERR_INVALID_ARG
        assert status_of(rb.rp_prefix_forward, *_prefix_args(h, stride=10))[0] == rb.RP_ERR_SHAPE
        st, msg = status_of(rb.rp_prefix_forward, *_prefix_args(h, ws_bytes=1000))
        assert st == rb.RP_ERR_WORKSPACE and "workspace" in msg
        assert status_of(rb.rp_prefix_forward, *_prefix_args(h, ws=FAKE + 8))[0] == rb.RP_ERR_INVALID_ARG
        args = list(_prefix_args(h))
        args[6] = 5  # n_visual > 0 with no visual pointer
        assert status_of(rb.rp_prefix_forward, *args)[0] == rb.RP_ERR_INVALID_ARG
    finally:
        rb.rp_destroy(h)


def test_empty_suffix_is_a_no_op(lib):
    h, keep = make()
    try:
        m = configs.TINY
        kv = rb.make_kv(FAKE, FAKE + (1 << 30), 8 * m.n_kv_heads * m.head_dim)
        need = rb.rp_suffix_workspace_bytes(h, 2, [0, 4, 8], [0, 0, 0])
        rb.rp_suffix_logprob(h, None, 2, [0, 4, 8], [0, 0, 0], kv, FAKE + (1 << 31), None, None,
                             FAKE + (1 << 32), need)
    finally:
        rb.rp_destroy(h)


def test_launch_fault_injection_reports_hip_error():
    """RP_FAULT_INJECT makes the first launch fail before any HIP call is made."""
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from tests.test_abi_cpu import make, _prefix_args, status_of\n"
        "from paper_2608_14498_amd import binding as rb\n"
        "h, keep = make()\n"
        "st, msg = status_of(rb.rp_prefix_forward, *_prefix_args(h))\n"
        "print(st, msg)\n"
        "assert st == rb.RP_ERR_HIP and 'injected' in msg\n" % ROOT)
    env = dict(os.environ, RP_FAULT_INJECT="1")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr


BF16_D64 = configs.ModelShape(n_layers=2, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=64,
                              ffn_dim=512, vocab=2051, dtype="bf16")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_unexplained_fault_combinations_are_disabled(lib, dtype):
    """Two combinations that ran in a GPU run which faulted with no known cause are turned
    away before any HIP call: the bf16 decode step at head_dim 64 (its fp16 twin has run
    cleanly on the GPU), and the 16-bit last-rows-only prefix at head_dim 64 with 1-D
    positions.  head_dim 128 and fp32 still pass validation (checked up to a workspace
    error, which comes after the gate)."""
    from dataclasses import replace
    model = replace(BF16_D64, dtype=dtype)
    h, keep = make(model, max_pos=1024)
    try:
        T = 64
        kv = rb.make_kv(FAKE + (1 << 32), FAKE + (1 << 33), T * model.n_kv_heads * model.head_dim)
        need = rb.rp_prefix_workspace_bytes(h, 1, [0, T])
        args = (h, None, 1, [0, T], FAKE, None, 0, None, None, rb.RP_PREFIX_LAST_ROWS_ONLY, kv,
                FAKE + (1 << 34), None, FAKE + (1 << 30), need)
        st, msg = status_of(rb.rp_prefix_forward_flags, *args)
        assert st == rb.RP_ERR_UNSUPPORTED and "head_dim 64" in msg
        cap, B = 128, 4
        cache = rb.make_kv(FAKE + (1 << 32), FAKE + (1 << 33), B * cap * model.n_kv_heads * model.head_dim)
        dneed = rb.rp_decode_workspace_bytes(h, B, cap)
        st, msg = status_of(rb.rp_decode_step, h, None, B, cache, cap, FAKE, FAKE + 256, None, FAKE + 512,
                            FAKE + (1 << 30), dneed if dtype == "bf16" else 100)
        if dtype == "bf16":
            assert st == rb.RP_ERR_UNSUPPORTED and "head_dim 64" in msg
        else:
            assert st == rb.RP_ERR_WORKSPACE
    finally:
        rb.rp_destroy(h)
    for other in (replace(model, head_dim=128, n_q_heads=4, n_kv_heads=2), configs.TINY):
        h, keep = make(other, max_pos=1024)
        try:
            cap, B = 128, 4
            cache = rb.make_kv(FAKE + (1 << 32), FAKE + (1 << 33), B * cap * other.n_kv_heads * other.head_dim)
            st, _ = status_of(rb.rp_decode_step, h, None, B, cache, cap, FAKE, FAKE + 256, None, FAKE + 512,
                              FAKE + (1 << 30), 100)
            assert st == rb.RP_ERR_WORKSPACE
        finally:
            rb.rp_destroy(h)


def test_static_decode_validation(lib):
    """rp_decode_step_static checks its arguments and the scratch it needs before any HIP
    call: more than RP_DECODE_STATIC_SCRATCH_BYTES is RP_ERR_WORKSPACE."""
    text = open(HEADER).read()
    assert re.search(r"#define RP_DECODE_STATIC_SCRATCH_BYTES \(96u << 20\)", text)
    assert rb.RP_DECODE_STATIC_SCRATCH_BYTES == 96 << 20
    m = configs.QWEN7B_SLICE
    h, keep = make(m, max_pos=8300)
    try:
        def call(B, cap, logits=FAKE + (1 << 36), next_ids=FAKE + 512):
            cache = rb.make_kv(FAKE + (1 << 32), FAKE + (1 << 33), B * cap * m.n_kv_heads * m.head_dim)
            return status_of(rb.rp_decode_step_static, h, None, B, cache, cap, FAKE, FAKE + 256, logits, next_ids)
        st, msg = call(256, 8256)
        assert st == rb.RP_ERR_WORKSPACE and "static scratch" in msg
        # a batch whose scratch fits only without the [B, V] logits: with logits=None the
        # library would keep them in the scratch, and says so (above 64 rows; up to 64 rows
        # a 16-bit model takes the argmax inside the lm_head and stores no logits)
        lim = rb.RP_DECODE_STATIC_SCRATCH_BYTES
        fits = [B for B in range(72, 257, 8)
                if rb.rp_decode_workspace_bytes(h, B, 8256) - B * m.vocab * 4 <= lim < rb.rp_decode_workspace_bytes(h, B, 8256)]
        assert fits
        st, msg = call(fits[-1], 8256, logits=None)
        assert st == rb.RP_ERR_WORKSPACE and "logits" in msg
        assert call(64, 8256, next_ids=None)[0] == rb.RP_ERR_INVALID_ARG
        assert call(0, 8256)[0] == rb.RP_ERR_SHAPE
        need = rb.rp_decode_workspace_bytes(h, 64, 8256) - 64 * m.vocab * 4
        assert need <= rb.RP_DECODE_STATIC_SCRATCH_BYTES
    finally:
        rb.rp_destroy(h)


def test_debug_mode_workspaces_hold_guards():
    """RP_DEBUG puts a 256-byte guard after every workspace slice: the sizes grow by that
    much per slice (read in a child process: the mode is read once per process)."""
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from tests.test_abi_cpu import make\n"
        "from paper_2608_14498_amd import binding as rb, configs\n"
        "h, keep = make(configs.QWEN7B_SLICE, max_pos=8300)\n"
        "print(rb.rp_prefix_workspace_bytes(h, 2, [0, 100, 300]), rb.rp_suffix_workspace_bytes(h, 2, [0, 100, 300], [0, 5, 9]),"
        " rb.rp_decode_workspace_bytes(h, 4, 128))\n" % ROOT)
    sizes = []
    for dbg in ("0", "1"):
        env = dict(os.environ, RP_DEBUG=dbg)
        r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stderr
        sizes.append([int(x) for x in r.stdout.split()])
    for plain, guarded in zip(*sizes):
        extra = guarded - plain
        assert extra > 0 and extra % 256 == 0 and extra // 512 >= 4, (plain, guarded)
