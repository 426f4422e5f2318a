"""Host-side checks of the C ABI: the library loads, exports what the header
declares, and rejects invalid arguments before touching the device."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2405_21060_amd import ssd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssd.h")

# Fake, never dereferenced addresses: every call below fails validation first.
FAKE = 0x10000


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\s*\*)\s*(ssd_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def lib():
    return ssd.load_library()


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(ssd.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", ssd.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s+(\w+)$", out, re.M))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def prob(**kw):
    base = dict(batch=4, seqlen=4096, nheads=80, headdim=64, dstate=128, ngroups=1,
                chunk_size=256, dtype=ssd.SSD_DTYPE_BF16, nseq=0)
    base.update(kw)
    return ssd.make_problem(base["batch"], base["seqlen"], base["nheads"], base["headdim"],
                            base["dstate"], base["ngroups"], base["chunk_size"], base["dtype"],
                            base["nseq"])


def fwd(p, ws_bytes=1 << 40, seq_idx=0, x=FAKE):
    return ssd.ssd_forward(p, x, FAKE, FAKE, FAKE, FAKE, 0, 0, seq_idx, FAKE, 0, FAKE,
                           ws_bytes, 0)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), ssd.SSD_ERR_BAD_DTYPE),
    (dict(nheads=80, ngroups=3), ssd.SSD_ERR_BAD_SHAPE),
    (dict(seqlen=0), ssd.SSD_ERR_BAD_SHAPE),
    (dict(batch=-1), ssd.SSD_ERR_BAD_SHAPE),
    (dict(chunk_size=48), ssd.SSD_ERR_BAD_CHUNK),
    (dict(chunk_size=512), ssd.SSD_ERR_BAD_CHUNK),
    (dict(headdim=24), ssd.SSD_ERR_UNSUPPORTED_DIMS),
    (dict(headdim=256), ssd.SSD_ERR_UNSUPPORTED_DIMS),
    (dict(dstate=512), ssd.SSD_ERR_UNSUPPORTED_DIMS),
    (dict(dstate=8), ssd.SSD_ERR_UNSUPPORTED_DIMS),
    (dict(nheads=70000, ngroups=1), ssd.SSD_ERR_TOO_LARGE),
])
def test_validation_errors(lib, kw, code):
    p = prob(**kw)
    with pytest.raises(ssd.SsdError) as e:
        ssd.ssd_workspace_bytes(p)
    assert e.value.code == code
    assert fwd(p) == code


def test_seq_idx_rules(lib):
    assert fwd(prob(batch=2, nseq=3), seq_idx=FAKE) == ssd.SSD_ERR_SEQIDX_BATCH
    assert fwd(prob(batch=1, nseq=0), seq_idx=FAKE) == ssd.SSD_ERR_BAD_SHAPE
    assert fwd(prob(batch=1, seqlen=10, nseq=11), seq_idx=FAKE) == ssd.SSD_ERR_BAD_SHAPE


def test_null_and_workspace_errors(lib):
    p = prob()
    assert fwd(p, x=0) == ssd.SSD_ERR_NULL_ARG
    need = ssd.ssd_workspace_bytes(p)
    assert fwd(p, ws_bytes=need - 1) == ssd.SSD_ERR_WORKSPACE
    assert lib.ssd_workspace_bytes(None, None) == ssd.SSD_ERR_NULL_ARG


def test_workspace_grows_with_problem(lib):
    small = ssd.ssd_workspace_bytes(prob(batch=1, seqlen=256))
    large = ssd.ssd_workspace_bytes(prob())
    assert 0 < small < large
    assert ssd.ssd_workspace_bytes(prob(seqlen=4097)) > large  # partial chunk counted


def test_workspace_is_that_of_the_path_taken(lib, tune):
    # the fused kernels (bf16, P 64, N 128, chunk 256) keep two ring slots of
    # states; the general kernels keep every chunk state: forcing the general
    # path asks for more, and a fused-sized workspace is then refused
    p = prob(dtype=ssd.SSD_DTYPE_BF16)
    fused = ssd.ssd_workspace_bytes(p)
    tune("force_general_path", 1)
    general = ssd.ssd_workspace_bytes(p)
    assert fused < general
    assert fwd(p, ws_bytes=fused) == ssd.SSD_ERR_WORKSPACE
    # f32 runs on the general kernels either way
    tune("force_general_path", 0)
    q = prob(dtype=ssd.SSD_DTYPE_F32)
    f32 = ssd.ssd_workspace_bytes(q)
    tune("force_general_path", 1)
    assert ssd.ssd_workspace_bytes(q) == f32


def test_timed_entry_validates_like_forward(lib):
    def timed(p, ws_bytes=1 << 40, seq_idx=0, x=FAKE):
        return ssd.ssd_forward_timed(p, x, FAKE, FAKE, FAKE, FAKE, 0, 0, seq_idx, FAKE, 0, FAKE,
                                     ws_bytes, 0, 0, 0)
    for kw in (dict(dtype=7), dict(chunk_size=48), dict(dstate=8), dict(seqlen=0)):
        assert timed(prob(**kw)) == fwd(prob(**kw)) < 0
    p = prob()
    assert timed(p, x=0) == ssd.SSD_ERR_NULL_ARG
    assert timed(p, ws_bytes=ssd.ssd_workspace_bytes(p) - 1) == ssd.SSD_ERR_WORKSPACE
    assert timed(prob(batch=2, nseq=3), seq_idx=FAKE) == ssd.SSD_ERR_SEQIDX_BATCH


def test_decode_step_validation(lib):
    def dec(p, state=FAKE, x=FAKE):
        return ssd.ssd_decode_step(p, x, FAKE, FAKE, FAKE, FAKE, 0, state, FAKE, 0)
    assert dec(prob(dtype=7)) == ssd.SSD_ERR_BAD_DTYPE
    assert dec(prob(nheads=80, ngroups=3)) == ssd.SSD_ERR_BAD_SHAPE
    assert dec(prob(dstate=8)) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert dec(prob(headdim=24)) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert dec(prob(), state=FAKE + 4) == ssd.SSD_ERR_UNSUPPORTED_DIMS   # state not 16-byte aligned
    assert dec(prob(), x=0) == ssd.SSD_ERR_NULL_ARG
    assert dec(prob(), state=0) == ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_decode_step(None, *([None] * 9)) == ssd.SSD_ERR_NULL_ARG
    # seqlen and chunk_size play no part in a decode step
    assert dec(prob(seqlen=0, chunk_size=48), x=0) == ssd.SSD_ERR_NULL_ARG


def test_block_validation(lib):
    inf = float("inf")

    def blk(opts, p=None, ws_bytes=0, y=FAKE):
        return ssd.ssd_forward_block(p or prob(), opts, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0, 0, y, 0,
                                     0, ws_bytes, 0)

    def opts(**kw):
        base = dict(dt_bias=None, dt_softplus=True, dt_min=0.0, dt_max=inf, z=None, norm_weight=None,
                    norm_group_size=0, norm_eps=1e-5)
        base.update(kw)
        o = ssd.SsdBlockOpts()
        for k, v in base.items():
            setattr(o, k, v)
        return o

    # valid options get as far as the workspace check (no workspace given)
    assert blk(opts()) == ssd.SSD_ERR_WORKSPACE
    assert blk(opts(z=FAKE, norm_group_size=64, norm_weight=FAKE)) == ssd.SSD_ERR_WORKSPACE
    assert blk(opts(norm_group_size=80 * 64)) == ssd.SSD_ERR_WORKSPACE
    assert blk(opts(dt_min=0.5, dt_max=0.5)) == ssd.SSD_ERR_WORKSPACE
    assert lib.ssd_forward_block(prob(), None, *([FAKE] * 5), None, None, None, FAKE, None, FAKE,
                                 0, None) == ssd.SSD_ERR_NULL_ARG
    for bad in (dict(dt_min=-1.0), dict(dt_min=2.0, dt_max=1.0), dict(dt_max=float("nan")),
                dict(norm_group_size=32), dict(norm_group_size=64 * 3), dict(norm_group_size=-64),
                dict(norm_group_size=64, norm_eps=-1.0), dict(norm_group_size=64, norm_eps=inf)):
        assert blk(opts(**bad)) == ssd.SSD_ERR_BAD_OPTION, bad
    # the output pass reads 16-byte vectors
    assert blk(opts(z=FAKE + 2)) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert blk(opts(norm_group_size=64), y=FAKE + 8) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert blk(opts(norm_group_size=64, norm_weight=FAKE + 4)) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    # shape errors come first, as in ssd_forward
    assert blk(opts(dt_min=-1.0), p=prob(chunk_size=48)) == ssd.SSD_ERR_BAD_CHUNK
    size = ctypes.c_size_t(0)
    assert lib.ssd_block_workspace_bytes(prob(), None, ctypes.byref(size)) == ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_block_workspace_bytes(prob(), ctypes.byref(opts()), ctypes.byref(size)) == ssd.SSD_OK
    assert size.value == ssd.ssd_workspace_bytes(prob())


def test_span_validation(lib):
    size = ctypes.c_size_t(0)
    assert ssd.load_library().ssd_span_decay(None, FAKE, FAKE, FAKE, 0) == ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_span_decay(ctypes.byref(prob(dstate=8)), FAKE, FAKE, FAKE, None) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert lib.ssd_span_decay(ctypes.byref(prob()), None, FAKE, FAKE, None) == ssd.SSD_ERR_NULL_ARG
    # chunk_size plays no part in the span entry points
    assert lib.ssd_span_decay(ctypes.byref(prob(chunk_size=48)), None, FAKE, FAKE, None) == ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_span_combine(0, ctypes.byref(prob()), FAKE, FAKE, None, FAKE, None, None) == ssd.SSD_ERR_BAD_SHAPE
    assert lib.ssd_span_combine(2, ctypes.byref(prob()), FAKE, FAKE + 4, None, FAKE, None, None) == \
        ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert lib.ssd_span_combine(2, ctypes.byref(prob()), FAKE, None, None, FAKE, None, None) == ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_span_correct_workspace_bytes(ctypes.byref(prob()), ctypes.byref(size)) == ssd.SSD_OK
    assert size.value == 4 * 4 * 80 * 16   # one float per (batch, head, 256-token chunk)
    assert lib.ssd_span_correct(ctypes.byref(prob()), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == \
        ssd.SSD_ERR_WORKSPACE
    assert lib.ssd_span_correct(ctypes.byref(prob()), FAKE, FAKE, FAKE + 8, FAKE, FAKE, FAKE, 1 << 30, None) == \
        ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert lib.ssd_span_correct(ctypes.byref(prob()), FAKE, FAKE, None, FAKE, FAKE, FAKE, 1 << 30, None) == \
        ssd.SSD_ERR_NULL_ARG


def bwd(p, ws_bytes=1 << 40, init=0, dfinal=0, dinit=0, dy=FAKE, D=0, dD=0):
    return ssd.ssd_backward(p, FAKE, FAKE, FAKE, FAKE, FAKE, D, init, dy, dfinal, FAKE, FAKE, FAKE, FAKE,
                            FAKE, dD, dinit, FAKE, ws_bytes, 0)


def test_backward_validation(lib):
    size = ctypes.c_size_t(0)
    assert lib.ssd_backward_workspace_bytes(None, ctypes.byref(size)) == ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_backward_workspace_bytes(ctypes.byref(prob()), None) == ssd.SSD_ERR_NULL_ARG
    assert bwd(prob(dtype=7)) == ssd.SSD_ERR_BAD_DTYPE
    assert bwd(prob(nheads=80, ngroups=3)) == ssd.SSD_ERR_BAD_SHAPE
    assert bwd(prob(headdim=24)) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert bwd(prob(dstate=272)) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    # chunk_size plays no part in the backward
    assert bwd(prob(chunk_size=48), dy=0) == ssd.SSD_ERR_NULL_ARG
    assert bwd(prob(), dy=0) == ssd.SSD_ERR_NULL_ARG
    assert bwd(prob(), init=FAKE + 4) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert bwd(prob(), dfinal=FAKE + 8) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert bwd(prob(), dinit=FAKE + 12) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    need = ssd.ssd_backward_workspace_bytes(prob())
    assert bwd(prob(), ws_bytes=need - 1) == ssd.SSD_ERR_WORKSPACE
    assert ssd.ssd_backward(prob(), FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0, FAKE, 0, FAKE, FAKE, FAKE, FAKE, FAKE,
                            0, 0, 0, need, 0) == ssd.SSD_ERR_WORKSPACE
    # two bf16 states per (batch, 64-token chunk, head) dominate the workspace of the
    # matrix-core shapes, two float32 states per 32 tokens the others'
    states = 4 * (4096 // 64) * 80 * 64 * 128 * 2
    assert 2 * states <= need <= 2 * states + (256 << 20)
    states = 4 * (4096 // 32) * 80 * 64 * 128 * 4
    need32 = ssd.ssd_backward_workspace_bytes(prob(dtype=ssd.SSD_DTYPE_F32))
    assert 2 * states <= need32 <= 2 * states + (128 << 20)
    assert bwd(prob(), dy=FAKE + 2) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert ssd.ssd_backward(prob(seqlen=0), FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0, FAKE, 0, FAKE, FAKE, FAKE,
                            FAKE, FAKE, 0, 0, FAKE, need, 0, FAKE, FAKE) == ssd.SSD_ERR_BAD_SHAPE


def test_block_backward_validation(lib):
    size = ctypes.c_size_t(0)
    o = ssd.SsdBlockOpts(0, 1, 0.0, float("inf"), 0, 0, 0, 1e-5)
    assert lib.ssd_backward_block_workspace_bytes(ctypes.byref(prob()), None, ctypes.byref(size)) == \
        ssd.SSD_ERR_NULL_ARG
    assert lib.ssd_backward_block_workspace_bytes(ctypes.byref(prob()), ctypes.byref(o), ctypes.byref(size)) == \
        ssd.SSD_OK
    need = size.value
    # at least the layer's backward workspace (shared with the recomputed forward)
    assert need >= ssd.ssd_backward_workspace_bytes(prob())

    def call(opts, dz=0, ws=need, x=FAKE, dout=FAKE):
        return ssd.ssd_backward_block(prob(), opts, x, FAKE, FAKE, FAKE, FAKE, 0, 0, dout, 0, FAKE, FAKE, FAKE,
                                      FAKE, FAKE, 0, 0, 0, dz, 0, FAKE, ws, 0)

    assert call(ssd.SsdBlockOpts(0, 1, 2.0, 1.0, 0, 0, 0, 1e-5)) == ssd.SSD_ERR_BAD_OPTION   # max < min
    assert call(ssd.SsdBlockOpts(0, 1, 0.0, float("inf"), 0, 0, 48, 1e-5)) == ssd.SSD_ERR_BAD_OPTION
    assert call(ssd.SsdBlockOpts(0, 1, 0.0, float("inf"), FAKE, 0, 0, 1e-5)) == ssd.SSD_ERR_NULL_ARG  # dz
    assert call(o, dout=0) == ssd.SSD_ERR_NULL_ARG
    assert call(o, x=FAKE + 2) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert call(o, ws=need - 1) == ssd.SSD_ERR_WORKSPACE


def test_varlen_backward_validation(lib):
    p = prob(batch=1, seqlen=1000, nseq=3)
    starts = [0, 100, 600, 1000]
    need = ssd.ssd_backward_varlen_workspace_bytes(p, starts)
    # at least the backward workspace of the longest sequence (500 tokens)
    assert need >= ssd.ssd_backward_workspace_bytes(prob(batch=1, seqlen=500))

    def call(pp, st, ws=need, x=FAKE):
        return ssd.ssd_backward_varlen(pp, st, x, FAKE, FAKE, FAKE, FAKE, 0, 0, FAKE, 0, FAKE, FAKE, FAKE, FAKE,
                                       FAKE, 0, 0, FAKE, ws, 0)

    assert call(prob(batch=2, seqlen=1000, nseq=3), starts) == ssd.SSD_ERR_SEQIDX_BATCH
    assert call(p, [0, 100, 100, 1000]) == ssd.SSD_ERR_BAD_SHAPE        # empty sequence
    assert call(p, [1, 100, 600, 1000]) == ssd.SSD_ERR_BAD_SHAPE        # does not start at 0
    assert call(p, [0, 100, 600, 999]) == ssd.SSD_ERR_BAD_SHAPE         # does not end at seqlen
    assert call(prob(batch=1, seqlen=1000, nseq=0), [0]) == ssd.SSD_ERR_BAD_SHAPE
    assert call(p, starts, x=FAKE + 2) == ssd.SSD_ERR_UNSUPPORTED_DIMS
    assert call(p, starts, ws=need - 1) == ssd.SSD_ERR_WORKSPACE


def test_varlen_forward_validation(lib):
    p = prob(batch=1, seqlen=1000, nseq=3)
    starts = [0, 100, 600, 1000]
    need = ssd.ssd_forward_varlen_workspace_bytes(p, starts)
    assert need >= ssd.ssd_workspace_bytes(prob(batch=1, seqlen=500))

    def call(pp, st, ws=need, y=FAKE):
        return ssd.ssd_forward_varlen(pp, st, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0, y, 0, FAKE, ws, 0)

    assert call(prob(batch=2, seqlen=1000, nseq=3), starts) == ssd.SSD_ERR_SEQIDX_BATCH
    assert call(p, [0, 600, 100, 1000]) == ssd.SSD_ERR_BAD_SHAPE
    assert call(p, [0, 100, 600, 1001]) == ssd.SSD_ERR_BAD_SHAPE
    assert call(p, starts, y=0) == ssd.SSD_ERR_NULL_ARG
    assert call(p, starts, ws=need - 1) == ssd.SSD_ERR_WORKSPACE


def test_error_strings(lib):
    for code in range(0, -11, -1):
        s = ssd.ssd_error_string(code)
        assert s and s != "unknown ssd status"
    assert ssd.ssd_error_string(-100) == "unknown ssd status"


def test_tuning_hook_validates_names_and_values(lib):
    assert ssd.ssd_set_tuning("no_such_setting", 1) == ssd.SSD_ERR_BAD_OPTION
    assert ssd.ssd_set_tuning("force_general_path", 2) == ssd.SSD_ERR_BAD_OPTION
    assert ssd.ssd_set_tuning("early_state_flag", -1) == ssd.SSD_ERR_BAD_OPTION
    assert lib.ssd_set_tuning(None, 1) == ssd.SSD_ERR_NULL_ARG
    for name in ("force_general_path", "heads_per_item", "early_state_flag", "max_workgroups",
                 "separate_block_post", "bwd_heads_per_slice", "varlen_per_sequence",
                 "state_wait_limit", "fused_right_factor", "packed_order"):
        assert ssd.ssd_set_tuning(name, 1) == ssd.SSD_OK, name
        assert ssd.ssd_set_tuning(name, 0) == ssd.SSD_OK, name


def test_tuning_context_leaves_nothing_set_on_a_refused_setting(lib):
    p = prob(dtype=ssd.SSD_DTYPE_BF16)
    fused = ssd.ssd_workspace_bytes(p)
    with pytest.raises(ssd.SsdError):
        with ssd.tuning(force_general_path=1, no_such_setting=1):
            pass
    assert ssd.ssd_workspace_bytes(p) == fused   # force_general_path was put back


def test_workspace_status_null(lib):
    assert ssd.ssd_workspace_status(0, 0) == ssd.SSD_ERR_NULL_ARG
    assert "state" in ssd.ssd_error_string(ssd.SSD_ERR_STATE_TIMEOUT)
