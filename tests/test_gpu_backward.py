"""Parity of the HIP backward (``ssd_backward`` through the C ABI) with the
backward oracle (oracle/backward.py: the float64 adjoint of the recurrence,
pinned by finite differences of the forward oracle).

Every output is compared by max |gpu - oracle| / max |oracle| against the
forward's tolerances (float32 1e-4, bfloat16 2e-2).  The oracle runs on the
same rounded inputs.  Sizes span several 32-token chunks with a ragged last
chunk, grouped heads, heads split into slices per workgroup (with a short last
slice), optional D / initial states / final-state gradient, and the dimension
limits.  At the 2.7B layer shape two checks run on the full launch: the
gradients of a subset of heads of one batch row (dx, ddt and the initial-state
gradient depend only on their own head), and a loss that reads only the first
40 tokens (dy zero after them, no final-state gradient), whose gradients equal
those of the 40-token problem and vanish beyond it.
"""
import numpy as np
import pytest

import oracle.backward as ob
from paper_2405_21060_amd.inputs import Problem, bf16_bits_to_f32, make_grad_inputs, make_inputs, workload
from tests.ssd_harness import TOL, act_to_device, announce, rel_err, to_device, to_f64

pytestmark = pytest.mark.gpu


def f64(a):
    if a is None:
        return None
    return bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


def gpu_backward(inp, dy, dfinal, use_D=True, use_init=True):
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    g = ssd.backward(d["x"], d["dt"], d["A_log"], d["B"], d["C"], act_to_device(dy),
                     D=d["D"] if use_D else None,
                     initial_states=d["initial_states"] if use_init else None,
                     dfinal_states=None if dfinal is None else torch.from_numpy(dfinal).cuda())
    torch.cuda.synchronize()
    out = {k: (None if v is None else to_f64(v)) for k, v in g.items()}
    return out


def oracle_backward(inp, dy, dfinal, use_D=True, use_init=True, heads=None, rows=None):
    sel_r = slice(None) if rows is None else rows
    sel_h = slice(None) if heads is None else heads
    x = f64(inp.x)[sel_r][:, :, sel_h]
    dt = f64(inp.dt)[sel_r][:, :, sel_h]
    B = f64(inp.B)[sel_r]
    C = f64(inp.C)[sel_r]
    A_log = inp.A_log.astype(np.float64)[sel_h]
    D = inp.D.astype(np.float64)[sel_h] if use_D else None
    init = None
    if use_init and inp.initial_states is not None:
        init = inp.initial_states.astype(np.float64)[sel_r][:, sel_h]
    dyv = f64(dy)[sel_r][:, :, sel_h]
    dfin = None if dfinal is None else dfinal.astype(np.float64)[sel_r][:, sel_h]
    return ob.backward(x, dt, A_log, B, C, dyv, D=D, initial_states=init, dfinal=dfin)


def check(name, got, ref, tol):
    e = rel_err(got, ref)
    print("  %-7s rel err %.2e" % (name, e), flush=True)
    assert np.all(np.isfinite(got)), name
    assert e <= tol, "%s: %g > %g" % (name, e, tol)


# (batch, seqlen, heads, headdim, dstate, groups, dtype, D, initial states, final-state gradient)
CASES = [
    (2, 100, 4, 32, 16, 2, "f32", True, True, True),
    (1, 64, 2, 16, 32, 1, "f32", False, False, False),
    (2, 257, 6, 64, 128, 2, "bf16", True, True, True),
    (1, 1, 2, 16, 16, 1, "f32", True, True, True),
    (1, 31, 2, 16, 16, 1, "bf16", True, False, True),
    (1, 200, 3, 128, 256, 1, "f32", True, True, False),
    (1, 33, 3, 48, 64, 3, "bf16", False, True, True),
    (3, 96, 8, 64, 64, 1, "bf16", True, False, True),
    # 80 heads per group over 64 chunks: four slices of 20 heads per workgroup
    (1, 2048, 80, 16, 16, 1, "f32", True, True, True),
    # six heads per group over 1024 (row, chunk, group) units: a whole group per workgroup
    (1, 16384, 12, 16, 16, 2, "f32", True, True, True),
    # matrix-core shapes (bf16, headdim 64, dstate 64 or 128)
    (1, 1, 2, 64, 64, 1, "bf16", True, True, True),
    (2, 130, 4, 64, 128, 2, "bf16", True, True, True),
    (1, 64, 3, 64, 64, 3, "bf16", False, False, False),
    (2, 200, 8, 64, 128, 1, "bf16", True, False, True),
    (1, 63, 2, 64, 128, 1, "bf16", True, True, False),
]

# shapes of the matrix-core path, also run on the general path (force_general_path),
# and with heads split into slices of 3 per workgroup (bwd_heads_per_slice)
FAST_SHAPES = [
    (2, 257, 6, 64, 128, 2, "bf16", True, True, True),
    (3, 96, 8, 64, 64, 1, "bf16", True, False, True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "b%d_T%d_H%d_P%d_N%d_G%d_%s_D%d_i%d_f%d" % c)
def test_backward_matches_oracle(case):
    b, T, H, P, N, G, dtype, use_D, use_init, use_dfinal = case
    p = Problem(b, T, H, P, N, G, 256, dtype, init_states=use_init)
    announce("backward %s" % (case,))
    inp = make_inputs(p, 11)
    dy, dfinal = make_grad_inputs(p, 11)
    if not use_dfinal:
        dfinal = None
    got = gpu_backward(inp, dy, dfinal, use_D, use_init)
    ref = oracle_backward(inp, dy, dfinal, use_D, use_init)
    tol = TOL[dtype]
    for k in ("dx", "ddt", "dB", "dC", "dA_log", "dinit"):
        check(k, got[k], ref[k], tol)
    if use_D:
        check("dD", got["dD"], ref["dD"], tol)
    else:
        assert got["dD"] is None


@pytest.mark.parametrize("knob", ["force_general_path=1", "bwd_heads_per_slice=3"])
@pytest.mark.parametrize("case", FAST_SHAPES, ids=lambda c: "b%d_T%d_H%d_P%d_N%d_G%d_%s_D%d_i%d_f%d" % c)
def test_backward_knobs_match_oracle(case, knob, tune):
    name, value = knob.split("=")
    tune(name, int(value))
    test_backward_matches_oracle(case)


def test_backward_full_size_head_subset():
    """2.7B layer shape, full launch: dx, ddt and the initial-state gradient of
    heads 0, 37 and 79 of batch row 0 (each depends only on its own head)."""
    p = workload("mamba2_2p7b")
    p = Problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size, p.dtype,
                init_states=True)
    announce("backward full size, head subset %s" % (p,))
    inp = make_inputs(p, 5)
    dy, dfinal = make_grad_inputs(p, 5)
    got = gpu_backward(inp, dy, dfinal)
    heads = [0, 37, 79]
    ref = oracle_backward(inp, dy, dfinal, heads=heads, rows=slice(0, 1))
    tol = TOL[p.dtype]
    check("dx", got["dx"][0:1, :, heads], ref["dx"], tol)
    check("ddt", got["ddt"][0:1, :, heads], ref["ddt"], tol)
    check("dinit", got["dinit"][0:1, heads], ref["dinit"], tol)


def test_backward_full_size_prefix_loss():
    """2.7B layer shape, full launch, dy zero after the first 40 tokens and no
    final-state gradient: every gradient equals the 40-token problem's on the
    prefix and is exactly zero after it."""
    p = workload("mamba2_2p7b")
    announce("backward full size, 40-token loss %s" % (p,))
    inp = make_inputs(p, 6)
    dy, _ = make_grad_inputs(p, 6)
    K = 40
    dy[:, K:] = 0
    got = gpu_backward(inp, dy, None)
    q = Problem(p.batch, K, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size, p.dtype)
    short = make_inputs(q, 0)
    for name in ("x", "dt", "B", "C"):
        setattr(short, name, np.ascontiguousarray(getattr(inp, name)[:, :K]))
    short.A_log, short.D = inp.A_log, inp.D
    ref = oracle_backward(short, np.ascontiguousarray(dy[:, :K]), None, use_init=False)
    tol = TOL[p.dtype]
    for k in ("dx", "ddt", "dB", "dC"):
        check(k, got[k][:, :K], ref[k], tol)
        assert not np.any(got[k][:, K:]), k
    for k in ("dA_log", "dD", "dinit"):
        check(k, got[k], ref[k], tol)



# ---- packed rows (ssd_backward_varlen): sequences given by host offsets

def gpu_backward_varlen(inp, dy, dfinal, starts, use_D=True):
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    g = ssd.backward_varlen(d["x"], d["dt"], d["A_log"], d["B"], d["C"], act_to_device(dy), starts,
                            D=d["D"] if use_D else None, initial_states=d["initial_states"],
                            dfinal_states=None if dfinal is None else torch.from_numpy(dfinal).cuda())
    torch.cuda.synchronize()
    return {k: (None if v is None else to_f64(v)) for k, v in g.items()}


def packed_inputs(p, lengths, seed):
    inp = make_inputs(p, seed)
    seq = np.repeat(np.arange(len(lengths), dtype=np.int32), lengths).reshape(1, -1)
    starts = [0] + list(np.cumsum(lengths))
    if inp.initial_states is not None:
        rng = np.random.default_rng([seed, 5])
        inp.initial_states = rng.standard_normal((len(lengths),) + inp.initial_states.shape[1:]).astype(np.float32)
    return inp, seq, starts


# (dtype, (T, H, P, N, G), sequence lengths, initial states, final-state gradient, D)
VARLEN_CASES = [
    ("bf16", (500, 4, 64, 128, 2), [37, 1, 200, 262], True, True, True),
    ("bf16", (300, 3, 64, 64, 1), [64, 64, 1, 171], False, True, False),
    ("f32", (300, 3, 32, 16, 1), [100, 64, 136], False, True, True),
    ("f32", (97, 2, 16, 32, 2), [5, 3, 1, 40, 48], True, False, True),
    # one launch over the row (matrix-core path): lengths around its 64-token
    # chunks, and many one-token sequences (more sequences than chunks)
    ("bf16", (1000, 8, 64, 128, 4), [64, 65, 63, 128, 300, 380], True, True, True),
    ("bf16", (700, 2, 64, 64, 1), [1] * 100 + [600], True, True, True),
]


@pytest.mark.parametrize("case", VARLEN_CASES, ids=lambda c: "%s_T%d_%dseq" % (c[0], c[1][0], len(c[2])))
def test_backward_packed_rows_match_oracle(case):
    dtype, (T, H, P, N, G), lengths, use_init, use_dfinal, use_D = case
    assert sum(lengths) == T
    p = Problem(1, T, H, P, N, G, 256, dtype, init_states=use_init)
    announce("backward packed rows %s" % (case,))
    inp, seq, starts = packed_inputs(p, lengths, 13)
    dy, dfinal = make_grad_inputs(p, 13, units=len(lengths))
    if not use_dfinal:
        dfinal = None
    got = gpu_backward_varlen(inp, dy, dfinal, starts, use_D)
    ref = ob.backward(f64(inp.x), f64(inp.dt), inp.A_log.astype(np.float64), f64(inp.B), f64(inp.C), f64(dy),
                      D=inp.D.astype(np.float64) if use_D else None, initial_states=inp.initial_states,
                      dfinal=dfinal, seq_idx=seq)
    tol = TOL[dtype]
    for k in ("dx", "ddt", "dB", "dC", "dA_log", "dinit"):
        check(k, got[k], ref[k], tol)
    if use_D:
        check("dD", got["dD"], ref["dD"], tol)


def test_backward_packed_rows_full_size_head_subset():
    """The packed 32768-token workload (64 heads in 8 groups, sequences of 256
    to 4096 tokens, initial states), full launch: dx, ddt and the initial-state
    gradients of heads 0, 8 and 63 (each depends only on its own head and
    group)."""
    p = workload("varlen_g8")
    announce("backward packed rows full size, head subset %s" % (p,))
    inp = make_inputs(p, 3)
    seq = inp.seq_idx.reshape(-1)
    starts = [0] + list(np.flatnonzero(np.diff(seq)) + 1) + [seq.size]
    dy, dfinal = make_grad_inputs(p, 3, units=inp.nseq)
    got = gpu_backward_varlen(inp, dy, dfinal, starts)
    heads, groups = [0, 8, 63], [0, 1, 7]
    ref = ob.backward(f64(inp.x)[:, :, heads], f64(inp.dt)[:, :, heads], inp.A_log.astype(np.float64)[heads],
                      f64(inp.B)[:, :, groups], f64(inp.C)[:, :, groups], f64(dy)[:, :, heads],
                      D=inp.D.astype(np.float64)[heads], initial_states=inp.initial_states[:, heads],
                      dfinal=dfinal[:, heads], seq_idx=inp.seq_idx)
    tol = TOL[p.dtype]
    check("dx", got["dx"][:, :, heads], ref["dx"], tol)
    check("ddt", got["ddt"][:, :, heads], ref["ddt"], tol)
    check("dinit", got["dinit"][:, heads], ref["dinit"], tol)


def test_backward_packed_rows_per_sequence_forced(tune):
    """The per-sequence launches (forced) at a shape that otherwise runs as
    one launch over the row."""
    tune("varlen_per_sequence", 1)
    test_backward_packed_rows_match_oracle(VARLEN_CASES[0])
