"""Parity of the block gradients (``ssd_backward_block`` through the C ABI)
with the block-backward oracle (oracle/block_backward.py: the chain rule
through the normalisation, the gate, the layer's adjoint and the dt step in
float64, pinned by finite differences of the block forward oracle).

Every gradient is compared by max |gpu - oracle| / max |oracle| against the
forward's tolerances; the oracle is the definition (float64 from the given
inputs, nothing rounded in between), for bf16 activations too.  Cases: each
combination of gate and normalisation (groups of one head, two heads, the
whole channel row, and rows of 1024 and 2048 channels, which take the
normalisation kernels for wide groups), with and without the norm weight,
the dt clamp active, dt used as given, float32 and bfloat16 (at the
matrix-core shapes, and at others, which run in float32 on widened copies),
and at the 2.7B layer shape every per-head gradient of three heads over all
batch rows (with one-head normalisation groups those depend only on their
own head).
"""
import numpy as np
import pytest

import oracle.block_backward as obb
from paper_2405_21060_amd.inputs import Problem, bf16_bits_to_f32, make_block_inputs, make_grad_inputs, workload
from tests.ssd_harness import TOL, act_to_device, announce, rel_err, to_f64

pytestmark = pytest.mark.gpu


def f64(a):
    if a is None:
        return None
    return bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


def run_gpu(bi, dout, dfinal, o):
    """ssd_backward_block through the binding, with a workspace of our own
    whose status word (the recomputed forward's state passing) must be clean."""
    import torch
    from paper_2405_21060_amd import ssd

    base = bi.base
    p = base.problem
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    bias = dev(bi.dt_bias) if o["bias"] else None
    z = act_to_device(bi.z) if o["gate"] else None
    w = dev(bi.norm_weight) if o["weight"] else None
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, 256,
                            ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32)
    opts = ssd.make_block_opts(bias, o["softplus"], o["lo"], o["hi"], z, w, o["group"], 1e-5)
    ws = torch.empty(ssd.ssd_backward_block_workspace_bytes(prob, opts), dtype=torch.uint8, device="cuda")
    g = ssd.backward_block(
        act_to_device(base.x), act_to_device(o["dt_raw"]), dev(base.A_log), act_to_device(base.B),
        act_to_device(base.C), act_to_device(dout), D=dev(base.D), initial_states=dev(base.initial_states),
        dfinal_states=dev(dfinal), dt_bias=bias, dt_softplus=o["softplus"],
        dt_min=o["lo"], dt_max=o["hi"], z=z, norm_weight=w, norm_group_size=o["group"], norm_eps=1e-5,
        workspace=ws)
    torch.cuda.synchronize()
    assert ssd.workspace_status(ws) == ssd.SSD_OK, "a chunk's state wait gave up"
    return {k: (None if v is None else to_f64(v)) for k, v in g.items()}


def run_oracle(bi, dout, dfinal, o, heads=None, rows=None):
    base = bi.base
    sr = slice(None) if rows is None else rows
    sh = slice(None) if heads is None else heads
    P = base.problem.headdim
    ch = None if heads is None else np.concatenate([np.arange(h * P, (h + 1) * P) for h in heads])
    w = None
    if o["weight"]:
        w = bi.norm_weight.astype(np.float64) if ch is None else bi.norm_weight.astype(np.float64)[ch]
    return obb.block_backward(
        f64(base.x)[sr][:, :, sh], f64(o["dt_raw"])[sr][:, :, sh], base.A_log.astype(np.float64)[sh],
        f64(base.B)[sr], f64(base.C)[sr], f64(dout)[sr][:, :, sh], D=base.D.astype(np.float64)[sh],
        initial_states=None if base.initial_states is None else base.initial_states[sr][:, sh],
        dfinal=None if dfinal is None else dfinal[sr][:, sh],
        dt_bias=bi.dt_bias.astype(np.float64)[sh] if o["bias"] else None, dt_softplus=o["softplus"],
        dt_lo=o["lo"], dt_hi=o["hi"], z=f64(bi.z)[sr][:, :, sh] if o["gate"] else None, norm_weight=w,
        norm_group_size=o["group"], norm_eps=1e-5)


def check(name, got, ref, tol):
    e = rel_err(got, ref)
    print("  %-13s rel err %.2e" % (name, e), flush=True)
    assert np.all(np.isfinite(got)), name
    assert e <= tol, "%s: %g > %g" % (name, e, tol)


BASE = dict(gate=True, group=64, weight=True, bias=True, softplus=True, lo=0.0, hi=float("inf"))
CASES = [
    ("bf16", (2, 200, 4, 64, 128, 1), {}),
    ("bf16", (2, 200, 4, 64, 128, 1), dict(group=128)),
    ("bf16", (1, 150, 4, 64, 64, 2), dict(group=256)),
    ("bf16", (2, 130, 4, 64, 128, 1), dict(gate=False)),
    ("bf16", (2, 130, 4, 64, 128, 1), dict(group=0)),
    ("bf16", (2, 130, 4, 64, 128, 1), dict(gate=False, group=0)),
    ("bf16", (1, 100, 4, 64, 128, 1), dict(weight=False)),
    ("bf16", (1, 100, 4, 64, 128, 1), dict(lo=0.01, hi=0.05)),
    ("bf16", (1, 100, 4, 64, 128, 1), dict(bias=False, softplus=False, raw="dt")),
    ("f32", (1, 100, 4, 32, 16, 2), dict(group=32)),
    ("f32", (2, 70, 3, 16, 32, 3), dict(group=48, lo=0.01, hi=0.05)),
    # wide normalisation groups: 1024 channels (two pieces per lane: the weight
    # gradient folded into the group pass), without weight (the plain group
    # pass), 2048 channels (pieces re-read, then the separate weight pass)
    ("bf16", (1, 100, 16, 64, 128, 1), dict(group=1024)),
    ("bf16", (1, 100, 16, 64, 128, 1), dict(group=1024, weight=False)),
    ("bf16", (1, 80, 32, 64, 64, 2), dict(group=2048)),
    ("f32", (1, 60, 64, 16, 16, 1), dict(group=1024)),
    ("f32", (1, 60, 64, 32, 16, 2), dict(group=2048)),
    # bf16 outside the matrix-core shapes: run in float32 on widened copies
    ("bf16", (2, 150, 4, 32, 48, 2), dict(group=64)),
    ("bf16", (1, 100, 3, 64, 256, 1), dict(gate=False)),
]


@pytest.mark.parametrize("dtype,shape,kw", CASES,
                         ids=lambda c: str(c).replace(" ", "") if not isinstance(c, str) else c)
def test_block_backward_matches_oracle(dtype, shape, kw):
    b, T, H, P, N, G = shape
    o = dict(BASE, **kw)
    p = Problem(b, T, H, P, N, G, 256, dtype, init_states=True)
    announce("block backward %s %s %s" % (dtype, shape, kw))
    bi = make_block_inputs(p, 21)
    dout, dfinal = make_grad_inputs(p, 21)
    o["dt_raw"] = bi.base.dt if o.pop("raw", None) == "dt" else bi.dt_raw
    got = run_gpu(bi, dout, dfinal, o)
    ref = run_oracle(bi, dout, dfinal, o)
    tol = TOL[dtype]
    for k in ("dx", "dA_log", "dB", "dC", "dD", "dinit"):
        check(k, got[k], ref[k], tol)
    check("ddt_raw", got["ddt"], ref["ddt_raw"], tol)
    for k in ("ddt_bias", "dz", "dnorm_weight"):
        if ref[k] is None:
            assert got[k] is None, k
        else:
            check(k, got[k], ref[k], tol)


def test_block_backward_full_size_head_subset():
    """2.7B layer shape, gate and one-head normalisation groups, full launch:
    for heads 0, 37 and 79 over all batch rows, every gradient that depends
    on those heads alone -- dx, d dt_raw, dz, the initial-state gradient, and
    dA_log, dD, d dt_bias and the norm weight's gradient of those heads."""
    p = workload("mamba2_2p7b")
    p = Problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size, p.dtype,
                init_states=True)
    announce("block backward full size, head subset %s" % (p,))
    bi = make_block_inputs(p, 8)
    dout, dfinal = make_grad_inputs(p, 8)
    o = dict(BASE, dt_raw=bi.dt_raw)
    got = run_gpu(bi, dout, dfinal, o)
    heads = [0, 37, 79]
    ref = run_oracle(bi, dout, dfinal, o, heads=heads)
    tol = TOL[p.dtype]
    ch = np.concatenate([np.arange(h * p.headdim, (h + 1) * p.headdim) for h in heads])
    check("dx", got["dx"][:, :, heads], ref["dx"], tol)
    check("ddt_raw", got["ddt"][:, :, heads], ref["ddt_raw"], tol)
    check("dz", got["dz"][:, :, heads], ref["dz"], tol)
    check("dinit", got["dinit"][:, heads], ref["dinit"], tol)
    check("dA_log", got["dA_log"][heads], ref["dA_log"], tol)
    check("dD", got["dD"][heads], ref["dD"], tol)
    check("ddt_bias", got["ddt_bias"][heads], ref["ddt_bias"], tol)
    check("dnorm_weight", got["dnorm_weight"][ch], ref["dnorm_weight"], tol)
