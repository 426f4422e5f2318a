"""GPU parity of the block path (ssd_forward_block) against the float64 oracle.

The dt parameterisation, the gate y * SiLU(z) and the grouped RMS
normalisation run in the HIP kernels (inside the fused chunk kernel where it
applies, else in the output pass); the oracle is oracle.block on the same
seeded inputs.  Tolerance as for the layer: max |gpu - oracle| / max |oracle|
per output tensor, 1e-4 for float32 inputs, 2e-2 for bfloat16.
"""
import numpy as np
import pytest

import oracle
import oracle.block as ob
from paper_2405_21060_amd.inputs import Problem, make_block_inputs
from tests.ssd_harness import TOL, announce, forward_workspace, rel_err, to_device, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2405_21060_amd import ssd

    ssd.load_library()


def _act(a):
    import torch

    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def run_block(bi, opts):
    import torch
    from paper_2405_21060_amd import ssd

    b = bi.base
    p = b.problem
    d = to_device(b)
    ws = forward_workspace(b)   # the block steps need no workspace of their own
    y, fin = ssd.forward_block(
        d["x"], _act(bi.dt_raw), d["A_log"], d["B"], d["C"], d["D"], chunk_size=p.chunk_size,
        initial_states=d["initial_states"], seq_idx=d["seq_idx"],
        nseq=b.nseq if b.seq_idx is not None else None, workspace=ws,
        dt_bias=torch.from_numpy(bi.dt_bias).cuda() if opts.get("dt_bias", True) else None,
        dt_softplus=opts.get("dt_softplus", True), dt_min=opts.get("dt_lo", 0.0),
        dt_max=opts.get("dt_hi", float("inf")),
        z=_act(bi.z) if opts.get("gate", True) else None,
        norm_weight=torch.from_numpy(bi.norm_weight).cuda() if opts.get("norm_weight", True) else None,
        norm_group_size=opts.get("norm_group_size", 0), norm_eps=opts.get("norm_eps", 1e-5))
    torch.cuda.synchronize()
    assert ssd.workspace_status(ws) == ssd.SSD_OK, "a chunk's state wait gave up"
    return y, fin


def check_block(bi, opts, tag):
    p = bi.base.problem
    announce("block %s %s b%d T%d H%d P%d N%d G%d Q%d varlen=%s opts=%s" % (
        tag, p.dtype, p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
        p.varlen, sorted(opts.items())))
    y, fin = run_block(bi, opts)
    y_ref, fin_ref = ob.block_forward_inputs(bi, opts)
    ey = rel_err(to_f64(y), y_ref)
    ef = rel_err(fin.cpu().numpy().astype(np.float64), fin_ref)
    announce("  rel err y %.3e final %.3e (tol %.0e)" % (ey, ef, TOL[p.dtype]))
    assert np.all(np.isfinite(to_f64(y)))
    assert ey <= TOL[p.dtype], ey
    assert ef <= TOL[p.dtype], ef


SHAPES = {
    # fused path: bf16, P 64, N 128 / 64, Q 256; ragged T, several chunks and items
    "fused_n128": Problem(2, 600, 8, 64, 128, 1, 256, "bf16", init_states=True),
    "fused_n64_g2": Problem(1, 700, 4, 64, 64, 2, 256, "bf16"),
    # the state in two column blocks (N 256)
    "fused_n256_g2": Problem(1, 900, 4, 64, 256, 2, 256, "bf16", init_states=True),
    # fused path on a packed row (the device chunk table), short and long sequences
    "fused_varlen": Problem(1, 1500, 8, 64, 128, 2, 256, "bf16", varlen=True, len_lo=1, len_hi=700,
                            init_states=True),
    # general path: fp32, and packed variable-length rows
    "general_f32": Problem(1, 200, 4, 16, 16, 2, 64, "f32", init_states=True),
    "general_varlen": Problem(1, 1500, 4, 32, 32, 2, 128, "bf16", varlen=True, len_lo=100,
                              len_hi=700, init_states=True),
}

OPTS = {
    "dt_only": dict(gate=False),
    "gate": dict(),
    "gate_headnorm": dict(norm_group_size="P"),
    "gate_norm2heads": dict(norm_group_size="2P"),
    "rownorm_clamp": dict(norm_group_size="HP", dt_lo=0.01, dt_hi=0.5),
    "norm_only_unit_weight": dict(gate=False, norm_group_size="P", norm_weight=False, norm_eps=1e-3),
    "no_softplus": dict(dt_softplus=False, dt_lo=0.002, norm_group_size="P"),
}


def resolve(opts, p):
    o = dict(opts)
    g = o.get("norm_group_size", 0)
    if isinstance(g, str):
        o["norm_group_size"] = {"P": p.headdim, "2P": 2 * p.headdim, "HP": p.nheads * p.headdim}[g]
    return o


@pytest.mark.parametrize("oname", sorted(OPTS))
@pytest.mark.parametrize("sname", sorted(SHAPES))
def test_block_matches_oracle(sname, oname):
    p = SHAPES[sname]
    check_block(make_block_inputs(p, 11), resolve(OPTS[oname], p), "%s/%s" % (sname, oname))


@pytest.mark.parametrize("early", ["0", "1"])
@pytest.mark.parametrize("sname", ["fused_n128", "fused_varlen"])
def test_block_state_flag_placement(sname, early, tune):
    # the gate and per-head normalisation in the chunk kernel's output stage with
    # either placement of the state flag, few persistent workgroups
    tune("early_state_flag", 2 if early == "1" else 1)
    tune("max_workgroups", 4)
    p = SHAPES[sname]
    check_block(make_block_inputs(p, 14), resolve(OPTS["gate_headnorm"], p), "flag%s/%s" % (early, sname))


@pytest.mark.parametrize("oname", ["gate_headnorm", "gate_norm2heads", "rownorm_clamp"])
def test_block_output_pass_separate(oname, tune):
    # the fused chunk kernel with gate and normalisation left to the output pass
    tune("separate_block_post", 1)
    p = SHAPES["fused_n128"]
    check_block(make_block_inputs(p, 12), resolve(OPTS[oname], p), "separate/" + oname)


@pytest.mark.parametrize("oname", ["gate_headnorm", "rownorm_clamp"])
def test_block_general_path_at_fused_shape(oname, tune):
    tune("force_general_path", 1)
    p = SHAPES["fused_n128"]
    check_block(make_block_inputs(p, 13), resolve(OPTS[oname], p), "unfused/" + oname)


def test_block_fused_equals_separate_output_pass(tune):
    # same inputs through the in-kernel gate/norm and through the output pass:
    # both within bf16 rounding of each other (one extra rounding of y)
    import torch

    p = SHAPES["fused_n128"]
    bi = make_block_inputs(p, 14)
    o = resolve(OPTS["gate_headnorm"], p)
    announce("block fused vs separate output pass")
    y1, f1 = run_block(bi, o)
    tune("separate_block_post", 1)
    y2, f2 = run_block(bi, o)
    assert torch.equal(f1, f2)   # the states do not depend on the output side
    e = rel_err(to_f64(y1), to_f64(y2))
    announce("  rel diff %.3e" % e)
    assert e <= 2e-2


def test_block_full_size_sampled_heads():
    # the 2.7B-layer shape with every step (per-head normalisation: heads are
    # independent, so the oracle runs only the sampled ones)
    import torch

    p = Problem(4, 4096, 80, 64, 128, 1, 256, "bf16")
    bi = make_block_inputs(p, 0)
    o = dict(norm_group_size=64, dt_lo=0.0, dt_hi=1.0)
    announce("block full size 2.7B sampled heads")
    y, fin = run_block(bi, o)
    heads = np.array([0, 1, 37, 40, 79])
    b = bi.base
    f64 = b.as_f64
    dt = ob.dt_transform(bi.as_f64("dt_raw")[:, :, heads], bi.dt_bias[heads], 0.0, 1.0)
    y_ref, fin_ref = oracle.forward(f64("x")[:, :, heads], dt, b.A_log[heads], f64("B"), f64("C"),
                                    b.D[heads])
    y_ref = ob.gate(y_ref, bi.as_f64("z")[:, :, heads])
    w = bi.norm_weight.reshape(80, 64)[heads].reshape(-1)
    y_ref = ob.group_rmsnorm(y_ref, w, 64, 1e-5)
    ey = rel_err(to_f64(y)[:, :, heads], y_ref)
    ef = rel_err(fin.cpu().numpy().astype(np.float64)[:, heads], fin_ref)
    announce("  rel err y %.3e final %.3e" % (ey, ef))
    assert ey <= TOL["bf16"] and ef <= TOL["bf16"]
