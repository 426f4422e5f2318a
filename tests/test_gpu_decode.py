"""GPU parity of the decode step (one token per sequence, state in place)
against the float64 oracle of the recurrence.

A run of K decode steps from an initial state must reproduce, token by token,
the oracle's outputs over those K tokens and its final state; a decode run
continuing from ssd_forward's final state must match the oracle over the whole
sequence.  Tolerance as for the forward (max |gpu - oracle| / max |oracle|).
"""
import numpy as np
import pytest

import oracle
from paper_2405_21060_amd.inputs import Problem, make_inputs
from tests.ssd_harness import TOL, announce, rel_err, to_device, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2405_21060_amd import ssd

    ssd.load_library()


def decode_run(inp, start=0, state=None):
    """Decode tokens start..T-1 one by one; returns (y of those tokens, state)."""
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    p = inp.problem
    if state is None:
        state = (d["initial_states"].clone() if d["initial_states"] is not None else
                 torch.zeros((p.batch, p.nheads, p.headdim, p.dstate), dtype=torch.float32, device="cuda"))
    ys = []
    for t in range(start, p.seqlen):
        ys.append(ssd.decode_step(d["x"][:, t].contiguous(), d["dt"][:, t].contiguous(), d["A_log"],
                                  d["B"][:, t].contiguous(), d["C"][:, t].contiguous(), state, D=d["D"]))
    torch.cuda.synchronize()
    return torch.stack(ys, dim=1), state


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dims", [(64, 128, 8, 2), (16, 16, 3, 1), (64, 256, 4, 4), (128, 64, 2, 1),
                                  (32, 48, 6, 3)])
def test_decode_steps_match_oracle(dtype, dims):
    P, N, H, G = dims
    p = Problem(3, 7, H, P, N, G, 256, dtype, init_states=True)
    inp = make_inputs(p, 21)
    announce("decode %s P%d N%d H%d G%d" % (dtype, P, N, H, G))
    y, state = decode_run(inp)
    y_ref, fin_ref = oracle.forward_inputs(inp)
    ey, ef = rel_err(to_f64(y), y_ref), rel_err(state.cpu().numpy().astype(np.float64), fin_ref)
    announce("  rel err y %.3e state %.3e (tol %.0e)" % (ey, ef, TOL[dtype]))
    assert ey <= TOL[dtype] and ef <= TOL[dtype]


def test_decode_continues_forward():
    """Prefix through ssd_forward (its final state), the rest through decode steps."""
    from tests.ssd_harness import run_gpu
    import dataclasses

    p = Problem(2, 300, 8, 64, 128, 1, 256, "bf16", init_states=True)
    inp = make_inputs(p, 22)
    T0 = 290
    pre = dataclasses.replace(p, seqlen=T0)
    inp_pre = make_inputs(p, 22)
    inp_pre.problem = pre
    inp_pre.x, inp_pre.dt = inp.x[:, :T0].copy(), inp.dt[:, :T0].copy()
    inp_pre.B, inp_pre.C = inp.B[:, :T0].copy(), inp.C[:, :T0].copy()
    y_pre, fin = run_gpu(inp_pre)
    y_dec, state = decode_run(inp, start=T0, state=fin.clone())
    y_ref, fin_ref = oracle.forward_inputs(inp)
    ey = rel_err(np.concatenate([to_f64(y_pre), to_f64(y_dec)], axis=1), y_ref)
    ef = rel_err(state.cpu().numpy().astype(np.float64), fin_ref)
    announce("decode after forward: rel err y %.3e state %.3e" % (ey, ef))
    assert ey <= TOL["bf16"] and ef <= TOL["bf16"]


def test_decode_large_batch_sampled():
    """Decode shape of the 2.7B layer at batch 64, one step, all heads vs the oracle."""
    p = Problem(64, 1, 80, 64, 128, 1, 256, "bf16", init_states=True)
    inp = make_inputs(p, 23)
    y, state = decode_run(inp)
    y_ref, fin_ref = oracle.forward_inputs(inp)
    ey, ef = rel_err(to_f64(y), y_ref), rel_err(state.cpu().numpy().astype(np.float64), fin_ref)
    announce("decode b64 H80: rel err y %.3e state %.3e" % (ey, ef))
    assert ey <= TOL["bf16"] and ef <= TOL["bf16"]
