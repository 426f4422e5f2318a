"""GPU parity of the sequence-span entry points (context parallelism).

A sequence is cut into spans; every span runs ssd_forward from a zero state;
ssd_span_decay, ssd_span_combine and ssd_span_correct then give the outputs,
the entering states and the final state of the whole sequence, which are
compared with the float64 oracle of the whole sequence (oracle.forward, and
oracle.span for the per-span pieces).  Tolerance as for the layer.
"""
import numpy as np
import pytest

import oracle
import oracle.span as osp
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


def split_run(inp, cuts):
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    p = inp.problem
    ys, fins, decs = [], [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        sl = lambda t: t[:, a:b].contiguous()
        y, fin = ssd.forward(sl(d["x"]), sl(d["dt"]), d["A_log"], sl(d["B"]), sl(d["C"]), d["D"],
                             chunk_size=p.chunk_size)
        ys.append(y)
        fins.append(fin)
        decs.append(ssd.span_decay(sl(d["dt"]), d["A_log"]))
    entering, final = ssd.span_combine(torch.stack(decs), torch.stack(fins), d["initial_states"])
    for r, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
        ssd.span_correct(d["dt"][:, a:b].contiguous(), d["A_log"], d["C"][:, a:b].contiguous(),
                         entering[r].contiguous(), ys[r])
    torch.cuda.synchronize()
    return torch.cat(ys, dim=1), final, entering, decs


CASES = {
    # fused-path spans (bf16, P 64, N 128), ragged spans, grouped B/C, initial state
    "fused": (Problem(2, 1200, 8, 64, 128, 2, 256, "bf16", init_states=True), [0, 300, 777, 1200]),
    # float32 (general path, plain-FMA correction)
    "f32": (Problem(1, 500, 4, 16, 32, 2, 64, "f32", init_states=True), [0, 130, 257, 500]),
    # N = 48: the matrix-core K-step of 32 padded with zeros
    "n48": (Problem(1, 600, 4, 32, 48, 1, 128, "bf16"), [0, 200, 600]),
    # P 128, N 256: 68 KB of LDS for the entering state
    "p128_n256": (Problem(1, 300, 2, 128, 256, 1, 64, "bf16", init_states=True), [0, 100, 300]),
    # one span only: the combine is the identity on the initial state
    "one_span": (Problem(1, 520, 4, 64, 64, 1, 256, "bf16", init_states=True), [0, 520]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_spans_reproduce_whole_sequence(name):
    p, cuts = CASES[name]
    inp = make_inputs(p, 31)
    announce("spans %s %s b%d T%d H%d P%d N%d G%d cuts=%s" % (name, p.dtype, p.batch, p.seqlen, p.nheads,
                                                           p.headdim, p.dstate, p.ngroups, cuts))
    y, final, entering, decs = split_run(inp, cuts)
    y_ref, fin_ref = oracle.forward_inputs(inp)
    ey, ef = rel_err(to_f64(y), y_ref), rel_err(final.cpu().numpy().astype(np.float64), fin_ref)
    # entering states and decays against oracle.span on the oracle's own span runs
    f = inp.as_f64
    dt = f("dt")
    dec_ref = np.stack([osp.span_decay(dt[:, a:b], inp.A_log) for a, b in zip(cuts[:-1], cuts[1:])])
    ed = rel_err(np.stack([d.cpu().numpy() for d in decs]).astype(np.float64), dec_ref)
    announce("  rel err y %.3e final %.3e decay %.3e (tol %.0e)" % (ey, ef, ed, TOL[p.dtype]))
    assert ey <= TOL[p.dtype] and ef <= TOL[p.dtype]
    assert ed <= 1e-5
    for r, a in enumerate(cuts[:-1]):
        if a == 0:
            ref = inp.initial_states if inp.initial_states is not None else np.zeros_like(fin_ref)
        else:
            _, ref = oracle.forward(f("x")[:, :a], dt[:, :a], inp.A_log, f("B")[:, :a], f("C")[:, :a],
                                    inp.D, initial_states=inp.initial_states)
        assert rel_err(entering[r].cpu().numpy().astype(np.float64), ref) <= TOL[p.dtype]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_span_correct_alone(dtype):
    # the correction kernel against oracle.span on one span with a random state
    import torch
    from paper_2405_21060_amd import ssd

    p = Problem(2, 700, 4, 32, 64, 2, 64, dtype, init_states=True)
    inp = make_inputs(p, 32)
    d = to_device(inp)
    announce("span_correct alone %s" % dtype)
    y0 = torch.zeros_like(d["x"])
    ssd.span_correct(d["dt"], d["A_log"], d["C"], d["initial_states"], y0)
    torch.cuda.synchronize()
    ref = osp.span_correction(inp.as_f64("dt"), inp.A_log, inp.as_f64("C"), inp.initial_states)
    e = rel_err(to_f64(y0), ref)
    announce("  rel err %.3e" % e)
    assert e <= TOL[dtype]


def test_spans_full_size_cp8():
    # the 2.7B layer cut into 8 spans of 512 tokens (one per GPU of an 8-way
    # context-parallel split), checked on sampled heads
    p = Problem(4, 4096, 80, 64, 128, 1, 256, "bf16")
    inp = make_inputs(p, 0)
    cuts = list(range(0, 4097, 512))
    announce("spans full size cp8")
    y, final, _, _ = split_run(inp, cuts)
    heads = [0, 1, 40, 79]
    y_ref, fin_ref = oracle.forward_inputs(inp, heads=heads)
    ey = rel_err(to_f64(y)[:, :, heads], y_ref)
    ef = rel_err(final.cpu().numpy().astype(np.float64)[:, heads], fin_ref)
    announce("  rel err y %.3e final %.3e" % (ey, ef))
    assert ey <= TOL["bf16"] and ef <= TOL["bf16"]
