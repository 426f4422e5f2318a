"""ssd_forward_noalloc (the forward on the library's fixed scratch array, for
callers that cannot allocate) against ssd_forward with a caller workspace,
through the C ABI: two calls in a row on the fused path, the second with a
smaller input, then the general path; outputs bit-identical to ssd_forward's
(the same kernels on the same inputs) and within the oracle's tolerance; the
status word clean; a problem too large for the array rejected before any
work is enqueued."""
import numpy as np
import pytest

import oracle
from paper_2405_21060_amd.inputs import Problem, make_inputs
from tests.ssd_harness import TOL, announce, forward_workspace, head_rel_err, rel_err, to_device, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2405_21060_amd import ssd

    ssd.load_library()


def _prob(inp, ssd):
    p = inp.problem
    return ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                            ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32, 0)


def _both(inp):
    """(y, final) from ssd_forward_noalloc and from ssd_forward, and the
    no-alloc call's status word."""
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    prob = _prob(inp, ssd)
    ptr = lambda t: 0 if t is None else t.data_ptr()
    b, T, H, P = d["x"].shape
    N = d["B"].shape[3]
    stream = torch.cuda.current_stream().cuda_stream
    out = []
    status = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    for noalloc in (True, False):
        y = torch.empty_like(d["x"])
        fin = torch.empty((b, H, P, N), dtype=torch.float32, device="cuda")
        args = (ptr(d["x"]), ptr(d["dt"]), ptr(d["A_log"]), ptr(d["B"]), ptr(d["C"]), ptr(d["D"]),
                ptr(d["initial_states"]), 0, ptr(y), ptr(fin))
        if noalloc:
            rc = ssd.ssd_forward_noalloc(prob, *args, ptr(status), stream)
        else:
            ws = forward_workspace(inp)
            rc = ssd.ssd_forward(prob, *args, ptr(ws), ws.numel(), stream)
        assert rc == ssd.SSD_OK, ssd.ssd_error_string(rc)
        out.append((y, fin))
    torch.cuda.synchronize()
    return out[0], out[1], int(status.item())


def _check(inp, tag):
    import torch

    p = inp.problem
    announce("no-alloc %s: b%d T%d H%d P%d N%d G%d Q%d %s" % (tag, p.batch, p.seqlen, p.nheads, p.headdim,
                                                               p.dstate, p.ngroups, p.chunk_size, p.dtype))
    (y1, f1), (y2, f2), status = _both(inp)
    assert status == 0
    if y1.dtype == torch.bfloat16:
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    else:
        assert torch.equal(y1, y2)
    assert torch.equal(f1, f2)
    y_ref, f_ref = oracle.forward_inputs(inp)
    yg, fg = to_f64(y1), f1.cpu().numpy().astype(np.float64)
    ey, ef = rel_err(yg, y_ref), rel_err(fg, f_ref)
    wy, wf = head_rel_err(yg, y_ref, 2).max(), head_rel_err(fg, f_ref, 1).max()
    announce("  bit-identical to ssd_forward; vs oracle y %.2e final %.2e (worst head %.2e %.2e)"
             % (ey, ef, wy, wf))
    tol = TOL[p.dtype]
    assert max(ey, ef, wy, wf) <= tol


def test_noalloc_equals_ssd_forward_two_calls():
    # fused path: a larger call, then a smaller one on the same scratch array
    _check(make_inputs(Problem(2, 3000, 16, 64, 128, 2, 256, "bf16", init_states=True), 71), "fused, first")
    _check(make_inputs(Problem(1, 700, 4, 64, 64, 1, 256, "bf16", init_states=True), 72), "fused, smaller")


def test_noalloc_general_path():
    _check(make_inputs(Problem(1, 500, 3, 32, 48, 3, 64, "f32", init_states=True), 73), "general f32")


def test_noalloc_rejects_problems_beyond_the_array():
    from paper_2405_21060_amd import ssd

    prob = ssd.make_problem(128, 512, 80, 64, 128, 1, 256, ssd.SSD_DTYPE_BF16, 0)   # state ring alone > 64 MiB
    assert ssd.ssd_workspace_bytes(prob) > ssd.SSD_NOALLOC_SCRATCH_BYTES
    fake = 0x10000   # never dereferenced: rejected before anything is enqueued
    rc = ssd.ssd_forward_noalloc(prob, fake, fake, fake, fake, fake, 0, 0, 0, fake, 0, 0, 0)
    assert rc == ssd.SSD_ERR_SCRATCH_TOO_SMALL
