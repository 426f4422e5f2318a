"""Helpers shared by the GPU tests: move seeded inputs to the device, run the
HIP path through the C ABI (with a caller-owned workspace whose status word
is checked after the call), compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

from paper_2405_21060_amd.device import act_to_device, to_device  # noqa: F401
from paper_2405_21060_amd.inputs import Inputs, bf16_bits_to_f32

TOL = {"f32": 1e-4, "bf16": 2e-2}


def to_f64(t) -> np.ndarray:
    import torch

    if t.dtype == torch.bfloat16:
        return bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def forward_workspace(inp: Inputs, chunk_size=None):
    """A device workspace sized for ``ssd_forward`` on ``inp``."""
    import torch
    from paper_2405_21060_amd import ssd

    p = inp.problem
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups,
                            chunk_size or p.chunk_size,
                            ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32,
                            inp.nseq if inp.seq_idx is not None else 0)
    return torch.empty(max(ssd.ssd_workspace_bytes(prob), 1), dtype=torch.uint8, device="cuda")


def run_gpu(inp: Inputs, chunk_size=None, use_D=True, use_init=True, final=True):
    """``ssd.forward`` on ``inp``; asserts that no state wait gave up."""
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    ws = forward_workspace(inp, chunk_size)
    y, fin = ssd.forward(d["x"], d["dt"], d["A_log"], d["B"], d["C"], d["D"] if use_D else None,
                         chunk_size=chunk_size or inp.problem.chunk_size,
                         initial_states=d["initial_states"] if use_init else None,
                         seq_idx=d["seq_idx"], nseq=inp.nseq if inp.seq_idx is not None else None,
                         return_final_states=final, workspace=ws)
    torch.cuda.synchronize()
    assert ssd.workspace_status(ws) == ssd.SSD_OK, "a chunk's state wait gave up"
    return y, fin


def rel_err(out: np.ndarray, ref: np.ndarray) -> float:
    """max |out - ref| / max |ref| (per output tensor)."""
    den = np.abs(ref).max() if ref.size else 0.0
    return float(np.abs(out - ref).max() / (den if den > 0 else 1.0)) if ref.size else 0.0


def head_rel_err(out: np.ndarray, ref: np.ndarray, axis: int) -> np.ndarray:
    """Per head (index ``axis``): max over the head's elements of |out - ref|,
    over max |ref| of that head (1 where the head's reference is all zero)."""
    o = np.moveaxis(out, axis, 0).reshape(out.shape[axis], -1)
    r = np.moveaxis(ref, axis, 0).reshape(ref.shape[axis], -1)
    den = np.abs(r).max(axis=1)
    return np.abs(o - r).max(axis=1) / np.where(den > 0, den, 1.0)


def elementwise_diag(out: np.ndarray, ref: np.ndarray) -> float:
    """Diagnostic only: max |out - ref| / (|ref| + mean |ref|)."""
    if not ref.size:
        return 0.0
    m = np.abs(ref).mean()
    return float((np.abs(out - ref) / (np.abs(ref) + (m if m > 0 else 1.0))).max())


def announce(msg: str):
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()
