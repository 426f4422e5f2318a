"""Helpers shared by the GPU tests: move seeded inputs to the device, run the
HIP path through the C ABI, compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

from paper_2405_21060_amd.inputs import Inputs, bf16_bits_to_f32

TOL = {"f32": 1e-4, "bf16": 2e-2}


def act_to_device(a: np.ndarray):
    """An activation array (float32, or bfloat16 bits as uint16) on the device."""
    import torch

    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_device(inp: Inputs):
    import torch

    act = act_to_device
    d = {
        "x": act(inp.x), "dt": act(inp.dt), "B": act(inp.B), "C": act(inp.C),
        "A_log": torch.from_numpy(inp.A_log).cuda(), "D": torch.from_numpy(inp.D).cuda(),
        "initial_states": None if inp.initial_states is None
        else torch.from_numpy(inp.initial_states).cuda(),
        "seq_idx": None if inp.seq_idx is None else torch.from_numpy(inp.seq_idx).cuda(),
    }
    return d


def to_f64(t) -> np.ndarray:
    import torch

    if t.dtype == torch.bfloat16:
        return bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def run_gpu(inp: Inputs, chunk_size=None, use_D=True, use_init=True, final=True):
    import torch
    from paper_2405_21060_amd import ssd

    d = to_device(inp)
    y, fin = ssd.forward(d["x"], d["dt"], d["A_log"], d["B"], d["C"], d["D"] if use_D else None,
                         chunk_size=chunk_size or inp.problem.chunk_size,
                         initial_states=d["initial_states"] if use_init else None,
                         seq_idx=d["seq_idx"], nseq=inp.nseq if inp.seq_idx is not None else None,
                         return_final_states=final)
    torch.cuda.synchronize()
    return y, fin


def rel_err(out: np.ndarray, ref: np.ndarray) -> float:
    """max |out - ref| / max |ref| (per output tensor)."""
    den = np.abs(ref).max()
    return float(np.abs(out - ref).max() / (den if den > 0 else 1.0))


def announce(msg: str):
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()
