"""Seeded host inputs (``inputs.Inputs``) onto the HIP device as torch
tensors in the library's layouts (argument marshalling only)."""
from __future__ import annotations

import numpy as np

from .inputs import Inputs


def act_to_device(a: np.ndarray):
    """An activation array (float32, or bfloat16 bits as uint16) on the device."""
    import torch

    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_device(inp: Inputs) -> dict:
    """Every input of ``ssd_forward`` on the device (None where absent)."""
    import torch

    act = act_to_device
    return {
        "x": act(inp.x), "dt": act(inp.dt), "B": act(inp.B), "C": act(inp.C),
        "A_log": torch.from_numpy(inp.A_log).cuda(), "D": torch.from_numpy(inp.D).cuda(),
        "initial_states": None if inp.initial_states is None
        else torch.from_numpy(inp.initial_states).cuda(),
        "seq_idx": None if inp.seq_idx is None else torch.from_numpy(inp.seq_idx).cuda(),
    }
