"""Seeded synthetic SSD-layer inputs shaped like the paper's Mamba-2 layers.

This module only draws and rounds random numbers; it holds none of the SSD
arithmetic.  Both the CPU oracle (through the tests) and the HIP path (through
the tests and the benchmark) consume what it produces, so the two sides always
see identical input bytes.

Shapes (row-major, contiguous):

* ``x``                 (batch, seqlen, nheads, headdim)  activation dtype
* ``dt``                (batch, seqlen, nheads)           activation dtype, > 0
* ``A_log``             (nheads,)                         float32
* ``B``, ``C``          (batch, seqlen, ngroups, dstate)  activation dtype
* ``D``                 (nheads,)                         float32
* ``initial_states``    (batch|nseq, nheads, headdim, dstate) float32 or None
* ``seq_idx``           (1, seqlen) int32 or None (packed variable-length rows)

Recipe (one ``numpy.random.default_rng(seed)`` PCG64 stream, draws in float64,
in this order): ``A_log ~ U(0, ln 16)`` per head (so ``A = -exp(A_log)`` lies in
``[-16, -1]``); ``D ~ N(0,1)`` per head; ``dt_init ~ U(1e-3, 1e-1)`` per head and
``dt_bias = log(expm1(dt_init))``; ``dt = softplus(N(0,1) + dt_bias)`` per
(batch, token, head); ``x ~ N(0,1)``; ``B ~ N(0,1)/sqrt(N)``;
``C ~ N(0,1)/sqrt(N)``; for packed rows the sequence lengths
``~ U{len_lo..len_hi}`` until they cover the row (the last one cut to fit),
then ``initial_states ~ N(0,1)`` per sequence.  Values are rounded float64 ->
float32 (round to nearest even) and, for bf16 workloads, float32 -> bf16
(round to nearest even).  The paper's Mamba-2 models use ``d_inner = 2 d_model``
and head dimension 64 (d_model 768 -> 24 heads, d_model 2560 -> 80 heads).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

__all__ = [
    "Problem", "Inputs", "BlockInputs", "WORKLOADS", "make_inputs", "make_block_inputs", "make_grad_inputs",
    "f32_to_bf16_bits", "bf16_bits_to_f32", "workload",
]


@dataclasses.dataclass(frozen=True)
class Problem:
    batch: int
    seqlen: int
    nheads: int
    headdim: int
    dstate: int
    ngroups: int
    chunk_size: int
    dtype: str  # "f32" or "bf16"
    varlen: bool = False          # one packed row with seq_idx
    len_lo: int = 256             # varlen length range (inclusive)
    len_hi: int = 4096
    init_states: bool = False     # draw nonzero initial states

    @property
    def tokens(self) -> int:
        return self.batch * self.seqlen


@dataclasses.dataclass
class Inputs:
    problem: Problem
    x: np.ndarray            # float32 or uint16 (bf16 bits)
    dt: np.ndarray
    A_log: np.ndarray        # float32
    B: np.ndarray
    C: np.ndarray
    D: np.ndarray            # float32
    initial_states: Optional[np.ndarray]   # float32
    seq_idx: Optional[np.ndarray]          # int32 (1, seqlen)
    nseq: int

    def as_f64(self, name: str) -> np.ndarray:
        """Exact float64 image of a stored tensor (bf16 bits widened)."""
        a = getattr(self, name)
        if a is None:
            return None
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (inputs are finite)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _store(a64: np.ndarray, dtype: str) -> np.ndarray:
    a32 = a64.astype(np.float32)
    return f32_to_bf16_bits(a32) if dtype == "bf16" else a32


def _normal_blocks(rng, shape, scale, dtype, block=1 << 22):
    """N(0,1)*scale drawn in float64 in row-major order, stored per block."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    for s in range(0, n, block):
        e = min(n, s + block)
        out[s:e] = _store(rng.standard_normal(e - s) * scale, dtype)
    return out.reshape(shape)


def _softplus(v: np.ndarray) -> np.ndarray:
    return np.where(v > 20.0, v, np.log1p(np.exp(np.minimum(v, 20.0))))


def make_inputs(p: Problem, seed: int) -> Inputs:
    rng = np.random.default_rng(seed)
    H, P, N, G = p.nheads, p.headdim, p.dstate, p.ngroups
    b, T = p.batch, p.seqlen
    A_log = rng.uniform(0.0, math.log(16.0), H).astype(np.float32)
    D = rng.standard_normal(H).astype(np.float32)
    dt_init = rng.uniform(1e-3, 1e-1, H)
    dt_bias = np.log(np.expm1(dt_init))
    dt = np.empty((b, T, H), dtype=np.uint16 if p.dtype == "bf16" else np.float32)
    dtf = dt.reshape(b * T, H)
    rows = max(1, (1 << 22) // H)
    for s in range(0, b * T, rows):
        e = min(b * T, s + rows)
        dtf[s:e] = _store(_softplus(rng.standard_normal((e - s, H)) + dt_bias), p.dtype)
    x = _normal_blocks(rng, (b, T, H, P), 1.0, p.dtype)
    B = _normal_blocks(rng, (b, T, G, N), 1.0 / math.sqrt(N), p.dtype)
    C = _normal_blocks(rng, (b, T, G, N), 1.0 / math.sqrt(N), p.dtype)
    seq_idx = None
    nseq = b
    if p.varlen:
        if b != 1:
            raise ValueError("packed variable-length rows use batch == 1")
        lens = []
        while sum(lens) < T:
            lens.append(int(rng.integers(p.len_lo, p.len_hi, endpoint=True)))
        lens[-1] -= sum(lens) - T
        seq_idx = np.repeat(np.arange(len(lens), dtype=np.int32), lens).reshape(1, T)
        nseq = len(lens)
    init = None
    if p.init_states:
        init = _normal_blocks(rng, (nseq, H, P, N), 1.0, "f32")
    return Inputs(p, x, dt, A_log, B, C, D, init, seq_idx, nseq)


@dataclasses.dataclass
class BlockInputs:
    """Inputs of the layer with the block steps around it: the layer's own
    (``base``; its ``dt`` is not used) plus the raw dt, its per-head bias, the
    gate branch ``z`` and the normalisation weight."""
    base: Inputs
    dt_raw: np.ndarray       # (b, T, H) activation dtype, before bias and softplus
    dt_bias: np.ndarray      # (H,) float32
    z: np.ndarray            # (b, T, H, P) activation dtype
    norm_weight: np.ndarray  # (H * P,) float32

    def as_f64(self, name: str) -> np.ndarray:
        a = getattr(self, name)
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)


def make_grad_inputs(p: Problem, seed: int, units: int = None):
    """Output gradients for the backward, from their own stream
    ``default_rng([seed, 0x6AD])``: ``dy`` (b, T, H, P) ~ N(0, 1) in the
    activation dtype, then ``dfinal`` (units, H, P, N) ~ N(0, 1) float32, one
    state per batch row (or per sequence of a packed row: ``units``)."""
    rng = np.random.default_rng([seed, 0x6AD])
    dy = _normal_blocks(rng, (p.batch, p.seqlen, p.nheads, p.headdim), 1.0, p.dtype)
    dfinal = _normal_blocks(rng, (units or p.batch, p.nheads, p.headdim, p.dstate), 1.0, "f32")
    return dy, dfinal


def make_block_inputs(p: Problem, seed: int) -> BlockInputs:
    """``make_inputs(p, seed)`` plus, from a second stream
    ``default_rng([seed, 0xB10C])`` in this order: ``dt_init ~ U(1e-3, 1e-1)``
    per head and ``dt_bias = log(expm1(dt_init))`` (float32);
    ``dt_raw ~ N(0,1)`` per (batch, token, head); ``z ~ N(0,1)``;
    ``norm_weight ~ 1 + 0.1 N(0,1)`` per channel (float32)."""
    base = make_inputs(p, seed)
    rng = np.random.default_rng([seed, 0xB10C])
    H, P, b, T = p.nheads, p.headdim, p.batch, p.seqlen
    dt_bias = np.log(np.expm1(rng.uniform(1e-3, 1e-1, H))).astype(np.float32)
    dt_raw = _normal_blocks(rng, (b, T, H), 1.0, p.dtype)
    z = _normal_blocks(rng, (b, T, H, P), 1.0, p.dtype)
    norm_weight = (1.0 + 0.1 * rng.standard_normal(H * P)).astype(np.float32)
    return BlockInputs(base, dt_raw, dt_bias, z, norm_weight)


# The workloads: one tiny fp32 parity case and Mamba-2 layer shapes in bf16.
WORKLOADS = {
    "tiny_f32": Problem(1, 256, 2, 16, 16, 1, 64, "f32"),
    "mamba2_130m": Problem(8, 2048, 24, 64, 128, 1, 256, "bf16"),
    "mamba2_2p7b": Problem(4, 4096, 80, 64, 128, 1, 256, "bf16"),
    "sweep_T512_N128": Problem(128, 512, 80, 64, 128, 1, 256, "bf16"),
    "sweep_T4096_N128": Problem(16, 4096, 80, 64, 128, 1, 256, "bf16"),
    "sweep_T16384_N128": Problem(4, 16384, 80, 64, 128, 1, 256, "bf16"),
    "sweep_T65536_N128": Problem(1, 65536, 80, 64, 128, 1, 256, "bf16"),
    "sweep_T16384_N64": Problem(4, 16384, 80, 64, 64, 1, 256, "bf16"),
    "sweep_T16384_N256": Problem(4, 16384, 80, 64, 256, 1, 256, "bf16"),
    "varlen_g8": Problem(1, 32768, 64, 64, 128, 8, 256, "bf16", varlen=True,
                         init_states=True),
    # one GPU's share of the 2.7B layer under 8-way sharding: heads (tensor
    # parallel, B and C replicated) or the sequence (context parallel: each
    # rank's span with the state entering it)
    "tp8_2p7b": Problem(4, 4096, 10, 64, 128, 1, 256, "bf16"),
    "cp8_2p7b": Problem(4, 512, 80, 64, 128, 1, 256, "bf16", init_states=True),
}


def workload(name: str) -> Problem:
    return WORKLOADS[name]
