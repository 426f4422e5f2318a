"""CPU oracle for the SSD layer forward -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never calls it, and it
shares no code with the HIP path.

* :func:`forward` -- the sequential float64 recurrence (``ssd_oracle.c``),
  Section 2 eq. (s6) with the scalar transition of Section 5, the
  discretisation ``exp(dt*A)`` / ``dt*x`` and the skip term ``D``.
* :mod:`oracle.chunked` -- the block decomposition of Section 6 written out step
  by step in float64 numpy, exposing its intermediates (chunk cumsums, chunk
  states, states entering chunks) for per-step comparisons.
* :mod:`oracle.backward` -- gradients of the layer: the adjoint of the
  recurrence, token by token in reverse (the paper gives no backward
  algorithm); pinned by finite differences of :func:`forward`.
* :mod:`oracle.span` -- a sequence split into spans (Section 8.2 state
  passing with the scan operator of Appendix B): span decays, the combine of
  (decay, state) pairs, and the output a span's entering state adds.
* :mod:`oracle.block` -- the Mamba-2 block steps on either side of the layer
  (dt parameterisation; gate ``y * SiLU(z)`` and grouped RMS normalisation of
  Sections 7.1 and 8.1) around :func:`forward`.
* :mod:`oracle.block_backward` -- gradients of those block steps by the chain
  rule around :mod:`oracle.backward`; pinned by finite differences of
  :mod:`oracle.block`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ssd_oracle.c")
_LIB = os.path.join(_HERE, "libssd_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle (plain IEEE float64: no fast-math) with OpenMP."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-fno-fast-math", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def load_library(path: str):
    """Load a build of ``ssd_oracle.c`` from ``path`` with its signatures set."""
    lib = ctypes.CDLL(path)
    d = ctypes.POINTER(ctypes.c_double)
    i64 = ctypes.c_int64
    lib.ssd_oracle_forward.restype = ctypes.c_int
    lib.ssd_oracle_forward.argtypes = [i64] * 6 + [d] * 7 + [
        ctypes.POINTER(ctypes.c_int32), i64, d, d, ctypes.c_int]
    lib.ssd_oracle_max_threads.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load_library(_LIB)
    return _lib


def _p(a, ctype=ctypes.c_double):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def forward(x, dt, A_log, B, C, D=None, initial_states=None, seq_idx=None,
            nseq: Optional[int] = None, nthreads: Optional[int] = None,
            lib=None) -> Tuple[np.ndarray, np.ndarray]:
    """Sequential float64 SSD forward.

    Arguments are array-likes with the library's layouts: x (b,T,H,P),
    dt (b,T,H), A_log (H), B/C (b,T,G,N), D (H) or None, initial_states
    (b|nseq,H,P,N) or None, seq_idx (1,T) int32 or None.
    Returns ``(y (b,T,H,P), final_states (b|nseq,H,P,N))`` in float64.
    ``lib`` substitutes another build of the same C source (see :func:`load_library`).
    """
    f = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.float64)
    x, dt, A_log, B, C, D, init = map(f, (x, dt, A_log, B, C, D, initial_states))
    b, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    if seq_idx is not None:
        seq_idx = np.ascontiguousarray(seq_idx, dtype=np.int32).reshape(-1)
        if nseq is None:
            nseq = int(seq_idx[-1]) + 1
        units = nseq
    else:
        nseq = b
        units = b
    y = np.empty((b, T, H, P), dtype=np.float64)
    fin = np.empty((units, H, P, N), dtype=np.float64)
    rc = (lib or _load()).ssd_oracle_forward(
        b, T, H, P, N, G, _p(x), _p(dt), _p(A_log), _p(B), _p(C), _p(D), _p(init),
        _p(seq_idx, ctypes.c_int32), nseq, _p(y), _p(fin),
        int(nthreads if nthreads else default_threads()))
    if rc != 0:
        raise ValueError("ssd_oracle_forward failed with code %d" % rc)
    return y, fin


def forward_inputs(inp, heads=None, nthreads=None):
    """Run :func:`forward` on a :class:`paper_2405_21060_amd.inputs.Inputs`.

    ``heads`` optionally selects a subset of heads (the result then covers
    only those heads, in that order).  Heads of one group share B and C, so a
    subset is computed exactly as in the full run: each selected head gets
    its own copy of its group's B and C.  Only the selected slices are
    widened to float64.
    """
    from paper_2405_21060_amd.inputs import bf16_bits_to_f32

    def f64(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)

    p = inp.problem
    x, dt, B, C = inp.x, inp.dt, inp.B, inp.C
    A_log, D, init = inp.A_log, inp.D, inp.initial_states
    if heads is not None:
        heads = np.asarray(heads)
        groups = heads // (p.nheads // p.ngroups)
        x, dt = x[:, :, heads], dt[:, :, heads]
        B, C = B[:, :, groups], C[:, :, groups]
        A_log, D = A_log[heads], D[heads]
        if init is not None:
            init = init[:, heads]
    return forward(f64(x), f64(dt), f64(A_log), f64(B), f64(C), f64(D), f64(init), inp.seq_idx,
                   nseq=inp.nseq, nthreads=nthreads)
