"""Sequence split into spans (context parallelism) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; it shares no code with the HIP path.

Section 8.2 passes the state between consecutive pieces of a sequence: each
piece runs the layer from a zero state, giving its outputs and its final
state; the state entering each piece then follows from the pieces before it
by the scalar-SSM scan of Appendix B, under the associative operator
``(a, h) * (a', h') = (a a', a' h + h')`` on pairs of (total decay, state);
finally each piece adds the output its entering state produces,
``y_t += exp(A_h sum_{s <= t} dt_s) (h_in C_t)``, the sum running from the
piece's first token, and its final state becomes ``exp(A_h sum dt) h_in +
h_local``.

Float64 throughout, from the exact values of the rounded inputs.
"""
from __future__ import annotations

import numpy as np


def span_decay(dt, A_log):
    """Total decay of a span per (batch, head): ``exp(A_h sum_t dt_t)`` with
    ``A_h = -exp(A_log[h])``.  ``dt`` (b, T, H)."""
    dt = np.asarray(dt, dtype=np.float64)
    A = -np.exp(np.asarray(A_log, dtype=np.float64))
    return np.exp(dt.sum(axis=1) * A)


def combine(left, right):
    """The scan operator on (decay, state) pairs: ``left`` then ``right``.
    decay (b, H), state (b, H, P, N)."""
    a, h = left
    a2, h2 = right
    return a * a2, a2[..., None, None] * h + h2


def combine_spans(decays, local_finals, initial=None):
    """Exclusive scan over spans: the state entering every span, and the final
    state after the last one.  ``decays`` (R, b, H); ``local_finals``
    (R, b, H, P, N) (each span from a zero state); ``initial`` (b, H, P, N)
    or None (zero)."""
    decays = np.asarray(decays, dtype=np.float64)
    local_finals = np.asarray(local_finals, dtype=np.float64)
    acc = (np.ones_like(decays[0]),
           np.zeros_like(local_finals[0]) if initial is None else np.asarray(initial, dtype=np.float64))
    entering = []
    for r in range(len(decays)):
        entering.append(acc[1])
        acc = combine(acc, (decays[r], local_finals[r]))
    return np.stack(entering), acc[1]


def span_correction(dt, A_log, C, entering, heads_per_group=None):
    """Output of a span due to its entering state alone:
    ``exp(A_h sum_{s<=t} dt_s) * (h_in[h] @ C_t[g])`` for every token, with
    ``g = h div (H/G)``.  dt (b, T, H); C (b, T, G, N); entering (b, H, P, N).
    Returns (b, T, H, P)."""
    dt = np.asarray(dt, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    E = np.asarray(entering, dtype=np.float64)
    b, T, H = dt.shape
    G = C.shape[2]
    hpg = H // G if heads_per_group is None else heads_per_group
    A = -np.exp(np.asarray(A_log, dtype=np.float64))
    decay = np.exp(np.cumsum(dt, axis=1) * A)                  # (b, T, H), inclusive
    Cg = C[:, :, np.arange(H) // hpg, :]                        # (b, T, H, N)
    out = np.einsum("bhpn,bthn->bthp", E, Cg)
    return out * decay[..., None]
