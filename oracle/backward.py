"""Gradients of the SSD layer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; it shares no code with the HIP path.

The paper states the training cost of the layer (Section 6.3, Theorem on the
SSD algorithm's complexity) but gives no backward algorithm.  What is
computed here is the plain definition: the adjoint (reverse-mode
derivative) of the sequential recurrence of eq. s6 with scalar decay, per
(batch row, head h), group g = h div (H/G), A_h = -exp(A_log[h]),
a_t = exp(dt_t A_h):

    S_t = a_t S_{t-1} + dt_t x_t B_t^T,    y_t = S_t C_t + D_h x_t.

Given the output gradient dy (and optionally dfinal, the gradient of the
final state), walking t from the last token back, with G the gradient of
S_t (G starts at dfinal):

    G      += dy_t C_t^T
    dC_t   += S_t^T dy_t                      (summed over the group's heads)
    dx_t    = D_h dy_t + dt_t G B_t
    dB_t   += dt_t G^T x_t                    (summed over the group's heads)
    ddt_t   = x_t . (G B_t) + A_h a_t <G, S_{t-1}>
    dA_h   += dt_t a_t <G, S_{t-1}>
    dD_h   += dy_t . x_t
    G       = a_t G

and finally d(initial state) = G, dA_log = A_h dA_h.  Float64 throughout,
vectorised over batch rows and heads, one loop over tokens.

Packed rows (Section 8.3: one row holding several sequences, ``seq_idx``
naming each token's sequence; the state starts from that sequence's initial
state at its first token): the sequences do not interact, so the gradients
are those of each sequence as a problem of its own -- concatenated along the
tokens for dx, ddt, dB, dC, one initial-state gradient per sequence, and
dA_log, dD summed over the sequences.
"""
from __future__ import annotations

import numpy as np


def _forward_states(x, dt, A, B, C, D, init):
    """S_t for every token (b, T, H, P, N) and y (b, T, H, P)."""
    b, T, H, P = x.shape
    N = B.shape[-1]
    S = np.zeros((b, H, P, N)) if init is None else np.array(init, dtype=np.float64)
    states = np.empty((b, T, H, P, N))
    y = np.empty((b, T, H, P))
    for t in range(T):
        a = np.exp(dt[:, t] * A)                                   # (b, H)
        S = a[..., None, None] * S + (dt[:, t, :, None] * x[:, t])[..., None] * B[:, t][:, :, None, :]
        states[:, t] = S
        y[:, t] = np.einsum("bhpn,bhn->bhp", S, C[:, t]) + D[None, :, None] * x[:, t]
    return states, y


def backward(x, dt, A_log, B, C, dy, D=None, initial_states=None, dfinal=None, seq_idx=None):
    """Gradients of the layer.  x (b,T,H,P), dt (b,T,H), A_log (H), B/C
    (b,T,G,N), dy (b,T,H,P), D (H) or None, initial_states (b,H,P,N) or None,
    dfinal (b,H,P,N) or None.  Returns a dict with dx, ddt, dA_log, dB, dC,
    dD, dinit (float64; dD and dinit zero-filled when not used).

    With ``seq_idx`` (1, T) (packed rows, batch 1) initial_states, dfinal and
    dinit are (nseq, H, P, N)."""
    if seq_idx is not None:
        return _backward_packed(x, dt, A_log, B, C, dy, D, initial_states, dfinal, seq_idx)
    f = lambda a: None if a is None else np.asarray(a, dtype=np.float64)
    x, dt, A_log, B, C, dy, D, init, dfinal = map(f, (x, dt, A_log, B, C, dy, D, initial_states, dfinal))
    b, T, H, P = x.shape
    G_ = B.shape[2]
    hpg = H // G_
    grp = np.arange(H) // hpg
    Bh, Ch = B[:, :, grp], C[:, :, grp]                             # (b, T, H, N) per head
    A = -np.exp(A_log)
    Dv = np.zeros(H) if D is None else D
    states, _ = _forward_states(x, dt, A, Bh, Ch, Dv, init)
    S0 = np.zeros((b, H, P, B.shape[-1])) if init is None else init
    Gs = np.zeros_like(S0) if dfinal is None else dfinal.copy()
    dx = np.empty_like(x)
    ddt = np.empty_like(dt)
    dBh = np.zeros_like(Bh)
    dCh = np.zeros_like(Ch)
    dA = np.zeros(H)
    dD = np.zeros(H)
    for t in range(T - 1, -1, -1):
        a = np.exp(dt[:, t] * A)                                    # (b, H)
        Gs = Gs + dy[:, t][..., None] * Ch[:, t][:, :, None, :]
        dCh[:, t] = np.einsum("bhpn,bhp->bhn", states[:, t], dy[:, t])
        GB = np.einsum("bhpn,bhn->bhp", Gs, Bh[:, t])
        dx[:, t] = Dv[None, :, None] * dy[:, t] + dt[:, t, :, None] * GB
        dBh[:, t] = dt[:, t, :, None] * np.einsum("bhpn,bhp->bhn", Gs, x[:, t])
        prev = states[:, t - 1] if t > 0 else S0
        gs = np.einsum("bhpn,bhpn->bh", Gs, prev)
        ddt[:, t] = np.einsum("bhp,bhp->bh", x[:, t], GB) + A * a * gs
        dA += np.sum(dt[:, t] * a * gs, axis=0)
        dD += np.einsum("bhp,bhp->h", dy[:, t], x[:, t])
        Gs = a[..., None, None] * Gs
    dB = np.zeros_like(B)
    dC = np.zeros_like(C)
    for h in range(H):
        dB[:, :, grp[h]] += dBh[:, :, h]
        dC[:, :, grp[h]] += dCh[:, :, h]
    return {"dx": dx, "ddt": ddt, "dA_log": A * dA, "dB": dB, "dC": dC, "dD": dD, "dinit": Gs}


def _backward_packed(x, dt, A_log, B, C, dy, D, init, dfinal, seq_idx):
    """Packed rows: each sequence's gradients on its own (see the module text)."""
    seq = np.asarray(seq_idx).reshape(-1)
    if np.asarray(x).shape[0] != 1:
        raise ValueError("packed rows use batch 1")
    nseq = int(seq.max()) + 1
    bounds = np.flatnonzero(np.diff(seq)) + 1
    starts = np.concatenate([[0], bounds])
    ends = np.concatenate([bounds, [seq.size]])
    parts = []
    for s, (t0, t1) in enumerate(zip(starts, ends)):
        sl = slice(t0, t1)
        one = lambda a: None if a is None else np.asarray(a)[s:s + 1]
        parts.append(backward(np.asarray(x)[:, sl], np.asarray(dt)[:, sl], A_log, np.asarray(B)[:, sl],
                              np.asarray(C)[:, sl], np.asarray(dy)[:, sl], D=D, initial_states=one(init),
                              dfinal=one(dfinal)))
    assert len(parts) == nseq
    cat = lambda k: np.concatenate([q[k] for q in parts], axis=1)
    return {"dx": cat("dx"), "ddt": cat("ddt"), "dB": cat("dB"), "dC": cat("dC"),
            "dA_log": sum(q["dA_log"] for q in parts), "dD": sum(q["dD"] for q in parts),
            "dinit": np.concatenate([q["dinit"] for q in parts], axis=0)}
