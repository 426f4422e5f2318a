"""Gradients of the block steps around the SSD layer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; it shares no code with the HIP path.

The forward is :func:`oracle.block.block_forward`: dt parameterisation, the
layer, the SiLU gate (Section 8.1), the grouped RMS normalisation (Section
7.1).  The paper gives no backward; what is computed here is the chain rule
through each step, in reverse order, float64 throughout:

* normalisation, per token and group of ``G`` channels, with ``g`` the gated
  output, ``r = sqrt(mean(g^2) + eps)``, ``n = g / r``, ``out = n w``:
  ``dn = dout w``, ``dg = (dn - n mean(dn n)) / r``, ``dw = sum over tokens
  of dout n``;
* gate ``g = y SiLU(z)``: ``dy = dg SiLU(z)``, ``dz = dg y SiLU'(z)`` with
  ``SiLU'(z) = s (1 + z (1 - s))``, ``s`` the logistic sigmoid;
* the layer: :func:`oracle.backward.backward` (its adjoint) with that ``dy``;
* dt step ``dt = clamp(softplus(dt_raw + bias), lo, hi)``: ``d dt_raw = ddt
  [lo < softplus(.) < hi] sigmoid(dt_raw + bias)`` (the factor 1 without
  softplus), ``d bias = sum over tokens of d dt_raw``.
"""
from __future__ import annotations

import numpy as np

import oracle as _oracle
import oracle.backward as _bwd
import oracle.block as _blk


def sigmoid(v):
    v = np.asarray(v, dtype=np.float64)
    e = np.exp(-np.abs(v))
    return np.where(v >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def block_backward(x, dt_raw, A_log, B, C, dout, D=None, initial_states=None, dfinal=None,
                   dt_bias=None, dt_softplus=True, dt_lo=0.0, dt_hi=np.inf, z=None,
                   norm_weight=None, norm_group_size=0, norm_eps=1e-5):
    """Gradients of the block (no packed rows).  Shapes as for
    :func:`oracle.block.block_forward`; ``dout`` (b, T, H, P), ``dfinal``
    (b, H, P, N) or None.  Returns a dict with the layer's gradients (``dx``,
    ``ddt`` is replaced by ``ddt_raw``, ``dA_log``, ``dB``, ``dC``, ``dD``,
    ``dinit``) and ``ddt_bias`` (or None), ``dz`` (or None), ``dnorm_weight``
    (or None).  Float64 throughout, from the given (possibly bf16-valued)
    inputs: nothing in between is rounded."""
    f = lambda a: None if a is None else np.asarray(a, dtype=np.float64)
    x, dt_raw, A_log, B, C, dout, D, init, dfinal = map(f, (x, dt_raw, A_log, B, C, dout, D,
                                                           initial_states, dfinal))
    z, w, bias = f(z), f(norm_weight), f(dt_bias)
    b, T, H, P = x.shape

    # forward, keeping what the backward needs
    v = dt_raw + (bias if bias is not None else 0.0)
    sp = _blk.softplus(v) if dt_softplus else v
    dt = np.minimum(np.maximum(sp, dt_lo), dt_hi)
    y, _ = _oracle.forward(x, dt, A_log, B, C, D, init)
    g = y * _blk.silu(z) if z is not None else y

    # normalisation
    if norm_group_size > 0:
        Cn = H * P
        G = norm_group_size
        rows = g.reshape(b, T, Cn // G, G)
        r = np.sqrt(np.mean(rows * rows, axis=-1, keepdims=True) + norm_eps)
        n = rows / r
        do = dout.reshape(b, T, Cn // G, G)
        wv = w.reshape(Cn // G, G) if w is not None else np.ones((Cn // G, G))
        dn = do * wv
        dg = (dn - n * np.mean(dn * n, axis=-1, keepdims=True)) / r
        dg = dg.reshape(b, T, H, P)
        dw = np.sum(do * n, axis=(0, 1)).reshape(Cn) if w is not None else None
    else:
        dg = dout
        dw = None

    # gate
    if z is not None:
        s = sigmoid(z)
        dy = dg * (z * s)
        dz = dg * y * (s * (1.0 + z * (1.0 - s)))
    else:
        dy = dg
        dz = None

    # the layer
    gr = _bwd.backward(x, dt, A_log, B, C, dy, D=D, initial_states=init, dfinal=dfinal)

    # dt step
    mask = (sp > dt_lo) & (sp < dt_hi)
    dv = gr["ddt"] * mask * (sigmoid(v) if dt_softplus else 1.0)
    out = {k: gr[k] for k in ("dx", "dA_log", "dB", "dC", "dD", "dinit")}
    out["ddt_raw"] = dv
    out["ddt_bias"] = np.sum(dv, axis=(0, 1)) if bias is not None else None
    out["dz"] = dz
    out["dnorm_weight"] = dw
    return out
