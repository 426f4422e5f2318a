"""Mamba-2 block steps on either side of the SSD layer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; it shares no code with the HIP path.

What is computed (float64 throughout, from the exact values of the rounded
inputs):

* **dt parameterisation** (step 0, before the layer).  The paper leaves the
  discretisation parameter to the caller (Section 2 defines the SSM on already
  discrete ``A``; Section 7 only says that ``Delta`` comes out of the block's
  input projection).  Reading used here: ``dt = clamp(softplus(dt_raw +
  dt_bias), lo, hi)`` with a per-head bias, ``softplus(v) = log(1 + e^v)``.
* **gate** (Section 8.1, the tensor-parallel block equations):
  ``y_g = y * phi(z)`` with ``phi`` the SiLU, ``phi(z) = z / (1 + e^-z)``.
* **grouped RMS normalisation** (Section 7.1: an extra normalisation right
  before the output projection, placed after the multiplicative gate;
  Section 8.1: a group norm whose number of groups the tensor-parallel degree
  divides).  Reading used here: RMSNorm per token over contiguous groups of
  ``group_size`` channels of the ``H * P`` channel row,
  ``y_n[c] = y_g[c] / sqrt(mean_{c' in group(c)} y_g[c']^2 + eps) * w[c]``.

``block_forward`` runs them around :func:`oracle.forward`.
"""
from __future__ import annotations

import numpy as np

import oracle as _oracle


def softplus(v):
    """``log(1 + e^v)`` written so that neither branch overflows:
    ``max(v, 0) + log(1 + e^{-|v|})``."""
    v = np.asarray(v, dtype=np.float64)
    return np.maximum(v, 0.0) + np.log1p(np.exp(-np.abs(v)))


def dt_transform(dt_raw, dt_bias, lo=0.0, hi=np.inf, apply_softplus=True):
    """dt of every (token, head): softplus of the raw value plus the head's
    bias (when ``apply_softplus``), then clamped to ``[lo, hi]``.
    ``dt_raw`` (..., H), ``dt_bias`` (H,) or None."""
    v = np.asarray(dt_raw, dtype=np.float64)
    if dt_bias is not None:
        v = v + np.asarray(dt_bias, dtype=np.float64)
    if apply_softplus:
        v = softplus(v)
    return np.minimum(np.maximum(v, lo), hi)


def silu(z):
    """SiLU (the gate nonlinearity of Section 8.1): z * sigmoid(z)."""
    z = np.asarray(z, dtype=np.float64)
    # sigmoid from e^{-|z|} on both sides, so no exponential overflows
    e = np.exp(-np.abs(z))
    sig = np.where(z >= 0, 1.0 / (1.0 + e), e / (1.0 + e))
    return z * sig


def gate(y, z):
    """Multiplicative gate branch: y * SiLU(z), elementwise."""
    return np.asarray(y, dtype=np.float64) * silu(z)


def group_rmsnorm(y, weight, group_size, eps):
    """RMS normalisation of each token's channel row in groups of
    ``group_size`` consecutive channels, then the per-channel weight.

    ``y`` (..., H, P): the channel row of a token is its ``H * P`` values in
    (head, feature) order.  ``weight`` (H * P,) or None (= 1)."""
    y = np.asarray(y, dtype=np.float64)
    lead, H, P = y.shape[:-2], y.shape[-2], y.shape[-1]
    C = H * P
    if group_size <= 0 or C % group_size:
        raise ValueError("group_size must divide the channel count")
    rows = y.reshape(lead + (C // group_size, group_size))
    ms = np.mean(rows * rows, axis=-1, keepdims=True)
    out = (rows / np.sqrt(ms + eps)).reshape(lead + (C,))
    if weight is not None:
        out = out * np.asarray(weight, dtype=np.float64)
    return out.reshape(y.shape)


def block_forward(x, dt_raw, A_log, B, C, D=None, initial_states=None, seq_idx=None, nseq=None,
                  dt_bias=None, dt_softplus=True, dt_lo=0.0, dt_hi=np.inf, z=None,
                  norm_weight=None, norm_group_size=0, norm_eps=1e-5, nthreads=None, lib=None):
    """dt parameterisation -> SSD layer (:func:`oracle.forward`) -> gate ->
    grouped RMS normalisation, each step only when asked for (``z`` given,
    ``norm_group_size > 0``).  Returns ``(out (b,T,H,P), final_states)`` in
    float64."""
    dt = dt_transform(dt_raw, dt_bias, dt_lo, dt_hi, dt_softplus)
    y, fin = _oracle.forward(x, dt, A_log, B, C, D, initial_states, seq_idx, nseq=nseq,
                             nthreads=nthreads, lib=lib)
    if z is not None:
        y = gate(y, z)
    if norm_group_size > 0:
        y = group_rmsnorm(y, norm_weight, norm_group_size, norm_eps)
    return y, fin


def block_forward_inputs(inp, opts, nthreads=None):
    """:func:`block_forward` on :class:`paper_2405_21060_amd.inputs.BlockInputs`
    with a dict of options (``dt_softplus``, ``dt_lo``, ``dt_hi``, ``gate``,
    ``norm_group_size``, ``norm_eps``)."""
    base = inp.base
    f64 = base.as_f64
    z = inp.as_f64("z") if opts.get("gate", True) else None
    return block_forward(
        f64("x"), inp.as_f64("dt_raw"), base.A_log, f64("B"), f64("C"), base.D,
        base.initial_states, base.seq_idx, nseq=base.nseq,
        dt_bias=inp.dt_bias if opts.get("dt_bias", True) else None,
        dt_softplus=opts.get("dt_softplus", True), dt_lo=opts.get("dt_lo", 0.0),
        dt_hi=opts.get("dt_hi", np.inf), z=z,
        norm_weight=inp.norm_weight if opts.get("norm_weight", True) else None,
        norm_group_size=opts.get("norm_group_size", 0), norm_eps=opts.get("norm_eps", 1e-5),
        nthreads=nthreads)
