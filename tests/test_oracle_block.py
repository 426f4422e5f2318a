"""Pins of the block-step oracle (oracle/block.py) -- CPU only.

Each pin ties a function to something other than itself: a library routine
(numpy's logaddexp, scipy's expit), an identity of the function, an
invariant, brute force on a tiny input, or a limit in which the result has a
closed form.  The mutant test plants plausible mistakes in copies of the
module's source and checks that every one of them fails at least one pin.
"""
import math
import os
import types

import numpy as np
import pytest
from scipy.special import expit

import oracle
import oracle.block as ob
from paper_2405_21060_amd.inputs import Problem, make_block_inputs

SRC = os.path.join(os.path.dirname(ob.__file__), "block.py")


def _tiny(seed=5, T=24, H=4, P=4, N=4, G=2):
    p = Problem(2, T, H, P, N, G, 8, "f32")
    return make_block_inputs(p, seed)


# ---- pins: each takes a module-like object m and returns True when it holds

def pin_softplus_logaddexp(m):
    v = np.linspace(-60.0, 60.0, 2401)
    return np.allclose(m.softplus(v), np.logaddexp(0.0, v), rtol=1e-13, atol=1e-300)


def pin_softplus_identity(m):
    # log(1+e^v) - log(1+e^-v) = v
    v = np.linspace(-30.0, 30.0, 601)
    return np.allclose(m.softplus(v) - m.softplus(-v), v, rtol=0, atol=1e-12)


def pin_silu_expit(m):
    z = np.linspace(-50.0, 50.0, 1001)
    return np.allclose(m.silu(z), z * expit(z), rtol=1e-13, atol=1e-300)


def pin_gate_limits(m):
    rng = np.random.default_rng(1)
    y = rng.standard_normal((3, 5))
    # SiLU(0) = 0; SiLU(z) -> z for large z
    return (np.all(m.gate(y, np.zeros_like(y)) == 0.0)
            and np.allclose(m.gate(y, np.full_like(y, 40.0)), 40.0 * y, rtol=1e-12, atol=0))


def pin_rmsnorm_brute_force(m):
    rng = np.random.default_rng(2)
    lead, H, P, gs, eps = (2, 3), 4, 3, 6, 0.25
    y = rng.standard_normal(lead + (H, P))
    w = 1.0 + 0.5 * rng.standard_normal(H * P)
    out = m.group_rmsnorm(y, w, gs, eps)
    ok = True
    for i in range(lead[0]):
        for j in range(lead[1]):
            row = [y[i, j, h, q] for h in range(H) for q in range(P)]
            for g0 in range(0, H * P, gs):
                ms = sum(row[c] * row[c] for c in range(g0, g0 + gs)) / gs
                for c in range(g0, g0 + gs):
                    ref = row[c] / math.sqrt(ms + eps) * w[c]
                    ok &= abs(out[i, j, c // P, c % P] - ref) <= 1e-12 * max(1.0, abs(ref))
    return bool(ok)


def pin_rmsnorm_unit_rms(m):
    rng = np.random.default_rng(3)
    y = rng.standard_normal((7, 8, 4))
    out = m.group_rmsnorm(y, None, 8, 0.0).reshape(7, 4, 8)
    return np.allclose(np.mean(out * out, axis=-1), 1.0, rtol=1e-12, atol=0)


def pin_rmsnorm_scale_invariant(m):
    rng = np.random.default_rng(4)
    y = rng.standard_normal((5, 6, 4))
    w = rng.standard_normal(24)
    return np.allclose(m.group_rmsnorm(3.5 * y, w, 12, 0.0), m.group_rmsnorm(y, w, 12, 0.0),
                       rtol=1e-12, atol=1e-14)


def pin_dt_transform_library(m):
    rng = np.random.default_rng(6)
    raw = rng.standard_normal((3, 9, 4)) * 4
    bias = rng.standard_normal(4)
    got = m.dt_transform(raw, bias, 0.05, 2.0)
    ref = np.clip(np.logaddexp(0.0, raw + bias), 0.05, 2.0)
    return np.allclose(got, ref, rtol=1e-13, atol=0)


def pin_block_plain_is_layer(m):
    bi = _tiny()
    b = bi.base
    f = b.as_f64
    dt = f("dt")
    y, fin = m.block_forward(f("x"), dt, b.A_log, f("B"), f("C"), b.D, dt_softplus=False)
    y0, fin0 = oracle.forward(f("x"), dt, b.A_log, f("B"), f("C"), b.D)
    return np.array_equal(y, y0) and np.array_equal(fin, fin0)


def pin_block_constant_dt(m):
    # lo == hi pins every dt to that value whatever the raw input and bias
    bi = _tiny()
    b = bi.base
    f = b.as_f64
    y, _ = m.block_forward(f("x"), bi.as_f64("dt_raw"), b.A_log, f("B"), f("C"), b.D,
                           dt_bias=bi.dt_bias, dt_lo=0.3, dt_hi=0.3)
    y0, _ = oracle.forward(f("x"), np.full(bi.dt_raw.shape, 0.3), b.A_log, f("B"), f("C"), b.D)
    return np.allclose(y, y0, rtol=1e-13, atol=1e-13)


def pin_block_gate_multiplies_output(m):
    # z = 40 everywhere: SiLU(z) = 40 (to 1e-16), so the gated block is 40 x the layer
    bi = _tiny()
    b = bi.base
    f = b.as_f64
    args = (f("x"), bi.as_f64("dt_raw"), b.A_log, f("B"), f("C"), b.D)
    y, _ = m.block_forward(*args, dt_bias=bi.dt_bias, z=np.full(b.x.shape, 40.0))
    y0, _ = m.block_forward(*args, dt_bias=bi.dt_bias)
    return np.allclose(y, 40.0 * y0, rtol=1e-12, atol=1e-12)


def pin_block_norm_is_last(m):
    # with unit weight and eps = 0 every normalisation group of the block's
    # output has mean square 1, which holds only if the norm is the last step
    bi = _tiny()
    b = bi.base
    f = b.as_f64
    y, _ = m.block_forward(f("x"), bi.as_f64("dt_raw"), b.A_log, f("B"), f("C"), b.D,
                           dt_bias=bi.dt_bias, z=bi.as_f64("z"), norm_group_size=8, norm_eps=0.0)
    g = y.reshape(y.shape[0], y.shape[1], -1, 8)
    return np.allclose(np.mean(g * g, axis=-1), 1.0, rtol=1e-10, atol=0)


def pin_block_gate_on_output(m):
    # the gate multiplies the layer's output, not its input: with the layer
    # linear in x, gating x by a constant c would give c * y as well, so use a
    # z that varies over tokens and compare against the gate of the layer output
    bi = _tiny()
    b = bi.base
    f = b.as_f64
    z = bi.as_f64("z")
    args = (f("x"), bi.as_f64("dt_raw"), b.A_log, f("B"), f("C"), b.D)
    y, _ = m.block_forward(*args, dt_bias=bi.dt_bias, z=z)
    y0, _ = m.block_forward(*args, dt_bias=bi.dt_bias)
    return np.allclose(y, y0 * z * expit(z), rtol=1e-12, atol=1e-12)


PINS = [pin_softplus_logaddexp, pin_softplus_identity, pin_silu_expit, pin_gate_limits,
        pin_rmsnorm_brute_force, pin_rmsnorm_unit_rms, pin_rmsnorm_scale_invariant,
        pin_dt_transform_library, pin_block_plain_is_layer, pin_block_constant_dt,
        pin_block_gate_multiplies_output, pin_block_norm_is_last, pin_block_gate_on_output]


@pytest.mark.parametrize("pin", PINS, ids=[f.__name__ for f in PINS])
def test_block_oracle_pin(pin):
    assert pin(ob)


# ---- mutants: plausible mistakes planted in copies of oracle/block.py

MUTANTS = {
    "softplus_without_log_term": ("np.maximum(v, 0.0) + np.log1p(np.exp(-np.abs(v)))",
                                  "np.maximum(v, 0.0)"),
    "softplus_wrong_sign": ("np.log1p(np.exp(-np.abs(v)))", "np.log1p(np.exp(np.abs(v)))"),
    "bias_dropped": ("        v = v + np.asarray(dt_bias, dtype=np.float64)", "        v = v"),
    "clamp_before_softplus": ("    if apply_softplus:\n        v = softplus(v)\n    return np.minimum(np.maximum(v, lo), hi)",
                              "    v = np.minimum(np.maximum(v, lo), hi)\n    if apply_softplus:\n        v = softplus(v)\n    return v"),
    "silu_is_sigmoid": ("    return z * sig", "    return sig"),
    "norm_over_tokens": ("    ms = np.mean(rows * rows, axis=-1, keepdims=True)",
                         "    ms = np.mean(rows * rows, axis=0, keepdims=True)"),
    "norm_sum_not_mean": ("    ms = np.mean(rows * rows, axis=-1, keepdims=True)",
                          "    ms = np.sum(rows * rows, axis=-1, keepdims=True)"),
    "eps_outside_sqrt": ("rows / np.sqrt(ms + eps)", "rows / (np.sqrt(ms) + eps)"),
    "weight_before_norm": ("    out = (rows / np.sqrt(ms + eps)).reshape(lead + (C,))\n    if weight is not None:\n        out = out * np.asarray(weight, dtype=np.float64)",
                           "    out = rows.reshape(lead + (C,))\n    if weight is not None:\n        out = out * np.asarray(weight, dtype=np.float64)\n    r2 = out.reshape(rows.shape)\n    out = (r2 / np.sqrt(np.mean(r2 * r2, axis=-1, keepdims=True) + eps)).reshape(lead + (C,))"),
    "norm_before_gate": ("    if z is not None:\n        y = gate(y, z)\n    if norm_group_size > 0:\n        y = group_rmsnorm(y, norm_weight, norm_group_size, norm_eps)",
                         "    if norm_group_size > 0:\n        y = group_rmsnorm(y, norm_weight, norm_group_size, norm_eps)\n    if z is not None:\n        y = gate(y, z)"),
    "gate_on_input": ("    dt = dt_transform(dt_raw, dt_bias, dt_lo, dt_hi, dt_softplus)\n",
                      "    dt = dt_transform(dt_raw, dt_bias, dt_lo, dt_hi, dt_softplus)\n    if z is not None:\n        x = gate(x, z)\n        z = None\n"),
}


def _mutant(name):
    a, b = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(a) == 1, name
    mod = types.ModuleType("oracle_block_" + name)
    mod.__dict__["__file__"] = SRC
    exec(compile(src.replace(a, b), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_block_mutant_is_caught(name):
    m = _mutant(name)
    failed = []
    for pin in PINS:
        try:
            ok = pin(m)
        except Exception:
            ok = False
        if not ok:
            failed.append(pin.__name__)
    assert failed, "mutant %s passes every pin" % name
