"""Pins of the span (context-parallel) oracle, oracle/span.py -- CPU only.

The pins tie it to the C oracle of the whole layer (an independent
implementation: linearity in the initial state, and the split-and-combine
identity of Section 8.2), to the associativity of the scan operator
(Appendix B) and to the multiplicativity of decays; planted mutants must each
fail one of them.
"""
import os
import types

import numpy as np
import pytest

import oracle
import oracle.span as osp
from paper_2405_21060_amd.inputs import Problem, make_inputs

SRC = os.path.join(os.path.dirname(osp.__file__), "span.py")


def _inp(seed=7, T=40, H=4, P=4, N=4, G=2):
    return make_inputs(Problem(2, T, H, P, N, G, 8, "f32", init_states=True), seed)


def pin_correction_is_initial_state_response(m):
    # y(h_in) - y(0) over one span: the layer is linear in its initial state
    inp = _inp()
    f = inp.as_f64
    args = (f("x"), f("dt"), inp.A_log, f("B"), f("C"), inp.D)
    y1, _ = oracle.forward(*args, initial_states=inp.initial_states)
    y0, _ = oracle.forward(*args)
    corr = m.span_correction(f("dt"), inp.A_log, f("C"), inp.initial_states)
    return np.allclose(corr, y1 - y0, rtol=1e-10, atol=1e-12)


def pin_split_and_combine(m):
    # spans from zero states, combined, corrected: the whole sequence's outputs,
    # entering states and final state (Section 8.2)
    inp = _inp(T=45)
    f = inp.as_f64
    x, dt, B, C = f("x"), f("dt"), f("B"), f("C")
    cuts = [0, 11, 12, 30, 45]
    ys, fins, decs = [], [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        y, fin = oracle.forward(x[:, a:b], dt[:, a:b], inp.A_log, B[:, a:b], C[:, a:b], inp.D)
        ys.append(y)
        fins.append(fin)
        decs.append(m.span_decay(dt[:, a:b], inp.A_log))
    entering, final = m.combine_spans(np.stack(decs), np.stack(fins), inp.initial_states)
    y_full, fin_full = oracle.forward(x, dt, inp.A_log, B, C, inp.D, initial_states=inp.initial_states)
    ok = np.allclose(final, fin_full, rtol=1e-10, atol=1e-12)
    for r, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
        _, fin_prefix = oracle.forward(x[:, :a], dt[:, :a], inp.A_log, B[:, :a], C[:, :a], inp.D,
                                       initial_states=inp.initial_states) if a else (None, inp.initial_states)
        ok &= np.allclose(entering[r], fin_prefix, rtol=1e-10, atol=1e-12)
        yc = ys[r] + m.span_correction(dt[:, a:b], inp.A_log, C[:, a:b], entering[r])
        ok &= np.allclose(yc, y_full[:, a:b], rtol=1e-10, atol=1e-12)
    return bool(ok)


def pin_decay_multiplicative(m):
    inp = _inp()
    dt = inp.as_f64("dt")
    whole = m.span_decay(dt, inp.A_log)
    parts = m.span_decay(dt[:, :13], inp.A_log) * m.span_decay(dt[:, 13:], inp.A_log)
    const = m.span_decay(np.full((1, 10, 4), 0.25), np.log([1.0, 2.0, 3.0, 4.0]))
    return (np.allclose(whole, parts, rtol=1e-12, atol=0)
            and np.allclose(const, np.exp(-2.5 * np.array([[1.0, 2.0, 3.0, 4.0]])), rtol=1e-12, atol=0))


def pin_operator_associative(m):
    rng = np.random.default_rng(3)
    pairs = [(rng.uniform(0.1, 1, (2, 3)), rng.standard_normal((2, 3, 4, 5))) for _ in range(3)]
    l1 = m.combine(m.combine(pairs[0], pairs[1]), pairs[2])
    l2 = m.combine(pairs[0], m.combine(pairs[1], pairs[2]))
    return np.allclose(l1[0], l2[0], rtol=1e-13) and np.allclose(l1[1], l2[1], rtol=1e-12, atol=1e-13)


PINS = [pin_correction_is_initial_state_response, pin_split_and_combine, pin_decay_multiplicative,
        pin_operator_associative]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_span_oracle_pin(pin):
    assert pin(osp)


MUTANTS = {
    "exclusive_decay": ("decay = np.exp(np.cumsum(dt, axis=1) * A)",
                        "decay = np.exp((np.cumsum(dt, axis=1) - dt) * A)"),
    "operator_swapped": ("return a * a2, a2[..., None, None] * h + h2",
                         "return a * a2, a[..., None, None] * h2 + h"),
    "decay_without_A": ("return np.exp(dt.sum(axis=1) * A)", "return np.exp(-dt.sum(axis=1))"),
    "inclusive_scan": ("        entering.append(acc[1])\n        acc = combine(acc, (decays[r], local_finals[r]))",
                       "        acc = combine(acc, (decays[r], local_finals[r]))\n        entering.append(acc[1])"),
    "interleaved_groups": ("Cg = C[:, :, np.arange(H) // hpg, :]", "Cg = C[:, :, np.arange(H) % G, :]"),
}


def _mutant(name):
    a, b = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(a) == 1, name
    mod = types.ModuleType("oracle_span_" + name)
    exec(compile(src.replace(a, b), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_span_mutant_is_caught(name):
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
