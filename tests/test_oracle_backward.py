"""Pins of the backward oracle (oracle/backward.py) -- CPU only.

Every gradient is checked against central finite differences of the C
oracle of the forward (an independent implementation), for the scalar loss
L = <W, y> + <V, final_state> with random W and V, so dy = W and dfinal = V.
Planted mistakes in copies of the module must each fail the check.
"""
import os
import types

import numpy as np
import pytest

import oracle
import oracle.backward as ob

SRC = os.path.join(os.path.dirname(ob.__file__), "backward.py")


def _problem(seed=3, b=2, T=7, H=4, P=3, N=5, G=2):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((b, T, H, P))
    dt = rng.uniform(0.05, 0.6, (b, T, H))
    A_log = rng.uniform(-0.5, 1.0, H)
    B = rng.standard_normal((b, T, G, N)) / np.sqrt(N)
    C = rng.standard_normal((b, T, G, N)) / np.sqrt(N)
    D = rng.standard_normal(H)
    init = rng.standard_normal((b, H, P, N))
    W = rng.standard_normal((b, T, H, P))
    V = rng.standard_normal((b, H, P, N))
    return dict(x=x, dt=dt, A_log=A_log, B=B, C=C, D=D, init=init), W, V


def _loss(inp, W, V):
    y, fin = oracle.forward(inp["x"], inp["dt"], inp["A_log"], inp["B"], inp["C"], inp["D"],
                            initial_states=inp["init"])
    return float(np.sum(W * y) + np.sum(V * fin))


NAMES = {"x": "dx", "dt": "ddt", "A_log": "dA_log", "B": "dB", "C": "dC", "D": "dD", "init": "dinit"}


def finite_difference_ok(m, seed=3, samples=6, h=1e-6, rtol=1e-6):
    inp, W, V = _problem(seed)
    g = m.backward(inp["x"], inp["dt"], inp["A_log"], inp["B"], inp["C"], W, D=inp["D"],
                   initial_states=inp["init"], dfinal=V)
    rng = np.random.default_rng(seed + 100)
    for name, gname in NAMES.items():
        arr = inp[name]
        for _ in range(samples):
            idx = tuple(rng.integers(0, s) for s in arr.shape)
            old = arr[idx]
            arr[idx] = old + h
            lp = _loss(inp, W, V)
            arr[idx] = old - h
            lm = _loss(inp, W, V)
            arr[idx] = old
            fd = (lp - lm) / (2 * h)
            got = g[gname][idx]
            if abs(got - fd) > rtol * max(1.0, abs(fd)) * 10:
                return False
    return True


@pytest.mark.parametrize("seed", [3, 4])
def test_backward_matches_finite_differences(seed):
    assert finite_difference_ok(ob, seed=seed)


def test_backward_without_optional_inputs():
    # no D, no initial state, no final-state gradient: the zero limits of the general case
    inp, W, V = _problem(5)
    g0 = ob.backward(inp["x"], inp["dt"], inp["A_log"], inp["B"], inp["C"], W)
    zero_init = np.zeros_like(inp["init"])
    g1 = ob.backward(inp["x"], inp["dt"], inp["A_log"], inp["B"], inp["C"], W, D=np.zeros(4),
                     initial_states=zero_init, dfinal=np.zeros_like(V))
    for k in ("dx", "ddt", "dA_log", "dB", "dC", "dinit"):
        assert np.allclose(g0[k], g1[k], rtol=1e-13, atol=1e-15), k


MUTANTS = {
    "ddt_without_decay_term": ("ddt[:, t] = np.einsum(\"bhp,bhp->bh\", x[:, t], GB) + A * a * gs",
                               "ddt[:, t] = np.einsum(\"bhp,bhp->bh\", x[:, t], GB)"),
    "dC_from_previous_state": ("dCh[:, t] = np.einsum(\"bhpn,bhp->bhn\", states[:, t], dy[:, t])",
                               "dCh[:, t] = np.einsum(\"bhpn,bhp->bhn\", states[:, t - 1] if t > 0 else S0, dy[:, t])"),
    "dB_without_dt": ("dBh[:, t] = dt[:, t, :, None] * np.einsum(", "dBh[:, t] = np.einsum("),
    "decay_before_output_term": ("        Gs = Gs + dy[:, t][..., None] * Ch[:, t][:, :, None, :]\n",
                                 "        Gs = a[..., None, None] * Gs + dy[:, t][..., None] * Ch[:, t][:, :, None, :]\n"),
    "dA_without_dt": ("dA += np.sum(dt[:, t] * a * gs, axis=0)", "dA += np.sum(a * gs, axis=0)"),
    "dA_log_sign": ("\"dA_log\": A * dA", "\"dA_log\": -A * dA"),
    "dx_without_skip": ("dx[:, t] = Dv[None, :, None] * dy[:, t] + dt[:, t, :, None] * GB",
                        "dx[:, t] = dt[:, t, :, None] * GB"),
}


def _mutant(name):
    a, b = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(a) == 1, name
    mod = types.ModuleType("oracle_backward_" + name)
    exec(compile(src.replace(a, b), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_backward_mutant_is_caught(name):
    assert not finite_difference_ok(_mutant(name))


def _packed_problem(seed=7, T=11, H=3, P=2, N=4, G=1):
    rng = np.random.default_rng(seed)
    seq_idx = np.array([[0] * 3 + [1] * 1 + [2] * 5 + [3] * 2], dtype=np.int32)   # lengths 3, 1, 5, 2
    nseq = 4
    inp = dict(x=rng.standard_normal((1, T, H, P)), dt=rng.uniform(0.05, 0.6, (1, T, H)),
               A_log=rng.uniform(-0.5, 1.0, H), B=rng.standard_normal((1, T, G, N)) / 2,
               C=rng.standard_normal((1, T, G, N)) / 2, D=rng.standard_normal(H),
               init=rng.standard_normal((nseq, H, P, N)))
    W = rng.standard_normal((1, T, H, P))
    V = rng.standard_normal((nseq, H, P, N))
    return inp, seq_idx, nseq, W, V


def packed_finite_difference_ok(m, samples=6, h=1e-6):
    inp, seq_idx, nseq, W, V = _packed_problem()
    g = m.backward(inp["x"], inp["dt"], inp["A_log"], inp["B"], inp["C"], W, D=inp["D"],
                   initial_states=inp["init"], dfinal=V, seq_idx=seq_idx)

    def loss():
        y, fin = oracle.forward(inp["x"], inp["dt"], inp["A_log"], inp["B"], inp["C"], inp["D"],
                                initial_states=inp["init"], seq_idx=seq_idx, nseq=nseq)
        return float(np.sum(W * y) + np.sum(V * fin))

    rng = np.random.default_rng(8)
    for name, gname in NAMES.items():
        arr = inp[name]
        for _ in range(samples):
            idx = tuple(rng.integers(0, s) for s in arr.shape)
            old = arr[idx]
            arr[idx] = old + h
            lp = loss()
            arr[idx] = old - h
            lm = loss()
            arr[idx] = old
            fd = (lp - lm) / (2 * h)
            if abs(g[gname][idx] - fd) > 1e-5 * max(1.0, abs(fd)):
                return False
    return True


def test_packed_rows_match_finite_differences():
    # the C oracle's forward resets the state token by token at each boundary
    assert packed_finite_difference_ok(ob)


def test_packed_rows_planted_mistake_is_caught():
    # a packed gradient that lets the carried state gradient cross a boundary
    src = open(SRC).read()
    a = "one = lambda a: None if a is None else np.asarray(a)[s:s + 1]"
    assert src.count(a) == 1
    bad = src.replace("    for s, (t0, t1) in enumerate(zip(starts, ends)):",
                      "    starts, ends = np.array([0]), np.array([seq.size])\n"
                      "    for s, (t0, t1) in enumerate(zip(starts, ends)):")
    bad = bad.replace("    assert len(parts) == nseq\n", "")
    mod = types.ModuleType("oracle_backward_packed_mutant")
    exec(compile(bad, SRC, "exec"), mod.__dict__)
    try:
        ok = packed_finite_difference_ok(mod)
    except Exception:
        ok = False
    assert not ok
