"""Pins of the block-backward oracle (oracle/block_backward.py) -- CPU only.

Every gradient is checked against central finite differences of the block
forward oracle (oracle/block.py around the C oracle of the layer: an
independent implementation), for the loss L = <W, out> + <V, final_state>.
Planted mistakes in copies of the module must each fail the check.
"""
import os
import types

import numpy as np
import pytest

import oracle.block as ob
import oracle.block_backward as obb

SRC = os.path.join(os.path.dirname(obb.__file__), "block_backward.py")


def _problem(seed, gate=True, group=6, weight=True, bias=True, softplus=True, lo=0.0, hi=np.inf):
    rng = np.random.default_rng(seed)
    b, T, H, P, N, G = 2, 7, 4, 3, 5, 2
    inp = dict(
        x=rng.standard_normal((b, T, H, P)),
        dt_raw=rng.standard_normal((b, T, H)) - 1.0,
        A_log=rng.uniform(-0.5, 1.0, H),
        B=rng.standard_normal((b, T, G, N)) / np.sqrt(N),
        C=rng.standard_normal((b, T, G, N)) / np.sqrt(N),
        D=rng.standard_normal(H),
        init=rng.standard_normal((b, H, P, N)),
        bias=rng.uniform(-1.0, 1.0, H) if bias else None,
        z=rng.standard_normal((b, T, H, P)) if gate else None,
        w=rng.uniform(0.5, 1.5, H * P) if weight and group else None,
    )
    opts = dict(group=group, softplus=softplus, lo=lo, hi=hi)
    W = rng.standard_normal((b, T, H, P))
    V = rng.standard_normal((b, H, P, N))
    return inp, opts, W, V


def _loss(inp, opts, W, V):
    out, fin = ob.block_forward(inp["x"], inp["dt_raw"], inp["A_log"], inp["B"], inp["C"], inp["D"],
                                initial_states=inp["init"], dt_bias=inp["bias"], dt_softplus=opts["softplus"],
                                dt_lo=opts["lo"], dt_hi=opts["hi"], z=inp["z"], norm_weight=inp["w"],
                                norm_group_size=opts["group"], norm_eps=1e-5)
    return float(np.sum(W * out) + np.sum(V * fin))


NAMES = {"x": "dx", "dt_raw": "ddt_raw", "A_log": "dA_log", "B": "dB", "C": "dC", "D": "dD", "init": "dinit",
         "bias": "ddt_bias", "z": "dz", "w": "dnorm_weight"}


def finite_difference_ok(m, seed=3, samples=5, h=1e-6, **kw):
    inp, opts, W, V = _problem(seed, **kw)
    g = m.block_backward(inp["x"], inp["dt_raw"], inp["A_log"], inp["B"], inp["C"], W, D=inp["D"],
                         initial_states=inp["init"], dfinal=V, dt_bias=inp["bias"], dt_softplus=opts["softplus"],
                         dt_lo=opts["lo"], dt_hi=opts["hi"], z=inp["z"], norm_weight=inp["w"],
                         norm_group_size=opts["group"], norm_eps=1e-5)
    rng = np.random.default_rng(seed + 100)
    for name, gname in NAMES.items():
        arr = inp[name]
        if arr is None:
            assert g[gname] is None, gname
            continue
        for _ in range(samples):
            idx = tuple(rng.integers(0, s) for s in arr.shape)
            old = arr[idx]
            arr[idx] = old + h
            lp = _loss(inp, opts, W, V)
            arr[idx] = old - h
            lm = _loss(inp, opts, W, V)
            arr[idx] = old
            fd = (lp - lm) / (2 * h)
            if abs(g[gname][idx] - fd) > 1e-5 * max(1.0, abs(fd)):
                return False
    return True


@pytest.mark.parametrize("kw", [
    dict(),                                        # gate, norm over groups of two heads, weight, bias, softplus
    dict(group=3),                                 # norm per head
    dict(group=12),                                # one group over the whole channel row
    dict(gate=False),                              # norm without gate
    dict(group=0),                                 # gate only
    dict(gate=False, group=0),                     # dt step only
    dict(weight=False),                            # norm without weight
    dict(bias=False, softplus=False),              # raw dt used as is
    dict(lo=0.12, hi=0.45),                        # clamp active on some tokens
], ids=lambda kw: ",".join("%s=%s" % i for i in kw.items()) or "default")
def test_block_backward_matches_finite_differences(kw):
    assert finite_difference_ok(obb, **kw)


def test_clamp_is_active_in_the_clamped_case():
    # the clamp case above is only a pin if some dt actually hit the bounds
    inp, opts, _, _ = _problem(3, lo=0.12, hi=0.45)
    sp = ob.softplus(inp["dt_raw"] + inp["bias"])
    assert np.any(sp < 0.12) and np.any(sp > 0.45) and np.any((sp > 0.12) & (sp < 0.45))


MUTANTS = {
    "norm_without_mean_term": ("dg = (dn - n * np.mean(dn * n, axis=-1, keepdims=True)) / r", "dg = dn / r"),
    "silu_derivative_without_z_term": ("(s * (1.0 + z * (1.0 - s)))", "s"),
    "dy_without_gate": ("dy = dg * (z * s)", "dy = dg"),
    "no_clamp_mask": ("mask = (sp > dt_lo) & (sp < dt_hi)", "mask = 1.0"),
    "softplus_derivative_missing": ("(sigmoid(v) if dt_softplus else 1.0)", "1.0"),
    "weight_gradient_from_gated": ("dw = np.sum(do * n, axis=(0, 1))", "dw = np.sum(do * rows, axis=(0, 1))"),
}


def _mutant(name):
    a, b = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(a) == 1, name
    mod = types.ModuleType("oracle_block_backward_" + name)
    exec(compile(src.replace(a, b), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_block_backward_mutant_is_caught(name):
    kw = dict(lo=0.12, hi=0.45) if name == "no_clamp_mask" else {}
    assert not finite_difference_ok(_mutant(name), **kw)
