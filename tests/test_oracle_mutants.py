"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a private copy of the oracle's C source
(CPU only: compiled with gcc into a temporary directory), then checks that the
pins of ``test_oracle_pins`` reject the mutant.  The real oracle is untouched.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from tests.test_oracle_pins import matrix_form, rand_problem

SRC = os.path.join(os.path.dirname(oracle.__file__), "ssd_oracle.c")

MUTANTS = {
    "decay_without_dt": ("const double decay = exp(dtt * A);", "const double decay = exp(A);"),
    "input_without_dt": ("const double xin = dtt * xt[p];", "const double xin = xt[p];"),
    "A_sign": ("const double A = -exp(A_log[h]);", "const double A = exp(-A_log[h]);"),
    "group_interleaved": ("g = h / heads_per_group;", "g = h % G;"),
    "decay_after_input": ("Sp[n] = decay * Sp[n] + xin * Bt[n];",
                          "Sp[n] = decay * (Sp[n] + xin * Bt[n]);"),
    "output_before_update": ("Sp[n] = decay * Sp[n] + xin * Bt[n];\n                    acc += Sp[n] * Ct[n];",
                             "acc += Sp[n] * Ct[n];\n                    Sp[n] = decay * Sp[n] + xin * Bt[n];"),
    "B_C_swapped": ("acc += Sp[n] * Ct[n];", "acc += Sp[n] * Bt[n];"),
    "D_dropped": ("yt[p] = acc + Dh * xt[p];", "yt[p] = acc;"),
    "no_varlen_reset": ("int first = (t == 0) || (seq_idx && seq_idx[t] != seq_idx[t - 1]);",
                        "int first = (t == 0);"),
}


def _pins_hold(lib):
    """True when the mutant passes every check (i.e. the pins are blind)."""
    rng = np.random.default_rng(21)
    args = rand_problem(rng, b=1, T=20, H=4, P=3, N=5, G=2)
    y, fin = oracle.forward(*args, lib=lib)
    y_ref, fin_ref = matrix_form(*args)
    ok = np.allclose(y, y_ref, rtol=1e-10, atol=1e-12) and np.allclose(fin, fin_ref, rtol=1e-10)
    # packed varlen = separate runs (catches reset mistakes)
    lens = [4, 7, 9]
    x, dt, A_log, B, C, D, _ = rand_problem(rng, b=1, T=20, H=2, G=1, init=False)
    h0 = rng.standard_normal((3, 2, 3, 5))
    seq = np.repeat(np.arange(3), lens).astype(np.int32)[None]
    yv, fv = oracle.forward(x, dt, A_log, B, C, D, h0, seq, lib=lib)
    s = 0
    for q, L in enumerate(lens):
        sl = slice(s, s + L)
        yq, fq = matrix_form(x[:, sl], dt[:, sl], A_log, B[:, sl], C[:, sl], D, h0[q:q + 1])
        ok = ok and np.allclose(yv[:, sl], yq, rtol=1e-10, atol=1e-12)
        ok = ok and np.allclose(fv[q], fq[0], rtol=1e-10, atol=1e-12)
        s += L
    return ok


@pytest.fixture(scope="module")
def workdir(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    return tmp_path_factory.mktemp("oracle_mutants")


def test_unmutated_copy_passes(workdir):
    so = str(workdir / "ref.so")
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                           SRC, "-o", so, "-lm"])
    assert _pins_hold(oracle.load_library(so))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(workdir, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: %s" % name
    path = workdir / ("%s.c" % name)
    path.write_text(src.replace(old, new))
    so = str(workdir / ("%s.so" % name))
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                           str(path), "-o", so, "-lm"])
    assert not _pins_hold(oracle.load_library(so))
