"""Plants plausible mistakes in the oracle (on the CPU) and checks that the
pins of test_oracle_pins.py catch every one of them.

C-level mutations are compiled from a text substitution of pgf_oracle.c into
a temporary library; Python-level mutations replace one oracle function.  For
each mutant, at least one pin must fail.
"""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest

from oracle import oracle
import tests.test_oracle_pins as pins

PIN_TESTS = [
    lambda: pins.test_lti_impulse_closed_form(),
    lambda: pins.test_quadratic_kernel_form(3, True),
    lambda: pins.test_softplus_identities(),
    lambda: pins.test_projection_bruteforce(),
    lambda: pins.test_tangent_central_differences(6, False),
    lambda: pins.test_tangent_forward_mode_autograd(),
    lambda: pins.test_entry_state_composition_eq5(),
    lambda: pins.test_stiff_underflow_is_exact_drive(),
    lambda: pins.test_causality_prefix_and_ghost_pulse_zeros(),
]

C_MUTANTS = {
    "drop K_t (dDelta through Abar)": ("const double Kt = abar * a * ddl;", "const double Kt = 0.0 * abar * a * ddl;"),
    "K_t sign": ("const double Kt = abar * a * ddl;", "const double Kt = -abar * a * ddl;"),
    "K_t without A": ("const double Kt = abar * a * ddl;", "const double Kt = abar * ddl;"),
    "drop dDelta*B*x": ("const double jt = dec * ddl * Bt[n] * xt + ", "const double jt = "),
    "drop Delta*dB*x": ("+ ec * dBm[kbtn] * xt ", ""),
    "drop Delta*B*dx": ("+ ec * Bt[n] * dxt;", ";"),
    "drop dC*h (paper's Eq. 2)": ("dyk[k] += dCm[kbtn] * hnew + Ct[n] * dhnew;", "dyk[k] += Ct[n] * dhnew;"),
    "output uses previous state": ("yt += Ct[n] * hnew;", "yt += Ct[n] * hprev;"),
    "tangent uses new state": ("Kt * hprev + jt", "Kt * hnew + jt"),
    "Euler decay 1+Delta*A": ("const double abar = exp(dl * a);", "const double abar = 1.0 + dl * a;"),
    "B index off by one": ("const double *Bt = Bm + (b * L + t) * N;",
                           "const double *Bt = Bm + (b * L + (t > 0 ? t - 1 : 0)) * N;"),
}


def _build_mutant(src_text, tmpdir, name):
    c = os.path.join(tmpdir, name + ".c")
    so = os.path.join(tmpdir, name + ".so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    "-o", so, c, "-lm"], check=True)
    return oracle.declare(ctypes.CDLL(so))


def _caught():
    for t in PIN_TESTS:
        try:
            t()
        except AssertionError:
            return True
    return False


def test_unmutated_oracle_passes_all_pins():
    assert not _caught()


@pytest.mark.parametrize("name", sorted(C_MUTANTS))
def test_c_mutant_is_caught(name, monkeypatch):
    with open(oracle._SRC) as f:
        src = f.read()
    old, new = C_MUTANTS[name]
    assert src.count(old) == 1, name
    with tempfile.TemporaryDirectory() as td:
        lib = _build_mutant(src.replace(old, new), td, "mut")
        monkeypatch.setattr(oracle, "_lib", lib)
        assert _caught(), name


def _softplus_wrong(x, dx, w_delta, b_delta):
    x = np.asarray(x, dtype=np.float64)
    z = x * np.asarray(w_delta, dtype=np.float64) + np.asarray(b_delta, dtype=np.float64)
    delta = np.log1p(np.exp(z)) * 1.0
    sw = 1.0 / (1.0 + np.exp(-z))             # derivative without the w factor
    return delta, sw[None] * np.asarray(dx, dtype=np.float64)


def _project_transposed(x, dx, W_B, W_C, b_B=None, b_C=None):
    Bm, Cm, dBm, dCm = _orig_project(x, dx, W_C, W_B, b_C, b_B)   # B and C swapped
    return Bm, Cm, dBm, dCm


def _project_no_bias(x, dx, W_B, W_C, b_B=None, b_C=None):
    return _orig_project(x, dx, W_B, W_C)


_orig_project = oracle.project


@pytest.mark.parametrize("name,attr,fn", [
    ("dDelta missing w_delta", "discretize", _softplus_wrong),
    ("B and C swapped", "project", _project_transposed),
    ("bias hooks dropped", "project", _project_no_bias),
])
def test_python_mutant_is_caught(name, attr, fn, monkeypatch):
    monkeypatch.setattr(oracle, attr, fn)
    assert _caught(), name
