"""Plants plausible mistakes in the second-order oracle (on the CPU) and
checks that the pins of test_oracle2_pins.py catch each one."""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest

from oracle import oracle
import tests.test_oracle2_pins as pins

PIN_TESTS = [
    lambda: pins.test_second_order_central_differences(21, False),
    lambda: pins.test_nested_forward_mode_autograd(),
    lambda: pins.test_quadratic_map_closed_form(),
    lambda: pins.test_segment_composition_closed_forms(),
    lambda: pins.test_linear_map_has_zero_second_derivative(),
]

C_MUTANTS = {
    "drop cross-talk Abar_w*hv": ("ab * hvw0 + ab_w * hv0 + ab_v * hw0", "ab * hvw0 + ab_v * hw0"),
    "cross-talk without Abar": ("const double ab_w = ab * a * dlw;", "const double ab_w = a * dlw;"),
    "drop curvature A^2 dv dw": ("const double ab_vw = ab * a * a * dlv * dlw + ab * a * dlvw;",
                                 "const double ab_vw = ab * a * dlvw;"),
    "drop softplus'' term": ("const double ab_vw = ab * a * a * dlv * dlw + ab * a * dlvw;",
                             "const double ab_vw = ab * a * a * dlv * dlw;"),
    "drop dvw*B*x": ("const double bt_vw = dlvw * Bt * xt + ", "const double bt_vw = "),
    "drop Delta*Bv*xw": ("+ dl * Bvt * xwt + dl * Bwt * xvt;", "+ dl * Bwt * xvt;"),
    "yvw without Cw*hv": ("s3 += Cvt * hw1 + Cwt * hv1 + Ct * hvw1;", "s3 += Cvt * hw1 + Ct * hvw1;"),
    "hvw uses new h": ("+ ab_vw * h0 + bt_vw;", "+ ab_vw * h1 + bt_vw;"),
}


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
        c, so = os.path.join(td, "m.c"), os.path.join(td, "m.so")
        with open(c, "w") as f:
            f.write(src.replace(old, new))
        subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                        "-o", so, c, "-lm"], check=True)
        lib = oracle.declare(ctypes.CDLL(so))
        monkeypatch.setattr(oracle, "_lib", lib)
        assert _caught(), name


def _disc2_no_curvature(x, xv, xw, w_delta, b_delta):
    d, dv, dw, dvw = _orig_disc2(x, xv, xw, w_delta, b_delta)
    return d, dv, dw, np.zeros_like(dvw)


def _disc2_wrong_sign(x, xv, xw, w_delta, b_delta):
    d, dv, dw, dvw = _orig_disc2(x, xv, xw, w_delta, b_delta)
    return d, dv, dw, -dvw


_orig_disc2 = oracle.discretize2


@pytest.mark.parametrize("name,fn", [("softplus'' dropped", _disc2_no_curvature),
                                     ("softplus'' sign", _disc2_wrong_sign)])
def test_python_mutant_is_caught(name, fn, monkeypatch):
    monkeypatch.setattr(oracle, "discretize2", fn)
    assert _caught(), name
