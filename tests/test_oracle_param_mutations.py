"""Plants plausible mistakes in the parameter-flow oracle (on the CPU) and
checks that the pins of test_oracle_param_pins.py catch each one."""
import ctypes
import os
import subprocess
import tempfile

import pytest

from oracle import oracle
import tests.test_oracle_param_pins as pins

PIN_TESTS = [
    lambda: pins.test_reverse_mode_autograd(40, False),
    lambda: pins.test_central_differences_of_the_primal(),
    lambda: pins.test_time_invariant_closed_form(),
    lambda: pins.test_one_step_adjoint_is_the_outer_product(),
    lambda: pins.test_segment_composition_closed_forms(),
    lambda: pins.test_zoh_reverse_mode_autograd("normal"),
    lambda: pins.test_zoh_reverse_mode_autograd("small_steps"),
    lambda: pins.test_zoh_central_differences_along_A(False),
    lambda: pins.test_zoh_central_differences_along_A(True),
    lambda: pins.test_output_map_reverse_mode_autograd("silu", "euler", False),
    lambda: pins.test_output_map_identity_residual_closed_form(),
    lambda: pins.test_output_map_central_differences(),
    lambda: pins.test_output_map_one_step_adjoint(),
    lambda: pins.test_step_size_reverse_mode_autograd("euler", "identity", False),
    lambda: pins.test_step_size_reverse_mode_autograd("zoh", "silu", False),
    lambda: pins.test_step_size_central_differences(),
    lambda: pins.test_step_size_segment_composition_and_chunks(),
    lambda: pins.test_step_size_one_step_adjoint(),
]

C_MUTANTS = {
    "GammaA without its drive": ("const double ga = abar * gA[i] + dl * abar * hprev + ea * Bm[btn + n] * xt;",
                                 "const double ga = abar * gA[i] + ea * Bm[btn + n] * xt;"),
    "GammaA drive without Abar": ("const double ga = abar * gA[i] + dl * abar * hprev + ea * Bm[btn + n] * xt;",
                                  "const double ga = abar * gA[i] + dl * hprev + ea * Bm[btn + n] * xt;"),
    "GammaA drive from the new state": (
        "const double ga = abar * gA[i] + dl * abar * hprev + ea * Bm[btn + n] * xt;",
        "const double ga = abar * gA[i] + dl * (abar * hprev + ec * Bm[btn + n] * xt) + ea * Bm[btn + n] * xt;"),
    "GammaA without the ZOH drive's A-derivative": (
        "const double ga = abar * gA[i] + dl * abar * hprev + ea * Bm[btn + n] * xt;",
        "const double ga = abar * gA[i] + dl * abar * hprev;"),
    "ZOH de/dA series coefficient (m+2) for (m+1)": ("s += (double)(m + 1) / fact * zm;",
                                                      "s += (double)(m + 2) / fact * zm;"),
    "ZOH de/dA closed form without the 1/A": ("if (fabs(z) >= 1e-3) return (dl * exp(z) - expm1(z) / a) / a;",
                                              "if (fabs(z) >= 1e-3) return dl * exp(z) - expm1(z) / a;"),
    "GammaB drive carries B": ("const double gb = abar * gB[i] + ec * xt;",
                               "const double gb = abar * gB[i] + ec * Bm[btn + n] * xt;"),
    "GammaB ZOH drive taken as Delta": ("const double gb = abar * gB[i] + ec * xt;",
                                        "const double gb = abar * gB[i] + dl * xt;"),
    "GammaB without decay": ("const double gb = abar * gB[i] + ec * xt;", "const double gb = gB[i] + ec * xt;"),
    "G_C from the state's B-flow": ("GC[i] += w * h[i];", "GC[i] += w * gB[i];"),
    "G_C against the raw adjoint": ("GC[i] += w * h[i];", "GC[i] += gy[btd] * h[i];"),
    "G_A without C": ("GA[i] += w * Ct * gA[i];", "GA[i] += w * gA[i];"),
    "G_B from GammaA": ("GB[i] += w * Ct * gB[i];", "GB[i] += w * Ct * gA[i];"),
    "output map without the residual": ("if (D_res) yhat += D_res[d] * xt;", "(void)0;"),
    "adjoint without act'": ("const double w = gy[btd] * slope;", "const double w = gy[btd];"),
    "SiLU slope without its second term": ("slope = sg + yhat * sg * (1.0 - sg);", "slope = sg;"),
    "SiLU slope with sigma' as sg^2": ("slope = sg + yhat * sg * (1.0 - sg);", "slope = sg + yhat * sg * sg;"),
    "G_D from the output": ("if (D_res) GD[b * D + d] += w * xt;", "if (D_res) GD[b * D + d] += w * yt;"),
    "G_D against the raw adjoint": ("if (D_res) GD[b * D + d] += w * xt;",
                                    "if (D_res) GD[b * D + d] += gy[btd] * xt;"),
    "dh/dDelta without the transition's term": (
        "const double hd = an * abar * hprev + (drive ? abar : 1.0) * Bm[btn + n] * xt;",
        "const double hd = (drive ? abar : 1.0) * Bm[btn + n] * xt;"),
    "dh/dDelta with the ZOH drive's derivative taken as 1": (
        "const double hd = an * abar * hprev + (drive ? abar : 1.0) * Bm[btn + n] * xt;",
        "const double hd = an * abar * hprev + Bm[btn + n] * xt;"),
    "dh/dDelta from the new state": (
        "const double hd = an * abar * hprev + (drive ? abar : 1.0) * Bm[btn + n] * xt;",
        "const double hd = an * hnew + (drive ? abar : 1.0) * Bm[btn + n] * xt;"),
    "Gamma_w without x": ("gW[i] = abar * gW[i] + sig[btd] * xt * hd;", "gW[i] = abar * gW[i] + sig[btd] * hd;"),
    "Gamma_w without decay": ("gW[i] = abar * gW[i] + sig[btd] * xt * hd;", "gW[i] = gW[i] + sig[btd] * xt * hd;"),
    "Gamma_s without sigma": ("gS[i] = abar * gS[i] + sig[btd] * hd;", "gS[i] = abar * gS[i] + hd;"),
    "G_w without C": ("cw += Cm[btn + n] * gW[i];", "cw += gW[i];"),
    "G_s from Gamma_w": ("cs += Cm[btn + n] * gS[i];", "cs += Cm[btn + n] * gW[i];"),
    "G_w against the raw adjoint": ("GW[b * D + d] += w * cw;", "GW[b * D + d] += gy[btd] * cw;"),
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


def test_python_mutant_is_caught(monkeypatch):
    """The projections of the parameter path without the bias of B."""
    orig = oracle.project

    def no_bias(x, dx, W_B, W_C, b_B=None, b_C=None):
        return orig(x, dx, W_B, W_C, None, b_C)

    monkeypatch.setattr(oracle, "project", no_bias)
    assert _caught()
