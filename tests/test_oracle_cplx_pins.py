"""Pins of the complex-transition oracle (Sec. 3: state in C^{D x N},
y = Re(C h)) against the real oracle at A_im = 0, the closed-form impulse
response of a damped oscillator, forward-mode autograd of an independent
complex torch loop, central differences, conjugation symmetry and the
segment composition; with the zero-order-hold drive, the real ZOH oracle
at A_im = 0, the exact solution of the oscillator ODE for a held input,
autograd and central differences; planted mistakes are caught."""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest
import torch

from oracle import oracle
from tests.test_oracle_pins import rand_problem, relerr


def problem(seed, B=2, L=14, D=3, N=4, K=2, stiff=False):
    p, x, dx = rand_problem(seed, B=B, L=L, D=D, N=N, K=K, stiff=stiff, bias=True)
    r = np.random.default_rng(seed + 900)
    p["A_im"] = np.pi * r.uniform(0.2, 4.0, (D, N)) * r.choice([-1, 1], (D, N))
    return p, x, dx


def test_real_limit():
    p, x, dx = problem(80)
    a = oracle.scan_jvp(x, dx, dict(p, A_im=np.zeros_like(p["A"])))
    b = oracle.scan_jvp(x, dx, {k: v for k, v in p.items() if k != "A_im"})
    for u, w in zip(a, b):
        assert relerr(np.real(u), w) < 1e-14 and np.abs(np.imag(u)).max() == 0


def test_damped_oscillator_impulse_response():
    """Constant Delta, B, C and an impulse x_0 = 1: h_t = exp(t Delta A) Delta B,
    so y_t = sum_n C_n Delta B_n exp(t Delta A_re) cos(t Delta A_im)."""
    g = np.random.default_rng(81)
    D, N, L = 3, 5, 40
    p = dict(A=-g.uniform(0.05, 1.0, (D, N)), A_im=g.uniform(-6, 6, (D, N)), w_delta=np.zeros(D),
             b_delta=g.uniform(-2, 1, D), W_B=np.zeros((D, N)), W_C=np.zeros((D, N)),
             b_B=g.standard_normal(N), b_C=g.standard_normal(N))
    x = np.zeros((1, L, D))
    x[0, 0] = 1.0
    y, _, _, _ = oracle.scan_jvp(x, np.zeros((1, 1, L, D)), p)
    dl = np.log1p(np.exp(p["b_delta"]))[None, :, None]
    t = np.arange(L)[:, None, None]
    ref = (p["b_C"] * dl * p["b_B"] * np.exp(t * dl * p["A"]) * np.cos(t * dl * p["A_im"])).sum(-1)
    assert relerr(y[0], ref) < 1e-13


def _torch_model(p, xt, drive="euler"):
    f64 = dict(dtype=torch.float64)
    z = xt * torch.tensor(p["w_delta"], **f64) + torch.tensor(p["b_delta"], **f64)
    delta = torch.logaddexp(z, torch.zeros((), **f64))
    Bm = xt @ torch.tensor(p["W_B"], **f64) + torch.tensor(p["b_B"], **f64)
    Cm = xt @ torch.tensor(p["W_C"], **f64) + torch.tensor(p["b_C"], **f64)
    A = torch.complex(torch.tensor(p["A"], **f64), torch.tensor(p["A_im"], **f64))
    Bsz, L, D = xt.shape
    h = torch.zeros(Bsz, D, A.shape[1], dtype=torch.complex128)
    ys = []
    for t in range(L):
        dl = delta[:, t, :, None]
        e = dl if drive == "euler" else torch.expm1(dl * A) / A   # ZOH: (exp(dl A) - 1) / A
        h = torch.exp(dl * A) * h + e * Bm[:, t, None, :] * xt[:, t, :, None]
        ys.append((h.real * Cm[:, t, None, :]).sum(-1))
    return torch.stack(ys, 1)


@pytest.mark.parametrize("stiff", [False, True])
def test_forward_mode_autograd(stiff):
    p, x, dx = problem(82 + stiff, stiff=stiff)
    y, dy, _, _ = oracle.scan_jvp(x, dx, p)
    f = lambda xt: _torch_model(p, xt)
    assert relerr(y, f(torch.tensor(x)).numpy()) < 1e-12
    for k in range(dx.shape[0]):
        _, jv = torch.func.jvp(f, (torch.tensor(x),), (torch.tensor(dx[k]),))
        assert relerr(dy[k], jv.numpy()) < 1e-11, k


@pytest.mark.parametrize("stiff", [False, True])
def test_zoh_forward_mode_autograd(stiff):
    p, x, dx = problem(92 + stiff, stiff=stiff)
    y, dy, _, _ = oracle.scan_jvp(x, dx, p, drive="zoh")
    f = lambda xt: _torch_model(p, xt, "zoh")
    assert relerr(y, f(torch.tensor(x)).numpy()) < 1e-12
    for k in range(dx.shape[0]):
        _, jv = torch.func.jvp(f, (torch.tensor(x),), (torch.tensor(dx[k]),))
        assert relerr(dy[k], jv.numpy()) < 1e-11, k


def test_zoh_real_limit_and_central_differences():
    p, x, dx = problem(94, L=20, K=1)
    a = oracle.scan_jvp(x, dx, dict(p, A_im=np.zeros_like(p["A"])), drive="zoh")
    b = oracle.scan_jvp(x, dx, {k: v for k, v in p.items() if k != "A_im"}, drive="zoh")
    for u, w in zip(a, b):
        assert relerr(np.real(u), w) < 1e-14 and np.abs(np.imag(u)).max() == 0
    _, dy, _, _ = oracle.scan_jvp(x, dx, p, drive="zoh")
    eps = 1e-6
    yp, _, _, _ = oracle.scan_jvp(x + eps * dx[0], dx, p, drive="zoh")
    ym, _, _, _ = oracle.scan_jvp(x - eps * dx[0], dx, p, drive="zoh")
    assert relerr(dy[0], (yp - ym) / (2 * eps)) < 1e-8


def test_zoh_is_exact_for_a_held_oscillator_input():
    """Constant Delta, B, C and a constant input c: zero-order hold gives the
    exact solution of the damped oscillator dh/ds = A h + B c (A complex) at
    s = t*Delta, h(s) = (exp(A s) - 1) / A * B c, for every step count t."""
    g = np.random.default_rng(95)
    D, N, L = 3, 5, 30
    p = dict(A=-g.uniform(0.05, 2, (D, N)), A_im=g.uniform(-6, 6, (D, N)), w_delta=np.zeros(D),
             b_delta=g.uniform(-2, 1, D), W_B=np.zeros((D, N)), W_C=np.zeros((D, N)),
             b_B=g.standard_normal(N), b_C=g.standard_normal(N))
    c = g.standard_normal(D)
    x = np.broadcast_to(c, (1, L, D)).copy()
    y, _, _, _ = oracle.scan_jvp(x, np.zeros((1, 1, L, D)), p, drive="zoh")
    dl = np.log1p(np.exp(p["b_delta"]))
    A = (p["A"] + 1j * p["A_im"])[None]
    t = np.arange(1, L + 1)[:, None, None]
    h = np.expm1(A * t * dl[None, :, None]) / A * p["b_B"] * c[None, :, None]
    assert relerr(y[0], (h.real * p["b_C"]).sum(-1)) < 1e-12


def test_central_differences():
    p, x, dx = problem(84, L=20, K=1)
    _, dy, _, _ = oracle.scan_jvp(x, dx, p)
    eps = 1e-6
    yp, _, _, _ = oracle.scan_jvp(x + eps * dx[0], dx, p)
    ym, _, _, _ = oracle.scan_jvp(x - eps * dx[0], dx, p)
    assert relerr(dy[0], (yp - ym) / (2 * eps)) < 1e-8


def test_conjugation_symmetry():
    """Real inputs: flipping the sign of A_im conjugates the state, so the
    real read-out is unchanged."""
    p, x, dx = problem(85)
    a = oracle.scan_jvp(x, dx, p)
    b = oracle.scan_jvp(x, dx, dict(p, A_im=-p["A_im"]))
    assert relerr(b[0], a[0]) < 1e-14 and relerr(b[1], a[1]) < 1e-14
    assert relerr(b[2], np.conj(a[2])) < 1e-14


def test_segment_composition_closed_forms():
    """Over a block, (h, dh) maps to (P h + h0, P dh + Q h + dh0) with the
    complex P = exp(A sum Delta), Q = P A sum dDelta."""
    p, x, dx = problem(86, L=17, K=1)
    r = np.random.default_rng(87)
    h_in = r.standard_normal((2, 3, 4)) + 1j * r.standard_normal((2, 3, 4))
    dh_in = r.standard_normal((1, 2, 3, 4)) + 1j * r.standard_normal((1, 2, 3, 4))
    _, _, h0, dh0 = oracle.scan_jvp(x, dx, p)
    _, _, h1, dh1 = oracle.scan_jvp(x, dx, p, h_in=h_in, dh_in=dh_in)
    delta, ddelta = oracle.discretize(x, dx, p["w_delta"], p["b_delta"])
    A = (p["A"] + 1j * p["A_im"])[None]
    S = delta.sum(1)[:, :, None]
    P = np.exp(A * S)
    Q = P * A * ddelta[0].sum(1)[:, :, None]
    assert relerr(h1, P * h_in + h0) < 1e-13
    assert relerr(dh1[0], P * dh_in[0] + Q * h_in + dh0[0]) < 1e-13


PIN_TESTS = [test_damped_oscillator_impulse_response, lambda: test_forward_mode_autograd(False),
             test_segment_composition_closed_forms, lambda: test_zoh_forward_mode_autograd(False),
             test_zoh_is_exact_for_a_held_oscillator_input]

C_MUTANTS = {
    "imaginary part dropped from exp": ("const double complex abar = cexp(dl * a);",
                                        "const double complex abar = cexp(dl * creal(a));"),
    "tangent uses the real part of A": ("abar * a * ddl * hprev", "abar * creal(a) * ddl * hprev"),
    "tangent uses Re(h)": ("abar * a * ddl * hprev", "abar * a * ddl * creal(hprev)"),
    "read-out of Im(h)": ("yt += Cm[btn + n] * creal(hnew);", "yt += Cm[btn + n] * cimag(hnew);"),
    "tangent read-out drops C*Re(dh)": ("dy[kbtd] += dCm[kbtn] * creal(hnew) + Cm[btn + n] * creal(dhnew);",
                                        "dy[kbtd] += dCm[kbtn] * creal(hnew);"),
    "ZOH coefficient from the real part of A": ("cexpm1_(dl * a) / a", "cexpm1_(dl * creal(a)) / creal(a)"),
    "ZOH coefficient without the sin^2 term": ("(expm1(u) * cos(v) - 2.0 * sh * sh)", "(expm1(u) * cos(v))"),
    "ZOH tangent drive without Abar": ("const double complex de = drive ? abar : 1.0;",
                                       "const double complex de = 1.0;"),
}


def _caught():
    for t in PIN_TESTS:
        try:
            t()
        except AssertionError:
            return True
    return False


def test_unmutated_oracle_passes_cplx_pins():
    assert not _caught()


@pytest.mark.parametrize("name", sorted(C_MUTANTS))
def test_cplx_c_mutant_is_caught(name, monkeypatch):
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
        monkeypatch.setattr(oracle, "_lib", oracle.declare(ctypes.CDLL(so)))
        assert _caught(), name
