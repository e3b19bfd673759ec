"""Pins of the oracle's model variants (survey row f, NEXT-3): the
zero-order-hold input drive of the appendix and the output map of Sec. 3
with a residual weight and an activation (y = act(C h + D_res x)).  Each
is pinned against something other than the oracle's own formula: the
exact solution of the continuous-time system for a held input,
forward-mode autograd of an independent torch loop, central differences
and closed forms; planted mistakes are caught."""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest
import torch

from oracle import oracle
from tests.test_oracle_pins import rand_problem, relerr


@pytest.fixture(autouse=True)
def _float64_default():
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)


def _torch_model(p, xt, drive, act):
    """The selective scan with the chosen drive and output map as a plain
    torch loop."""
    f64 = dict(dtype=torch.float64)
    z = xt * torch.tensor(p["w_delta"], **f64) + torch.tensor(p["b_delta"], **f64)
    delta = torch.logaddexp(z, torch.zeros((), **f64))
    Bm = xt @ torch.tensor(p["W_B"], **f64) + torch.tensor(p["b_B"], **f64)
    Cm = xt @ torch.tensor(p["W_C"], **f64) + torch.tensor(p["b_C"], **f64)
    A = torch.tensor(p["A"], **f64)
    Bsz, L, D = xt.shape
    h = torch.zeros(Bsz, D, A.shape[1], **f64)
    ys = []
    for t in range(L):
        dl = delta[:, t, :, None]
        coef = dl if drive == "euler" else torch.expm1(dl * A) / A
        h = torch.exp(dl * A) * h + coef * Bm[:, t, None, :] * xt[:, t, :, None]
        yh = (h * Cm[:, t, None, :]).sum(-1)
        if p.get("D_res") is not None:
            yh = yh + torch.tensor(p["D_res"], **f64) * xt[:, t]
        ys.append(yh if act == "identity" else torch.nn.functional.silu(yh))
    return torch.stack(ys, 1)


def problem(seed, L=14, D=3, N=4, K=2, stiff=False, dres=True):
    p, x, dx = rand_problem(seed, B=2, L=L, D=D, N=N, K=K, stiff=stiff, bias=True)
    if dres:
        p["D_res"] = np.random.default_rng(seed + 500).standard_normal(D)
    return p, x, dx


@pytest.mark.parametrize("drive,act,stiff", [("zoh", "identity", False), ("zoh", "identity", True),
                                             ("euler", "silu", False), ("zoh", "silu", False)])
def test_forward_mode_autograd(drive, act, stiff):
    p, x, dx = problem(60 + stiff, stiff=stiff)
    y, dy, _, _ = oracle.scan_jvp(x, dx, p, drive=drive, act=act)
    f = lambda xt: _torch_model(p, xt, drive, act)
    assert relerr(y, f(torch.tensor(x)).numpy()) < 1e-12
    for k in range(dx.shape[0]):
        _, jv = torch.func.jvp(f, (torch.tensor(x),), (torch.tensor(dx[k]),))
        assert relerr(dy[k], jv.numpy()) < 1e-11, k


@pytest.mark.parametrize("drive,act", [("zoh", "identity"), ("zoh", "silu")])
def test_central_differences(drive, act):
    p, x, dx = problem(62, L=20, K=1)
    _, dy, _, _ = oracle.scan_jvp(x, dx, p, drive=drive, act=act)
    eps = 1e-6
    yp, _, _, _ = oracle.scan_jvp(x + eps * dx[0], dx, p, drive=drive, act=act)
    ym, _, _, _ = oracle.scan_jvp(x - eps * dx[0], dx, p, drive=drive, act=act)
    assert relerr(dy[0], (yp - ym) / (2 * eps)) < 1e-8


def test_zoh_is_exact_for_a_held_input():
    """Constant Delta, B, C and a constant input c: zero-order hold gives the
    exact solution of dh/ds = A h + B c at s = t*Delta, h(s) = (exp(A s) - 1)
    / A * B c, for every step count t (the Euler drive does not)."""
    g = np.random.default_rng(63)
    D, N, L = 3, 5, 30
    p = dict(A=-g.uniform(0.1, 3, (D, N)), w_delta=np.zeros(D), b_delta=g.uniform(-2, 1, D),
             W_B=np.zeros((D, N)), W_C=np.zeros((D, N)), b_B=g.standard_normal(N), b_C=g.standard_normal(N))
    c = g.standard_normal(D)
    x = np.broadcast_to(c, (1, L, D)).copy()
    dx = np.zeros((1, 1, L, D))
    y, _, _, _ = oracle.scan_jvp(x, dx, p, drive="zoh")
    dl = np.log1p(np.exp(p["b_delta"]))
    t = np.arange(1, L + 1)[:, None, None]
    h = np.expm1(p["A"][None] * t * dl[None, :, None]) / p["A"][None] * p["b_B"] * c[None, :, None]
    ref = (h * p["b_C"]).sum(-1)
    assert relerr(y[0], ref) < 1e-13
    ye, _, _, _ = oracle.scan_jvp(x, dx, p, drive="euler")
    assert relerr(ye[0], ref) > 1e-3


def test_zoh_limit_at_zero_A():
    """A = 0 lanes: the ZOH coefficient (exp(Delta A) - 1)/A tends to Delta,
    the Euler coefficient, and Abar = 1: both drives agree exactly."""
    p, x, dx = problem(64)
    p["A"] = np.zeros_like(p["A"])
    a = oracle.scan_jvp(x, dx, p, drive="zoh")
    b = oracle.scan_jvp(x, dx, p, drive="euler")
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def test_residual_only_closed_form():
    """B = 0 keeps the state at zero: y = act(D_res x) and
    dy = act'(D_res x) D_res dx exactly, for both activations."""
    p, x, dx = problem(65)
    p = dict(p, W_B=np.zeros_like(p["W_B"]), b_B=np.zeros_like(p["b_B"]))
    z = p["D_res"] * x
    y, dy, _, _ = oracle.scan_jvp(x, dx, p, act="identity")
    assert np.array_equal(y, z) and np.array_equal(dy, p["D_res"] * dx)
    y, dy, _, _ = oracle.scan_jvp(x, dx, p, act="silu")
    s = 1 / (1 + np.exp(-z))
    assert relerr(y, z * s) < 1e-15
    assert relerr(dy, (s + z * s * (1 - s)) * p["D_res"] * dx) < 1e-14


PIN_TESTS = [
    lambda: test_forward_mode_autograd("zoh", "identity", False),
    lambda: test_forward_mode_autograd("zoh", "silu", False),
    lambda: test_zoh_is_exact_for_a_held_input(),
    lambda: test_zoh_limit_at_zero_A(),
    lambda: test_residual_only_closed_form(),
]

C_MUTANTS = {
    "ZOH coefficient replaced by Delta": ("const double ec = drive ? (a != 0.0 ? expm1(dl * a) / a : dl) : dl;",
                                          "const double ec = dl;"),
    "ZOH coefficient Abar*Delta": ("const double ec = drive ? (a != 0.0 ? expm1(dl * a) / a : dl) : dl;",
                                   "const double ec = drive ? (a != 0.0 ? abar * dl : dl) : dl;"),
    "ZOH limit at A = 0 dropped": ("expm1(dl * a) / a : dl) : dl;", "expm1(dl * a) / a : 0.0) : dl;"),
    "ZOH tangent without Abar": ("const double dec = drive ? abar : 1.0;", "const double dec = 1.0;"),
}


def _caught():
    for t in PIN_TESTS:
        try:
            t()
        except AssertionError:
            return True
    return False


def test_unmutated_oracle_passes_variant_pins():
    assert not _caught()


@pytest.mark.parametrize("name", sorted(C_MUTANTS))
def test_variant_c_mutant_is_caught(name, monkeypatch):
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


def _silu_derivative_without_curvature(yr, dyr, x, dx, D_res=None, act="identity"):
    yh = yr + (0 if D_res is None else D_res * x)
    dyh = dyr + (0 if D_res is None else D_res * dx)
    if act == "identity":
        return yh, dyh
    s = 1 / (1 + np.exp(-yh))
    return yh * s, s[None] * dyh


def _residual_missing_in_tangent(yr, dyr, x, dx, D_res=None, act="identity"):
    return _ORIG_MAP(yr, dyr, x, np.zeros_like(dx), D_res, act)


_ORIG_MAP = oracle.output_map


@pytest.mark.parametrize("fn", [_silu_derivative_without_curvature, _residual_missing_in_tangent])
def test_variant_python_mutant_is_caught(fn, monkeypatch):
    monkeypatch.setattr(oracle, "output_map", fn)
    assert _caught()
