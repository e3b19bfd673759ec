"""Pins of the oracle's low-rank step size (Mamba's dt projection: z =
(x W_dx) W_dt + b, Delta = softplus(z), over all channels through a rank-R
bottleneck): the depthwise model when W_dx W_dt is diagonal, forward-mode
autograd of an independent torch loop, central differences; planted
mistakes are caught."""
import numpy as np
import pytest
import torch

from oracle import oracle
from tests.test_oracle_pins import rand_problem, relerr


def problem(seed, R=2, D=5, N=4, L=12, K=2):
    p, x, dx = rand_problem(seed, B=2, L=L, D=D, N=N, K=K, bias=True)
    r = np.random.default_rng(seed + 700)
    p.update(W_dx=r.standard_normal((D, R)) / np.sqrt(D), W_dt=r.standard_normal((R, D)))
    del p["w_delta"]
    return p, x, dx


def test_diagonal_low_rank_is_depthwise():
    """R = D, W_dx = I, W_dt = diag(w): z = x*w + b exactly (the tangent's
    products associate differently: equal to rounding)."""
    p, x, dx = rand_problem(100, B=2, L=10, D=4, N=3, K=2, bias=True)
    a = oracle.scan_jvp(x, dx, p)
    q = {k: v for k, v in p.items() if k != "w_delta"}
    q.update(W_dx=np.eye(4), W_dt=np.diag(p["w_delta"]))
    b = oracle.scan_jvp(x, dx, q)
    assert np.array_equal(a[0], b[0])
    for u, v in zip(a[1:], b[1:]):
        assert relerr(v, u) < 1e-14


def _torch_model(p, xt):
    f64 = dict(dtype=torch.float64)
    z = (xt @ torch.tensor(p["W_dx"], **f64)) @ torch.tensor(p["W_dt"], **f64) + torch.tensor(p["b_delta"], **f64)
    delta = torch.logaddexp(z, torch.zeros((), **f64))
    Bm = xt @ torch.tensor(p["W_B"], **f64) + torch.tensor(p["b_B"], **f64)
    Cm = xt @ torch.tensor(p["W_C"], **f64) + torch.tensor(p["b_C"], **f64)
    A = torch.tensor(p["A"], **f64)
    h = torch.zeros(xt.shape[0], xt.shape[2], A.shape[1], **f64)
    ys = []
    for t in range(xt.shape[1]):
        dl = delta[:, t, :, None]
        h = torch.exp(dl * A) * h + dl * Bm[:, t, None, :] * xt[:, t, :, None]
        ys.append((h * Cm[:, t, None, :]).sum(-1))
    return torch.stack(ys, 1)


@pytest.mark.parametrize("R", [1, 3])
def test_forward_mode_autograd(R):
    p, x, dx = problem(101 + R, R=R)
    y, dy, _, _ = oracle.scan_jvp(x, dx, p)
    f = lambda xt: _torch_model(p, xt)
    assert relerr(y, f(torch.tensor(x)).numpy()) < 1e-12
    for k in range(dx.shape[0]):
        _, jv = torch.func.jvp(f, (torch.tensor(x),), (torch.tensor(dx[k]),))
        assert relerr(dy[k], jv.numpy()) < 1e-12


def test_central_differences():
    p, x, dx = problem(104, L=18, K=1)
    _, dy, _, _ = oracle.scan_jvp(x, dx, p)
    eps = 1e-6
    yp, _, _, _ = oracle.scan_jvp(x + eps * dx[0], dx, p)
    ym, _, _, _ = oracle.scan_jvp(x - eps * dx[0], dx, p)
    assert relerr(dy[0], (yp - ym) / (2 * eps)) < 1e-8


def _tangent_without_projection(x, dx, W_dx, W_dt, b_dt):
    d, _ = _ORIG(x, dx, W_dx, W_dt, b_dt)
    z = (np.asarray(x, float) @ W_dx) @ W_dt + b_dt
    return d, (1 / (1 + np.exp(-z)))[None] * np.asarray(dx, float)      # forgot the projection of dx


def _bias_in_tangent(x, dx, W_dx, W_dt, b_dt):
    d, _ = _ORIG(x, dx, W_dx, W_dt, b_dt)
    z = (np.asarray(x, float) @ W_dx) @ W_dt + b_dt
    dz = (np.asarray(dx, float) @ W_dx) @ W_dt + b_dt
    return d, (1 / (1 + np.exp(-z)))[None] * dz


_ORIG = oracle.discretize_lowrank


@pytest.mark.parametrize("fn", [_tangent_without_projection, _bias_in_tangent])
def test_planted_mistakes_are_caught(fn, monkeypatch):
    monkeypatch.setattr(oracle, "discretize_lowrank", fn)
    with pytest.raises(AssertionError):
        test_forward_mode_autograd(3)
