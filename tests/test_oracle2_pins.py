"""Pins of the second-order (App. G Hessian flow) oracle against facts that
do not come from its own formula: finite differences of the separately
pinned first-order oracle, nested forward-mode autograd of an independent
torch loop, symmetry and bilinearity in the two directions, exact zeros for
a linear map and ahead of the directions' support, a closed form for a map
that is quadratic in the input, and the segment-composition closed forms
the GPU carry uses."""
import numpy as np
import pytest
import torch

from oracle import oracle
from tests.test_oracle_pins import _torch_primal, rand_problem, relerr


@pytest.fixture(autouse=True)
def _float64_default():
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)


def problem(seed, B=1, L=12, D=3, N=4, stiff=False, bias=True):
    p, x, dx = rand_problem(seed, B=B, L=L, D=D, N=N, K=2, stiff=stiff, bias=bias)
    return p, x, dx[0], dx[1]


def test_first_order_parts_match_first_order_oracle():
    p, x, v, w = problem(20, B=2, L=15)
    (y, yv, yw, _), _ = oracle.scan_jvp2(x, v, w, p)
    y1, dy1, _, _ = oracle.scan_jvp(x, np.stack([v, w]), p)
    assert relerr(y, y1) < 1e-15 and relerr(yv, dy1[0]) < 1e-15 and relerr(yw, dy1[1]) < 1e-15


@pytest.mark.parametrize("seed,stiff", [(21, False), (22, True)])
def test_second_order_central_differences(seed, stiff):
    """y_vw is the derivative along w of the (pinned) first-order y_v."""
    p, x, v, w = problem(seed, B=2, L=20, stiff=stiff)
    (_, _, _, yvw), _ = oracle.scan_jvp2(x, v, w, p)
    eps = 1e-5
    _, dyp, _, _ = oracle.scan_jvp(x + eps * w, v[None], p)
    _, dym, _, _ = oracle.scan_jvp(x - eps * w, v[None], p)
    assert relerr(yvw, (dyp[0] - dym[0]) / (2 * eps)) < 1e-8


def test_nested_forward_mode_autograd():
    p, x, v, w = problem(23, B=2, L=9, D=3, N=3)
    (y, yv, yw, yvw), _ = oracle.scan_jvp2(x, v, w, p)
    f = lambda xt: _torch_primal(p, xt)
    jv = lambda xt: torch.func.jvp(f, (xt,), (torch.tensor(v),))[1]
    _, hvp = torch.func.jvp(jv, (torch.tensor(x),), (torch.tensor(w),))
    assert relerr(yvw, hvp.numpy()) < 1e-12
    assert relerr(yv, jv(torch.tensor(x)).numpy()) < 1e-12


def test_symmetry_and_bilinearity():
    p, x, v, w = problem(24, L=18)
    (_, _, _, a), _ = oracle.scan_jvp2(x, v, w, p)
    (_, _, _, b), _ = oracle.scan_jvp2(x, w, v, p)
    assert relerr(a, b) < 1e-13
    (_, _, _, c), _ = oracle.scan_jvp2(x, 2.5 * v, -0.5 * w, p)
    assert relerr(c, -1.25 * a) < 1e-13
    v2 = np.random.default_rng(25).standard_normal(v.shape)
    (_, _, _, d1), _ = oracle.scan_jvp2(x, v2, w, p)
    (_, _, _, d12), _ = oracle.scan_jvp2(x, v + v2, w, p)
    assert relerr(d12, a + d1) < 1e-12


def test_linear_map_has_zero_second_derivative():
    """w_delta = 0 and W_B = W_C = 0 make y linear in x (constant Delta, B, C
    from the biases): every mixed second derivative is exactly zero."""
    p, x, v, w = problem(26, L=16)
    p = dict(p, w_delta=np.zeros(3), W_B=np.zeros((3, 4)), W_C=np.zeros((3, 4)))
    (_, _, _, yvw), st = oracle.scan_jvp2(x, v, w, p)
    assert np.all(yvw == 0.0) and np.all(st[3] == 0.0)


def test_quadratic_map_closed_form():
    """With Delta constant (w_delta = 0) and C constant (W_C = 0), y is
    quadratic in x through b = Delta*(x W_B + b_B)*x, so
    y_vw,t = sum_n C_n sum_{s<=t} exp((t-s) Delta A_n) Delta
             (v_s.W_B[:,n] w_s + w_s.W_B[:,n] v_s)."""
    g = np.random.default_rng(27)
    D, N, L = 3, 4, 14
    p = dict(A=-g.uniform(0.1, 2, (D, N)), w_delta=np.zeros(D), b_delta=g.uniform(-2, 1, D),
             W_B=g.standard_normal((D, N)), W_C=np.zeros((D, N)), b_B=g.standard_normal(N),
             b_C=g.standard_normal(N))
    x = g.standard_normal((1, L, D)); v = g.standard_normal((1, L, D)); w = g.standard_normal((1, L, D))
    (_, _, _, yvw), _ = oracle.scan_jvp2(x, v, w, p)
    delta = np.log1p(np.exp(p["b_delta"]))
    vW = v[0] @ p["W_B"]                    # [L, N]
    wW = w[0] @ p["W_B"]
    ref = np.zeros((L, D))
    for t in range(L):
        for s in range(t + 1):
            decay = np.exp((t - s) * delta[:, None] * p["A"])               # [D, N]
            drive = delta[:, None] * (vW[s][None, :] * w[0, s][:, None] + wW[s][None, :] * v[0, s][:, None])
            ref[t] += (p["b_C"][None, :] * decay * drive).sum(-1)
    assert relerr(yvw[0], ref) < 1e-13


def test_zero_ahead_of_the_directions():
    p, x, v, w = problem(28, L=25)
    t0 = 11
    v[:, :t0] = 0.0
    (_, yv, _, yvw), _ = oracle.scan_jvp2(x, v, w, p)
    assert np.all(yvw[:, :t0] == 0.0) and np.all(yv[:, :t0] == 0.0)
    assert np.all(np.abs(yvw[:, t0:]).sum(-1) > 0)


def test_segment_composition_closed_forms():
    """Over a block of steps, the exit state from entry state (h, hv, hw, hvw)
    equals P h + h0, P hv + P_v h + hv0, P hw + P_w h + hw0 and
    P hvw + P_w hv + P_v hw + P_vw h + hvw0, with P = exp(A S), P_v = P A S_v,
    P_w = P A S_w, P_vw = P (A S_v)(A S_w) + P A S_vw (S* the block sums of
    Delta and its derivatives) and *0 the exit state from a zero start:
    the composition the L-parallel evaluation uses."""
    p, x, v, w = problem(29, B=2, L=17)
    g = np.random.default_rng(30)
    ent = tuple(g.standard_normal((2, 3, 4)) for _ in range(4))
    _, z = oracle.scan_jvp2(x, v, w, p)
    _, e = oracle.scan_jvp2(x, v, w, p, state=ent)
    delta, dv, dw, dvw = oracle.discretize2(x, v, w, p["w_delta"], p["b_delta"])
    A = p["A"][None]
    S, Sv, Sw, Svw = (a.sum(1)[:, :, None] for a in (delta, dv, dw, dvw))
    P = np.exp(A * S)
    Pv, Pw = P * A * Sv, P * A * Sw
    Pvw = P * (A * Sv) * (A * Sw) + P * A * Svw
    h, hv, hw, hvw = ent
    assert relerr(e[0], P * h + z[0]) < 1e-13
    assert relerr(e[1], P * hv + Pv * h + z[1]) < 1e-13
    assert relerr(e[2], P * hw + Pw * h + z[2]) < 1e-13
    assert relerr(e[3], P * hvw + Pw * hv + Pv * hw + Pvw * h + z[3]) < 1e-13


def test_chunked_equals_whole():
    p, x, v, w = problem(31, B=2, L=33)
    a, sa = oracle.scan_jvp2(x, v, w, p)
    b, sb = oracle.scan_jvp2(x, v, w, p, chunk=7)
    for i in range(4):
        assert relerr(b[i], a[i]) < 1e-15 and relerr(sb[i], sa[i]) < 1e-15
