"""Pins of the parameter-flow oracle (App. E, Alg. 2: sensitivity flows of
A and of per-lane offsets of B and C, accumulated against an adjoint
signal) against facts that do not come from its own formula: reverse-mode
autograd of an independent torch loop, central differences of the
separately pinned primal, a closed form for a time-invariant system, the
outer-product form of G_C at a one-step adjoint, and the segment
composition the GPU carry uses."""
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


def problem(seed, B=2, L=14, D=3, N=4, stiff=False):
    p, x, _ = rand_problem(seed, B=B, L=L, D=D, N=N, K=1, stiff=stiff, bias=True)
    gy = np.random.default_rng(seed + 1000).standard_normal(x.shape)
    return p, x, gy


def _torch_loss(p, x, gy, A, beta_B, beta_C, drive="euler", act="identity", D_res=None, w_delta=None,
                b_delta=None):
    """l = sum gy*y of the selective scan as a plain torch loop, with the
    per-lane offsets beta_B, beta_C [D,N] added to B_t and C_t; drive "zoh"
    takes b = expm1(Delta A)/A * B x (A != 0 everywhere here); act "silu"
    and D_res [D] (a tensor) give y = silu(C h + D_res x); w_delta, b_delta
    (tensors) replace the step size's parameters of p."""
    xt = torch.tensor(x)
    w_delta = torch.tensor(p["w_delta"]) if w_delta is None else w_delta
    b_delta = torch.tensor(p["b_delta"]) if b_delta is None else b_delta
    z = xt * w_delta + b_delta
    delta = torch.logaddexp(z, torch.zeros((), dtype=torch.float64))
    Bm = xt @ torch.tensor(p["W_B"]) + torch.tensor(p["b_B"])
    Cm = xt @ torch.tensor(p["W_C"]) + torch.tensor(p["b_C"])
    Bsz, L, D = xt.shape
    h = torch.zeros(Bsz, D, A.shape[1], dtype=torch.float64)
    loss = torch.zeros((), dtype=torch.float64)
    for t in range(L):
        dl = delta[:, t, :, None]
        Bt = Bm[:, t, None, :] + beta_B
        Ct = Cm[:, t, None, :] + beta_C
        e = torch.expm1(dl * A) / A if drive == "zoh" else dl
        h = torch.exp(dl * A) * h + e * Bt * xt[:, t, :, None]
        yt = (h * Ct).sum(-1)
        if D_res is not None:
            yt = yt + D_res * xt[:, t]
        if act == "silu":
            yt = torch.nn.functional.silu(yt)
        loss = loss + (torch.tensor(gy[:, t]) * yt).sum()
    return loss


@pytest.mark.parametrize("seed,stiff", [(40, False), (41, True)])
def test_reverse_mode_autograd(seed, stiff):
    p, x, gy = problem(seed, stiff=stiff)
    y, (GA, GB, GC), _ = oracle.param_grads(x, gy, p)
    A = torch.tensor(p["A"], requires_grad=True)
    bB = torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    bC = torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    _torch_loss(p, x, gy, A, bB, bC).backward()
    assert relerr(GA, A.grad.numpy()) < 1e-12
    assert relerr(GB, bB.grad.numpy()) < 1e-12
    assert relerr(GC, bC.grad.numpy()) < 1e-12


def _loss_np(p, x, gy):
    y, _, _, _ = oracle.scan_jvp(x, x[None] * 0.0, p)
    return float((gy * y).sum())


def test_central_differences_of_the_primal():
    """Directional derivatives of l along A, b_B and b_C from the pinned
    first-order oracle's primal: <G_A, dA>, <sum_d G_B, db_B>, <sum_d G_C, db_C>."""
    p, x, gy = problem(42, L=18)
    _, (GA, GB, GC), _ = oracle.param_grads(x, gy, p)
    g = np.random.default_rng(43)
    eps = 1e-6
    dA = g.standard_normal(p["A"].shape)
    fd = (_loss_np(dict(p, A=p["A"] + eps * dA), x, gy) - _loss_np(dict(p, A=p["A"] - eps * dA), x, gy)) / (2 * eps)
    assert abs(fd - (GA * dA).sum()) < 1e-7 * max(1.0, abs(fd))
    for key, G in (("b_B", GB), ("b_C", GC)):
        db = g.standard_normal(p[key].shape)
        fd = (_loss_np(dict(p, **{key: p[key] + eps * db}), x, gy)
              - _loss_np(dict(p, **{key: p[key] - eps * db}), x, gy)) / (2 * eps)
        assert abs(fd - (G.sum(0) * db).sum()) < 1e-7 * max(1.0, abs(fd)), key


def test_time_invariant_closed_form():
    """w_delta = 0, W_B = W_C = 0: Delta, B, C constant, h_t = sum_{s<=t}
    a^(t-s) Delta B x_s with a = exp(Delta A), so dh_t/dA = sum_s (t-s) Delta
    a^(t-s) Delta B x_s, dh_t/dB = sum_s a^(t-s) Delta x_s."""
    g = np.random.default_rng(44)
    D, N, L = 3, 4, 16
    p = dict(A=-g.uniform(0.1, 2, (D, N)), w_delta=np.zeros(D), b_delta=g.uniform(-2, 1, D),
             W_B=np.zeros((D, N)), W_C=np.zeros((D, N)), b_B=g.standard_normal(N), b_C=g.standard_normal(N))
    x = g.standard_normal((1, L, D))
    gy = g.standard_normal((1, L, D))
    _, (GA, GB, GC), _ = oracle.param_grads(x, gy, p)
    dl = np.log1p(np.exp(p["b_delta"]))[:, None]
    a = np.exp(dl * p["A"])
    rA = np.zeros((D, N)); rB = np.zeros((D, N)); rC = np.zeros((D, N))
    for t in range(L):
        h = np.zeros((D, N)); hA = np.zeros((D, N)); hB = np.zeros((D, N))
        for s in range(t + 1):
            k = t - s
            h += a ** k * dl * p["b_B"] * x[0, s][:, None]
            hA += k * dl * a ** k * dl * p["b_B"] * x[0, s][:, None]
            hB += a ** k * dl * x[0, s][:, None]
        gt = gy[0, t][:, None]
        rA += gt * p["b_C"] * hA
        rB += gt * p["b_C"] * hB
        rC += gt * h
    assert relerr(GA, rA) < 1e-12 and relerr(GB, rB) < 1e-12 and relerr(GC, rC) < 1e-12


def test_one_step_adjoint_is_the_outer_product():
    """An adjoint at a single (b, t0, d) gives G_C[d] = gy * h_t0[b, d] with
    h_t0 the state after step t0 from the first-order oracle."""
    p, x, _ = problem(45, B=2, L=20)
    t0, b, d = 11, 1, 2
    gy = np.zeros_like(x)
    gy[b, t0, d] = 1.7
    _, (GA, GB, GC), _ = oracle.param_grads(x, gy, p)
    _, _, h, _ = oracle.scan_jvp(x[:, :t0 + 1], np.zeros((1,) + x[:, :t0 + 1].shape), p)
    ref = np.zeros_like(GC)
    ref[d] = 1.7 * h[b, d]
    assert relerr(GC, ref) < 1e-15
    assert np.all(GA[np.arange(3) != d] == 0) and np.all(GB[np.arange(3) != d] == 0)


def test_linear_in_the_adjoint_and_primal_unchanged():
    p, x, gy = problem(46)
    y, G1, _ = oracle.param_grads(x, gy, p)
    g2 = np.random.default_rng(47).standard_normal(x.shape)
    _, G2, _ = oracle.param_grads(x, g2, p)
    _, G12, _ = oracle.param_grads(x, 2.0 * gy - 0.5 * g2, p)
    for a, b, c in zip(G1, G2, G12):
        assert relerr(c, 2.0 * a - 0.5 * b) < 1e-13
    y1, _, _, _ = oracle.scan_jvp(x, np.zeros((1,) + x.shape), p)
    assert np.array_equal(y, y1)
    _, G0, _ = oracle.param_grads(x, np.zeros_like(x), p)
    assert all(np.all(g == 0) for g in G0)


def test_segment_composition_closed_forms():
    """Over a block with S = sum Delta and P = exp(A S), the exit state from
    entry (h, GA, GB) is (P h + h0, P GA + S P h + GA0, P GB + GB0), with
    *0 the exit state from a zero start: what the L-parallel carry uses."""
    p, x, gy = problem(48, L=17)
    g = np.random.default_rng(49)
    ent = tuple(g.standard_normal((2, 3, 4)) for _ in range(3))
    _, _, z = oracle.param_grads(x, gy, p)
    _, _, e = oracle.param_grads(x, gy, p, state=ent)
    delta, _ = oracle.discretize(x, x[None], p["w_delta"], p["b_delta"])
    S = delta.sum(1)[:, :, None]
    P = np.exp(p["A"][None] * S)
    assert relerr(e[0], P * ent[0] + z[0]) < 1e-13
    assert relerr(e[1], P * ent[1] + S * P * ent[0] + z[1]) < 1e-13
    assert relerr(e[2], P * ent[2] + z[2]) < 1e-13


def test_chunked_equals_whole():
    p, x, gy = problem(50, L=31)
    y, G, st = oracle.param_grads(x, gy, p)
    y2, G2, st2 = oracle.param_grads(x, gy, p, chunk=6)
    assert relerr(y2, y) < 1e-15
    for a, b in zip(G, G2):
        assert relerr(b, a) < 1e-14
    for a, b in zip(st, st2):
        assert relerr(b, a) < 1e-15


# ---------------------------------------------------------------- zero-order-hold drive
# App. E's "A via ZOH" case: the drive e(A) B x with e = expm1(Delta A)/A
# depends on A, so GammaA gains the term (de/dA) B x.

def small_step_problem(seed, B=1, L=30, D=3, N=4):
    """Delta ~ 1.2e-4: |Delta A| < 1e-3, where the oracle takes de/dA from
    its series."""
    p, x, gy = problem(seed, B=B, L=L, D=D, N=N)
    p["b_delta"] = np.full(D, -9.0)
    p["w_delta"] = p["w_delta"] * 0.1
    return p, x, gy


@pytest.mark.parametrize("case", ["normal", "stiff", "small_steps"])
def test_zoh_reverse_mode_autograd(case):
    if case == "small_steps":
        p, x, gy = small_step_problem(60)
    else:
        p, x, gy = problem(61, stiff=case == "stiff")
    _, (GA, GB, GC), _ = oracle.param_grads(x, gy, p, drive="zoh")
    A = torch.tensor(p["A"], requires_grad=True)
    bB = torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    bC = torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    _torch_loss(p, x, gy, A, bB, bC, drive="zoh").backward()
    assert relerr(GA, A.grad.numpy()) < 1e-10
    assert relerr(GB, bB.grad.numpy()) < 1e-12
    assert relerr(GC, bC.grad.numpy()) < 1e-12
    # and the Euler flows differ (the drive's A-dependence is not negligible)
    _, (GA_e, _, _), _ = oracle.param_grads(x, gy, p)
    assert relerr(GA_e, GA) > 1e-6


def _loss_zoh(p, x, gy):
    y, _, _, _ = oracle.scan_jvp(x, x[None] * 0.0, p, drive="zoh")
    return float((gy * y).sum())


@pytest.mark.parametrize("small", [False, True])
def test_zoh_central_differences_along_A(small):
    """<G_A, dA> against central differences of the separately pinned ZOH
    primal, with one column of A exactly 0 (the A = 0 limit of the drive)."""
    p, x, gy = small_step_problem(62) if small else problem(62, L=18)
    p["A"][:, 1] = 0.0
    _, (GA, _, _), _ = oracle.param_grads(x, gy, p, drive="zoh")
    dA = np.random.default_rng(63).standard_normal(p["A"].shape)
    eps = 1e-6 if not small else 1e-3
    fd = (_loss_zoh(dict(p, A=p["A"] + eps * dA), x, gy) - _loss_zoh(dict(p, A=p["A"] - eps * dA), x, gy)) / (2 * eps)
    assert abs(fd - (GA * dA).sum()) < 1e-7 * max(1.0, abs(fd)), (fd, (GA * dA).sum())


def test_zoh_segment_composition_closed_forms():
    """The carry's composition is the same as with the Euler drive: the
    drive's A-dependence is inside the zero-start end state GA0."""
    p, x, gy = problem(64, L=17)
    g = np.random.default_rng(65)
    ent = tuple(g.standard_normal((2, 3, 4)) for _ in range(3))
    _, _, z = oracle.param_grads(x, gy, p, drive="zoh")
    _, _, e = oracle.param_grads(x, gy, p, state=ent, drive="zoh")
    delta, _ = oracle.discretize(x, x[None], p["w_delta"], p["b_delta"])
    S = delta.sum(1)[:, :, None]
    P = np.exp(p["A"][None] * S)
    assert relerr(e[0], P * ent[0] + z[0]) < 1e-13
    assert relerr(e[1], P * ent[1] + S * P * ent[0] + z[1]) < 1e-13
    assert relerr(e[2], P * ent[2] + z[2]) < 1e-13


# ---------------------------------------------------------------- output map
# y = act(C h + D_res x): the adjoint reaches the state through act' (the
# sigma' factor of App. E's G_C update), and D_res gains dl/dD_res = sum gy act' x.

@pytest.mark.parametrize("act,drive,stiff", [("silu", "euler", False), ("silu", "zoh", True),
                                             ("identity", "euler", False)])
def test_output_map_reverse_mode_autograd(act, drive, stiff):
    p, x, gy = problem(70, stiff=stiff)
    p["D_res"] = np.random.default_rng(71).standard_normal(p["A"].shape[0])
    y, (GA, GB, GC, GD), _ = oracle.param_grads(x, gy, p, drive=drive, act=act)
    A = torch.tensor(p["A"], requires_grad=True)
    bB = torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    bC = torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    Dr = torch.tensor(p["D_res"], requires_grad=True)
    _torch_loss(p, x, gy, A, bB, bC, drive=drive, act=act, D_res=Dr).backward()
    tolA = 1e-10 if drive == "zoh" else 1e-12
    assert relerr(GA, A.grad.numpy()) < tolA
    assert relerr(GB, bB.grad.numpy()) < 1e-12
    assert relerr(GC, bC.grad.numpy()) < 1e-12
    assert relerr(GD, Dr.grad.numpy()) < 1e-12
    # the primal is the first-order oracle's, output map included
    y1, _, _, _ = oracle.scan_jvp(x, np.zeros((1,) + x.shape), p, drive=drive, act=act)
    assert relerr(y, y1) < 1e-14


def test_output_map_identity_residual_closed_form():
    """With the identity map, y = C h + D_res x: the flows of A, B, C are
    those without D_res, and dl/dD_res[d] = sum_{b,t} gy x."""
    p, x, gy = problem(72)
    _, G0, _ = oracle.param_grads(x, gy, p)
    p["D_res"] = np.random.default_rng(73).standard_normal(p["A"].shape[0])
    _, G, _ = oracle.param_grads(x, gy, p)
    for a, b in zip(G0, G[:3]):
        assert relerr(b, a) < 1e-15
    assert relerr(G[3], (gy * x).sum((0, 1))) < 1e-14


def _loss_map(p, x, gy, act):
    y, _, _, _ = oracle.scan_jvp(x, x[None] * 0.0, p, act=act)
    return float((gy * y).sum())


def test_output_map_central_differences():
    """<G, dP> along A, b_C and D_res against central differences of the
    separately pinned first-order primal with the SiLU map."""
    p, x, gy = problem(74, L=18)
    p["D_res"] = np.random.default_rng(75).standard_normal(p["A"].shape[0])
    _, (GA, GB, GC, GD), _ = oracle.param_grads(x, gy, p, act="silu")
    g = np.random.default_rng(76)
    eps = 1e-6
    for key, G in (("A", GA), ("b_B", GB.sum(0)), ("b_C", GC.sum(0)), ("D_res", GD)):
        dP = g.standard_normal(p[key].shape)
        fd = (_loss_map(dict(p, **{key: p[key] + eps * dP}), x, gy, "silu")
              - _loss_map(dict(p, **{key: p[key] - eps * dP}), x, gy, "silu")) / (2 * eps)
        assert abs(fd - (G * dP).sum()) < 1e-7 * max(1.0, abs(fd)), (key, fd, (G * dP).sum())


def test_output_map_one_step_adjoint():
    """An adjoint at one (b, t0, d): G_C[d] = gy * silu'(yhat) * h_t0 and
    G_D[d] = gy * silu'(yhat) * x, with yhat from the first-order primal
    (identity map) at that step: the sigma' factor of the G_C update."""
    p, x, _ = problem(77, B=2, L=20)
    p["D_res"] = np.random.default_rng(78).standard_normal(3)
    t0, b, d = 9, 0, 1
    gy = np.zeros_like(x)
    gy[b, t0, d] = -0.8
    _, (GA, GB, GC, GD), _ = oracle.param_grads(x, gy, p, act="silu")
    yh, _, h, _ = oracle.scan_jvp(x[:, :t0 + 1], np.zeros((1,) + x[:, :t0 + 1].shape), p)
    v = yh[b, t0, d]
    sg = 1.0 / (1.0 + np.exp(-v))
    w = -0.8 * (sg + v * sg * (1.0 - sg))
    ref = np.zeros_like(GC)
    ref[d] = w * h[b, d]
    assert relerr(GC, ref) < 1e-14
    refD = np.zeros(3)
    refD[d] = w * x[b, t0, d]
    assert relerr(GD, refD) < 1e-14


# ---------------------------------------------------------------- step-size parameters
# Delta = softplus(w_delta x + b_delta): the flows Gamma_w = dh/dw_delta and
# Gamma_s = dh/db_delta, driven by dh'/dDelta times sigma*x and sigma.

@pytest.mark.parametrize("drive,act,stiff", [("euler", "identity", False), ("zoh", "identity", True),
                                             ("euler", "silu", False), ("zoh", "silu", False)])
def test_step_size_reverse_mode_autograd(drive, act, stiff):
    p, x, gy = problem(80, stiff=stiff)
    if act == "silu":
        p["D_res"] = np.random.default_rng(81).standard_normal(p["A"].shape[0])
    y, G, _ = oracle.param_grads(x, gy, p, drive=drive, act=act, delta_params=True)
    GW, GS = G[-2], G[-1]
    A = torch.tensor(p["A"], requires_grad=True)
    zero = lambda: torch.zeros(p["A"].shape, dtype=torch.float64, requires_grad=True)
    bB, bC = zero(), zero()
    w = torch.tensor(p["w_delta"], requires_grad=True)
    b = torch.tensor(p["b_delta"], requires_grad=True)
    Dr = None if act != "silu" else torch.tensor(p["D_res"])
    _torch_loss(p, x, gy, A, bB, bC, drive=drive, act=act, D_res=Dr, w_delta=w, b_delta=b).backward()
    assert relerr(GW, w.grad.numpy()) < 1e-11
    assert relerr(GS, b.grad.numpy()) < 1e-11
    # the other gradients and the primal do not change with the extra flows
    y0, G0, _ = oracle.param_grads(x, gy, p, drive=drive, act=act)
    assert np.array_equal(y, y0) and all(np.array_equal(a, c) for a, c in zip(G0, G[:len(G0)]))
    assert relerr(G[0], A.grad.numpy()) < (1e-10 if drive == "zoh" else 1e-12)


def test_step_size_central_differences():
    """<G_w, dw> and <G_s, db> against central differences of the separately
    pinned first-order primal (ZOH drive, SiLU map, residual weight)."""
    p, x, gy = problem(82, L=18)
    p["D_res"] = np.random.default_rng(83).standard_normal(p["A"].shape[0])
    _, G, _ = oracle.param_grads(x, gy, p, drive="zoh", act="silu", delta_params=True)

    def loss(q):
        y, _, _, _ = oracle.scan_jvp(x, x[None] * 0.0, q, drive="zoh", act="silu")
        return float((gy * y).sum())

    g = np.random.default_rng(84)
    eps = 1e-6
    for key, Gk in (("w_delta", G[-2]), ("b_delta", G[-1])):
        dP = g.standard_normal(p[key].shape)
        fd = (loss(dict(p, **{key: p[key] + eps * dP})) - loss(dict(p, **{key: p[key] - eps * dP}))) / (2 * eps)
        assert abs(fd - (Gk * dP).sum()) < 1e-7 * max(1.0, abs(fd)), (key, fd, (Gk * dP).sum())


def test_step_size_segment_composition_and_chunks():
    """Over a block with S = sum Delta, P = exp(A S), the step-size flows'
    exit state from entry (h, .., Gamma_w, Gamma_s) is P Gamma + P A S_theta h
    + Gamma0 (Gamma0 from a zero start, S_theta = sum sigma x for w and
    sum sigma for b): the carry the GPU uses.  Chunked evaluation equals one
    pass."""
    p, x, gy = problem(85, L=17)
    g = np.random.default_rng(86)
    ent = tuple(g.standard_normal((2, 3, 4)) for _ in range(5))
    _, _, z = oracle.param_grads(x, gy, p, delta_params=True)
    _, _, e = oracle.param_grads(x, gy, p, state=ent, delta_params=True)
    delta, _ = oracle.discretize(x, x[None], p["w_delta"], p["b_delta"])
    sg = 1.0 / (1.0 + np.exp(-(x * p["w_delta"] + p["b_delta"])))
    S = delta.sum(1)[:, :, None]
    P = np.exp(p["A"][None] * S)
    Sw = (sg * x).sum(1)[:, :, None]
    Ss = sg.sum(1)[:, :, None]
    assert relerr(e[3], P * ent[3] + P * p["A"][None] * Sw * ent[0] + z[3]) < 1e-13
    assert relerr(e[4], P * ent[4] + P * p["A"][None] * Ss * ent[0] + z[4]) < 1e-13
    y, G, st = oracle.param_grads(x, gy, p, delta_params=True)
    y2, G2, st2 = oracle.param_grads(x, gy, p, chunk=5, delta_params=True)
    assert relerr(y2, y) < 1e-15
    for a, b in zip(G + st, G2 + st2):
        assert relerr(b, a) < 1e-13


def test_step_size_one_step_adjoint():
    """An adjoint at one (b, t0, d) and a single step: from a zero state,
    h_1 = Delta B x, so dh_1/dDelta = B x and G_s = gy sigma sum_n C B x,
    G_w = G_s x (Euler drive, identity map)."""
    p, x, _ = problem(87, B=1, L=1)
    gy = np.zeros_like(x)
    gy[0, 0, 2] = 1.3
    _, G, _ = oracle.param_grads(x, gy, p, delta_params=True)
    Bm, Cm, _, _ = oracle.project(x, x[None], p["W_B"], p["W_C"], p["b_B"], p["b_C"])
    xv = x[0, 0, 2]
    sg = 1.0 / (1.0 + np.exp(-(xv * p["w_delta"][2] + p["b_delta"][2])))
    ref_s = 1.3 * sg * (Cm[0, 0] * Bm[0, 0]).sum() * xv
    assert abs(G[-1][2] - ref_s) < 1e-14 * abs(ref_s) and abs(G[-2][2] - ref_s * xv) < 1e-14 * abs(ref_s * xv)
    assert np.all(G[-1][[0, 1]] == 0) and np.all(G[-2][[0, 1]] == 0)



def test_step_size_summation_scale():
    """The scale returned beside dl/dw_delta and dl/db_delta is the sum of
    the absolute values of their terms: at least |G|, equal to it for a
    single nonzero adjoint, and additive over the batch."""
    p, x, gy = problem(88)
    _, G, _, sc = oracle.param_grads(x, gy, p, delta_params=True, return_scale=True)
    assert np.all(sc[0] >= np.abs(G[-2]) - 1e-15) and np.all(sc[1] >= np.abs(G[-1]) - 1e-15)
    assert np.all(sc[0] > np.abs(G[-2])) and np.all(sc[1] > np.abs(G[-1]))
    one = np.zeros_like(gy)
    one[1, 7, 0] = -2.0
    _, G1, _, sc1 = oracle.param_grads(x, one, p, delta_params=True, return_scale=True)
    assert sc1[0][0] == abs(G1[-2][0]) and sc1[1][0] == abs(G1[-1][0])
    _, _, _, sa = oracle.param_grads(x[:1], gy[:1], p, delta_params=True, return_scale=True)
    _, _, _, sb = oracle.param_grads(x[1:], gy[1:], p, delta_params=True, return_scale=True)
    assert relerr(sa[0] + sb[0], sc[0]) < 1e-15 and relerr(sa[1] + sb[1], sc[1]) < 1e-15
