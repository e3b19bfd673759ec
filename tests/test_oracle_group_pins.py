"""Pins of the oracle's channel groups (survey row f, NEXT-3: Mamba-style
grouped B and C): channel d reads the B, C of group d // (D/G).  Pinned to
the ungrouped oracle when the groups share their weights, and to
forward-mode autograd of an independent torch loop that gathers each
channel's B and C; a planted mis-assignment of groups is caught."""
import numpy as np
import torch

from oracle import oracle
from tests.test_oracle_pins import rand_problem, relerr


def problem(seed, G=3, D=6, N=4, L=12, K=2):
    p, x, dx = rand_problem(seed, B=2, L=L, D=D, N=N, K=K, bias=True)
    r = np.random.default_rng(seed + 300)
    p.update(n_groups=G, W_B=r.standard_normal((D, G * N)) / np.sqrt(D), W_C=r.standard_normal((D, G * N)) / np.sqrt(D),
             b_B=r.standard_normal(G * N), b_C=r.standard_normal(G * N))
    return p, x, dx


def test_shared_group_weights_equal_one_group():
    p, x, dx = rand_problem(90, B=2, L=10, D=6, N=3, K=2, bias=True)
    a = oracle.scan_jvp(x, dx, p)
    G = 3
    p2 = dict(p, n_groups=G, W_B=np.tile(p["W_B"], (1, G)), W_C=np.tile(p["W_C"], (1, G)),
              b_B=np.tile(p["b_B"], G), b_C=np.tile(p["b_C"], G))
    b = oracle.scan_jvp(x, dx, p2)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def _torch_grouped(p, xt):
    f64 = dict(dtype=torch.float64)
    D = xt.shape[-1]
    G = p["n_groups"]
    N = p["A"].shape[1]
    z = xt * torch.tensor(p["w_delta"], **f64) + torch.tensor(p["b_delta"], **f64)
    delta = torch.logaddexp(z, torch.zeros((), **f64))
    Bg = (xt @ torch.tensor(p["W_B"], **f64) + torch.tensor(p["b_B"], **f64)).reshape(*xt.shape[:2], G, N)
    Cg = (xt @ torch.tensor(p["W_C"], **f64) + torch.tensor(p["b_C"], **f64)).reshape(*xt.shape[:2], G, N)
    gidx = torch.arange(D) // (D // G)
    Bd, Cd = Bg[:, :, gidx], Cg[:, :, gidx]            # [B, L, D, N] per channel
    A = torch.tensor(p["A"], **f64)
    h = torch.zeros(xt.shape[0], D, N, **f64)
    ys = []
    for t in range(xt.shape[1]):
        dl = delta[:, t, :, None]
        h = torch.exp(dl * A) * h + dl * Bd[:, t] * xt[:, t, :, None]
        ys.append((h * Cd[:, t]).sum(-1))
    return torch.stack(ys, 1)


def test_forward_mode_autograd():
    p, x, dx = problem(91)
    y, dy, _, _ = oracle.scan_jvp(x, dx, p)
    f = lambda xt: _torch_grouped(p, xt)
    assert relerr(y, f(torch.tensor(x)).numpy()) < 1e-12
    for k in range(dx.shape[0]):
        _, jv = torch.func.jvp(f, (torch.tensor(x),), (torch.tensor(dx[k]),))
        assert relerr(dy[k], jv.numpy()) < 1e-12


def test_interleaved_groups_are_caught(monkeypatch):
    """A planted mistake: groups interleaved (d % G) instead of contiguous."""
    monkeypatch.setattr(oracle, "channel_groups", lambda ch, D, G: np.asarray(ch) % G)
    try:
        test_forward_mode_autograd()
    except AssertionError:
        return
    raise AssertionError("interleaved groups were not caught")
