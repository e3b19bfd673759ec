"""Pins of the decaying-linear-attention oracle (App. F) against facts that
do not come from its recurrence: the parallel (attention) form of the same
map, RetNet's and the undecayed linear transformer's closed forms,
forward-mode autograd of an independent torch loop, central differences,
and the segment composition a blocked evaluation uses; planted mistakes
are caught."""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest
import torch

from oracle import oracle


def relerr(a, b):
    return np.linalg.norm((np.asarray(a) - np.asarray(b)).ravel()) / max(np.linalg.norm(np.ravel(b)), 1e-300)


def problem(seed, B=2, H=2, L=12, DK=4, DV=3, K=2, decay="data"):
    r = np.random.default_rng(seed)
    q, k = r.standard_normal((2, B, H, L, DK))
    v = r.standard_normal((B, H, L, DV))
    if decay == "data":
        g = -np.exp(r.uniform(-4, 0, (B, H, L, DK)))
    elif decay == "retnet":
        g = np.broadcast_to(np.log(r.uniform(0.5, 0.99, (1, H, 1, 1))), (B, H, L, DK)).copy()
    else:
        g = np.zeros((B, H, L, DK))
    dq, dk, dg = r.standard_normal((3, K, B, H, L, DK))
    dv = r.standard_normal((K, B, H, L, DV))
    return q, k, v, g, dq, dk, dv, dg


def attention_form(q, k, v, g, S0=None):
    """o_t = sum_{s<=t} sum_i q_t[i] k_s[i] exp(G_t[i] - G_s[i]) v_s + the
    decayed entry state, G the cumulative log-decay."""
    G = np.cumsum(g, axis=2)
    B, H, L, DK = q.shape
    o = np.zeros(v.shape[:3] + (v.shape[-1],))
    for t in range(L):
        w = np.exp(G[:, :, t:t + 1] - G[:, :, :t + 1])                  # [B,H,s,DK]
        att = np.einsum("bhi,bhsi->bhs", q[:, :, t], k[:, :, :t + 1] * w)
        o[:, :, t] = np.einsum("bhs,bhsj->bhj", att, v[:, :, :t + 1])
        if S0 is not None:
            o[:, :, t] += np.einsum("bhi,bhij->bhj", q[:, :, t] * np.exp(G[:, :, t]), S0)
    return o


def test_parallel_attention_form():
    q, k, v, g, dq, dk, dv, dg = problem(70)
    S0 = np.random.default_rng(71).standard_normal((2, 2, 4, 3))
    o, _, _, _ = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg, state=(S0, np.zeros((2, 2, 2, 4, 3))))
    assert relerr(o, attention_form(q, k, v, g, S0)) < 1e-13


def test_retnet_and_linear_transformer_closed_forms():
    q, k, v, g, dq, dk, dv, dg = problem(72, decay="retnet")
    o, _, _, _ = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg)
    gam = np.exp(g[:, :, 0, 0])                                          # [B,H]
    L = q.shape[2]
    t, s = np.arange(L)[:, None], np.arange(L)[None, :]
    mask = np.where(s <= t, gam[..., None, None] ** np.maximum(t - s, 0), 0.0)   # [B,H,L,L]
    ref = np.einsum("bhts,bhsj->bhtj", np.einsum("bhti,bhsi->bhts", q, k) * mask, v)
    assert relerr(o, ref) < 1e-13
    q, k, v, g, dq, dk, dv, dg = problem(73, decay="none")
    o, _, _, _ = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg)
    Sc = np.cumsum(np.einsum("bhti,bhtj->bhtij", k, v), axis=2)
    assert relerr(o, np.einsum("bhti,bhtij->bhtj", q, Sc)) < 1e-13


def _torch_la(q, k, v, g):
    B, H, L, DK = q.shape
    S = torch.zeros(B, H, DK, v.shape[-1], dtype=torch.float64)
    outs = []
    for t in range(L):
        S = torch.exp(g[:, :, t])[..., None] * S + k[:, :, t, :, None] * v[:, :, t, None, :]
        outs.append((q[:, :, t, :, None] * S).sum(-2))
    return torch.stack(outs, 2)


@pytest.mark.parametrize("decay", ["data", "retnet"])
def test_forward_mode_autograd(decay):
    q, k, v, g, dq, dk, dv, dg = problem(74, decay=decay)
    o, do, _, _ = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg)
    T = lambda a: torch.tensor(a, dtype=torch.float64)
    for kk in range(dq.shape[0]):
        _, jv = torch.func.jvp(_torch_la, (T(q), T(k), T(v), T(g)), (T(dq[kk]), T(dk[kk]), T(dv[kk]), T(dg[kk])))
        assert relerr(do[kk], jv.numpy()) < 1e-12, kk


def test_central_differences():
    q, k, v, g, dq, dk, dv, dg = problem(75, L=20, K=1)
    _, do, _, _ = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg)
    eps = 1e-6
    shift = lambda sgn: [u + sgn * eps * du[0] for u, du in ((q, dq), (k, dk), (v, dv), (g, dg))]
    op, _, _, _ = oracle.la_scan_jvp(*shift(1), dq, dk, dv, dg)
    om, _, _, _ = oracle.la_scan_jvp(*shift(-1), dq, dk, dv, dg)
    assert relerr(do[0], (op - om) / (2 * eps)) < 1e-8


def test_segment_composition_closed_forms():
    """Over a block, the exit state from entry (S, dS) is (P S + S0,
    P dS + P sum(dg) S + dS0) with P = exp(sum g) per key dimension."""
    q, k, v, g, dq, dk, dv, dg = problem(76, L=15, K=1)
    r = np.random.default_rng(77)
    ent = (r.standard_normal((2, 2, 4, 3)), r.standard_normal((1, 2, 2, 4, 3)))
    _, _, S0, dS0 = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg)
    _, _, S1, dS1 = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg, state=ent)
    P = np.exp(g.sum(2))[..., None]                       # [B,H,DK,1]
    Q = P * dg[0].sum(2)[..., None]
    assert relerr(S1, P * ent[0] + S0) < 1e-13
    assert relerr(dS1[0], P * ent[1][0] + Q * ent[0] + dS0[0]) < 1e-13


def test_chunked_and_linear_in_the_direction():
    q, k, v, g, dq, dk, dv, dg = problem(78, L=23)
    a = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg)
    b = oracle.la_scan_jvp(q, k, v, g, dq, dk, dv, dg, chunk=5)
    for u, w in zip(a, b):
        assert relerr(w, u) < 1e-14
    c = oracle.la_scan_jvp(q, k, v, g, 2 * dq[:1] - dq[1:], 2 * dk[:1] - dk[1:], 2 * dv[:1] - dv[1:],
                           2 * dg[:1] - dg[1:])
    assert relerr(c[1][0], 2 * a[1][0] - a[1][1]) < 1e-13


PIN_TESTS = [test_parallel_attention_form, lambda: test_forward_mode_autograd("data"),
             test_segment_composition_closed_forms]

C_MUTANTS = {
    "drop the decay-variation term": ("+ alpha * dg[tk] * sprev ", ""),
    "decay variation without alpha": ("+ alpha * dg[tk] * sprev ", "+ dg[tk] * sprev "),
    "decay variation on the new state": ("+ alpha * dg[tk] * sprev ", "+ alpha * dg[tk] * (alpha * sprev) "),
    "drop dk*v": ("+ dk[tk] * v[rv] ", ""),
    "drop k*dv": ("+ k[rk + i] * dv[tv];", ";"),
    "output tangent without dq*S": ("do_[tv] += dq[tk] * snew + q[rk + i] * dsnew;", "do_[tv] += q[rk + i] * dsnew;"),
    "decay after the update": ("const double snew = alpha * sprev + k[rk + i] * v[rv];",
                               "const double snew = alpha * (sprev + k[rk + i] * v[rv]);"),
    "output from the old state": ("ot += q[rk + i] * snew;", "ot += q[rk + i] * sprev;"),
}


def _caught():
    for t in PIN_TESTS:
        try:
            t()
        except AssertionError:
            return True
    return False


def test_unmutated_oracle_passes_la_pins():
    assert not _caught()


@pytest.mark.parametrize("name", sorted(C_MUTANTS))
def test_la_c_mutant_is_caught(name, monkeypatch):
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
